// Randomized driver for the host routing library (include/eldr_route.h), built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_routing_sanitized.py: every entry point on random shapes, sparse
// counts, repeated layers, zero signatures, ties, tau of 0, 0.1, 1, negative,
// NaN and infinite, and NaN signatures and centroids.  Return codes are not
// checked here (the parity tests do that); the sanitizers report any invalid
// memory access or undefined behaviour.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>
#include "eldr_route.h"
int main() {
  std::mt19937 rng(1234);
  auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  auto F = [&]() { return std::uniform_real_distribution<float>(-1.f, 1.f)(rng); };
  int calls = 0, errs = 0;
  for (int it = 0; it < 400; ++it) {
    const int N = U(1, 40), L = U(1, 6), E = U(1, 20), K = U(1, std::min(N, 8));
    std::vector<int32_t> counts((size_t)N * L * E);
    for (auto& c : counts) c = (U(0, 3) == 0) ? U(0, 50) : 0;
    std::vector<float> idf((size_t)L * E);
    errs += eldr_idf(counts.data(), N, L, E, idf.data()) != 0; ++calls;
    const int nl = U(1, L);
    std::vector<int32_t> layers(nl);
    for (auto& l : layers) l = U(0, L - 1);
    const int d = nl * E;
    std::vector<float> S((size_t)N * d);
    for (int n = 0; n < N; ++n)
      errs += eldr_signature(counts.data() + (size_t)n * L * E, idf.data(), L, E, layers.data(), nl,
                             S.data() + (size_t)n * d) != 0, ++calls;
    const int dp = U(1, 10);
    std::vector<float> P((size_t)N * dp);
    for (auto& p : P) p = std::fabs(F());
    const int np = U(0, 30);
    std::vector<int32_t> pairs((size_t)np * 2 + 2);
    for (int i = 0; i < np; ++i) { pairs[2 * i] = U(0, N - 1); pairs[2 * i + 1] = U(0, N - 1); }
    double rho = 0;
    eldr_rho(S.data(), N, d, P.data(), dp, pairs.data(), np, &rho); ++calls;
    std::vector<int32_t> order(L); std::vector<double> curve(L); int32_t nstar = 0;
    eldr_greedy_layers(counts.data(), N, L, E, idf.data(), P.data(), dp, pairs.data(), np, order.data(),
                       curve.data(), &nstar); ++calls;
    std::vector<int32_t> init(K);
    for (int k = 0; k < K; ++k) init[k] = U(0, N - 1);
    std::vector<float> cent((size_t)K * d); std::vector<int32_t> assign(N); int32_t iters = 0;
    eldr_balanced_kmeans(S.data(), N, d, K, init.data(), U(0, 20), cent.data(), assign.data(), &iters); ++calls;
    std::vector<int32_t> loads(K);
    for (auto& l : loads) l = U(0, 5);
    const float taus[] = {0.f, 0.1f, 1.f, -0.1f, NAN, INFINITY};
    for (float tau : taus) {
      int32_t w = -2;
      eldr_route(S.data(), d, cent.data(), K, loads.data(), tau, &w); ++calls;
      std::vector<int32_t> ws(N); std::vector<int32_t> l2 = loads;
      eldr_route_batch(S.data(), N, d, cent.data(), K, l2.data(), tau, ws.data()); ++calls;
    }
    // a NaN signature and a NaN centroid
    std::vector<float> sn(S.begin(), S.begin() + d); sn[0] = NAN;
    int32_t w = -2;
    eldr_route(sn.data(), d, cent.data(), K, loads.data(), 0.1f, &w); ++calls;
    std::vector<float> cn = cent; cn[0] = NAN;
    eldr_route(S.data(), d, cn.data(), K, loads.data(), 0.1f, &w); ++calls;
  }
  // one worker, one dimension, a zero signature
  {
    float z = 0.f;
    int32_t one_load = 0, w1 = -2;
    eldr_route(&z, 1, &z, 1, &one_load, 0.1f, &w1);
  }
  printf("calls %d, signature errors %d\n", calls, errs);
  return 0;
}
