// ELDR's expert signature, offline fit and locality-band routing: native host
// code (Design: Expert Signature, Offline clustering, Online routing).
//
// The greedy layer search evaluates rho for O(L^2) layer sets.  A signature's
// cosine distances only need dot products and norms of the IDF-weighted
// counts, and both are sums over layers, so they are precomputed per layer
// (per pair for the dots, per request for the norms) and each trial set
// costs O(pairs), not O(pairs * E * layers).
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <limits>
#include <numeric>
#include <cmath>
#include <vector>

#include "eldr_route.h"

namespace {

double cos_dist(const double* a, const double* b, int n) {
  double ab = 0.0, aa = 0.0, bb = 0.0;
  for (int i = 0; i < n; ++i) {
    ab += a[i] * b[i];
    aa += a[i] * a[i];
    bb += b[i] * b[i];
  }
  if (aa == 0.0 || bb == 0.0) return 1.0;
  return 1.0 - ab / (sqrt(aa) * sqrt(bb));
}

// Fractional ranks (ties get the mean of the ranks they span), 1-based.
std::vector<double> ranks(const std::vector<double>& x) {
  const size_t n = x.size();
  std::vector<size_t> idx(n);
  std::iota(idx.begin(), idx.end(), 0);
  std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) { return x[a] < x[b]; });
  std::vector<double> r(n);
  size_t i = 0;
  while (i < n) {
    size_t j = i;
    while (j + 1 < n && x[idx[j + 1]] == x[idx[i]]) ++j;
    const double avg = 0.5 * (double)(i + j) + 1.0;
    for (size_t k = i; k <= j; ++k) r[idx[k]] = avg;
    i = j + 1;
  }
  return r;
}

// Spearman rank correlation = Pearson correlation of the fractional ranks.
double spearman(const std::vector<double>& a, const std::vector<double>& b) {
  const size_t n = a.size();
  if (n < 2) return 0.0;
  const auto ra = ranks(a), rb = ranks(b);
  double ma = 0.0, mb = 0.0;
  for (size_t i = 0; i < n; ++i) {
    ma += ra[i];
    mb += rb[i];
  }
  ma /= (double)n;
  mb /= (double)n;
  double sab = 0.0, saa = 0.0, sbb = 0.0;
  for (size_t i = 0; i < n; ++i) {
    const double da = ra[i] - ma, db = rb[i] - mb;
    sab += da * db;
    saa += da * da;
    sbb += db * db;
  }
  if (saa == 0.0 || sbb == 0.0) return 0.0;
  return sab / sqrt(saa * sbb);
}

bool pairs_ok(const int32_t* pairs, int32_t n_pairs, int32_t N) {
  for (int32_t p = 0; p < 2 * n_pairs; ++p)
    if (pairs[p] < 0 || pairs[p] >= N) return false;
  return true;
}

// Distances of the decode patterns P over the pairs.
std::vector<double> pattern_dists(const float* P, int32_t dp, const int32_t* pairs, int32_t n_pairs) {
  std::vector<double> out(n_pairs);
  std::vector<double> a(dp), b(dp);
  for (int32_t p = 0; p < n_pairs; ++p) {
    const float* pa = P + (size_t)pairs[2 * p] * dp;
    const float* pb = P + (size_t)pairs[2 * p + 1] * dp;
    for (int32_t k = 0; k < dp; ++k) {
      a[k] = pa[k];
      b[k] = pb[k];
    }
    out[p] = cos_dist(a.data(), b.data(), dp);
  }
  return out;
}

// Minimum-cost assignment of the n rows to distinct columns of an n x m cost
// (n <= m), by successive shortest augmenting paths with row and column
// potentials (the Hungarian method).  cost(i, j) is evaluated on demand.
// Returns the column of each row.
template <class Cost>
std::vector<int> hungarian(int n, int m, Cost cost) {
  const double inf = std::numeric_limits<double>::infinity();
  std::vector<double> u(n + 1, 0.0), v(m + 1, 0.0), minv(m + 1);
  std::vector<int> match(m + 1, 0), way(m + 1, 0);  // match[j]: row on column j (1-based, 0 = free)
  std::vector<char> used(m + 1);
  for (int i = 1; i <= n; ++i) {
    match[0] = i;
    int j0 = 0;
    std::fill(minv.begin(), minv.end(), inf);
    std::fill(used.begin(), used.end(), 0);
    do {
      used[j0] = 1;
      const int i0 = match[j0];
      double delta = inf;
      int j1 = 0;
      for (int j = 1; j <= m; ++j) {
        if (used[j]) continue;
        const double cur = cost(i0 - 1, j - 1) - u[i0] - v[j];
        if (cur < minv[j]) {
          minv[j] = cur;
          way[j] = j0;
        }
        if (minv[j] < delta) {
          delta = minv[j];
          j1 = j;
        }
      }
      for (int j = 0; j <= m; ++j) {
        if (used[j]) {
          u[match[j]] += delta;
          v[j] -= delta;
        } else {
          minv[j] -= delta;
        }
      }
      j0 = j1;
    } while (match[j0] != 0);
    do {
      const int j1 = way[j0];
      match[j0] = match[j1];
      j0 = j1;
    } while (j0 != 0);
  }
  std::vector<int> col(n, -1);
  for (int j = 1; j <= m; ++j)
    if (match[j] != 0) col[match[j] - 1] = j - 1;
  return col;
}

}  // namespace

extern "C" int eldr_idf(const int32_t* counts, int32_t N, int32_t L, int32_t E, float* idf) {
  if (!counts || !idf || N <= 0 || L <= 0 || E <= 0) return MOE_ERR_INVALID;
  const size_t cells = (size_t)L * E;
  std::vector<int32_t> df(cells, 0);
  for (int32_t r = 0; r < N; ++r)
    for (size_t c = 0; c < cells; ++c) df[c] += counts[(size_t)r * cells + c] > 0 ? 1 : 0;
  for (size_t c = 0; c < cells; ++c) idf[c] = (float)log((N + 1.0) / (df[c] + 1.0));
  return MOE_OK;
}

extern "C" int eldr_signature(const int32_t* counts, const float* idf, int32_t L, int32_t E,
                              const int32_t* layers, int32_t n_layers, float* s) {
  if (!counts || !idf || !s || L <= 0 || E <= 0 || n_layers < 0) return MOE_ERR_INVALID;
  if (n_layers > 0 && !layers) return MOE_ERR_INVALID;
  for (int32_t k = 0; k < n_layers; ++k)
    if (layers[k] < 0 || layers[k] >= L) return MOE_ERR_INVALID;
  std::vector<double> x((size_t)n_layers * E);
  double nn = 0.0;
  for (int32_t k = 0; k < n_layers; ++k)
    for (int32_t e = 0; e < E; ++e) {
      const size_t c = (size_t)layers[k] * E + e;
      const double v = (double)counts[c] * (double)idf[c];
      x[(size_t)k * E + e] = v;
      nn += v * v;
    }
  const double inv = nn > 0.0 ? 1.0 / sqrt(nn) : 0.0;
  for (size_t i = 0; i < x.size(); ++i) s[i] = (float)(x[i] * inv);
  return MOE_OK;
}

extern "C" int eldr_rho(const float* S, int32_t N, int32_t d, const float* P, int32_t dp,
                        const int32_t* pairs, int32_t n_pairs, double* rho) {
  if (!S || !P || !pairs || !rho || N <= 0 || d <= 0 || dp <= 0 || n_pairs < 0)
    return MOE_ERR_INVALID;
  if (!pairs_ok(pairs, n_pairs, N)) return MOE_ERR_INVALID;
  std::vector<double> ds(n_pairs);
  std::vector<double> a(d), b(d);
  for (int32_t p = 0; p < n_pairs; ++p) {
    const float* sa = S + (size_t)pairs[2 * p] * d;
    const float* sb = S + (size_t)pairs[2 * p + 1] * d;
    for (int32_t k = 0; k < d; ++k) {
      a[k] = sa[k];
      b[k] = sb[k];
    }
    ds[p] = cos_dist(a.data(), b.data(), d);
  }
  *rho = spearman(ds, pattern_dists(P, dp, pairs, n_pairs));
  return MOE_OK;
}

extern "C" int eldr_greedy_layers(const int32_t* counts, int32_t N, int32_t L, int32_t E,
                                  const float* idf, const float* P, int32_t dp,
                                  const int32_t* pairs, int32_t n_pairs, int32_t* order,
                                  double* curve, int32_t* n_star) {
  if (!counts || !idf || !P || !pairs || !order || !curve || !n_star || N <= 0 || L <= 0 ||
      E <= 0 || dp <= 0 || n_pairs < 0)
    return MOE_ERR_INVALID;
  if (!pairs_ok(pairs, n_pairs, N)) return MOE_ERR_INVALID;
  // per-layer IDF-weighted counts of each request, their squared norms, and
  // the per-layer dot products of every pair
  const size_t cells = (size_t)L * E;
  std::vector<double> x((size_t)N * cells);
  for (int32_t r = 0; r < N; ++r)
    for (size_t c = 0; c < cells; ++c)
      x[(size_t)r * cells + c] = (double)counts[(size_t)r * cells + c] * (double)idf[c];
  std::vector<double> norm2((size_t)L * N, 0.0), dot((size_t)L * n_pairs, 0.0);
  for (int32_t l = 0; l < L; ++l) {
    for (int32_t r = 0; r < N; ++r) {
      const double* xr = &x[(size_t)r * cells + (size_t)l * E];
      double s = 0.0;
      for (int32_t e = 0; e < E; ++e) s += xr[e] * xr[e];
      norm2[(size_t)l * N + r] = s;
    }
    for (int32_t p = 0; p < n_pairs; ++p) {
      const double* xa = &x[(size_t)pairs[2 * p] * cells + (size_t)l * E];
      const double* xb = &x[(size_t)pairs[2 * p + 1] * cells + (size_t)l * E];
      double s = 0.0;
      for (int32_t e = 0; e < E; ++e) s += xa[e] * xb[e];
      dot[(size_t)l * n_pairs + p] = s;
    }
  }
  const std::vector<double> dpat = pattern_dists(P, dp, pairs, n_pairs);
  std::vector<double> cur_dot(n_pairs, 0.0), cur_norm(N, 0.0), ds(n_pairs);
  std::vector<char> used(L, 0);
  for (int32_t step = 0; step < L; ++step) {
    int best = -1;
    double best_rho = -std::numeric_limits<double>::infinity();
    for (int32_t l = 0; l < L; ++l) {
      if (used[l]) continue;
      for (int32_t p = 0; p < n_pairs; ++p) {
        const double na = cur_norm[pairs[2 * p]] + norm2[(size_t)l * N + pairs[2 * p]];
        const double nb = cur_norm[pairs[2 * p + 1]] + norm2[(size_t)l * N + pairs[2 * p + 1]];
        const double ab = cur_dot[p] + dot[(size_t)l * n_pairs + p];
        ds[p] = (na == 0.0 || nb == 0.0) ? 1.0 : 1.0 - ab / (sqrt(na) * sqrt(nb));
      }
      const double r = spearman(ds, dpat);
      if (r > best_rho) {
        best_rho = r;
        best = l;
      }
    }
    used[best] = 1;
    order[step] = best;
    curve[step] = best_rho;
    for (int32_t p = 0; p < n_pairs; ++p) cur_dot[p] += dot[(size_t)best * n_pairs + p];
    for (int32_t r = 0; r < N; ++r) cur_norm[r] += norm2[(size_t)best * N + r];
  }
  int32_t ns = 1;
  for (int32_t k = 1; k < L; ++k)
    if (curve[k] > curve[ns - 1]) ns = k + 1;
  *n_star = ns;
  return MOE_OK;
}

extern "C" int eldr_balanced_kmeans(const float* S, int32_t N, int32_t d, int32_t K,
                                    const int32_t* init, int32_t max_iters, float* centroids,
                                    int32_t* assign, int32_t* iters) {
  if (!S || !init || !centroids || !assign || !iters || N <= 0 || d <= 0 || K <= 0 || K > N ||
      max_iters <= 0)
    return MOE_ERR_INVALID;
  for (int32_t k = 0; k < K; ++k)
    if (init[k] < 0 || init[k] >= N) return MOE_ERR_INVALID;
  const int cap = (N + K - 1) / K;
  std::vector<double> X((size_t)N * d), C((size_t)K * d), cost((size_t)N * K);
  for (size_t i = 0; i < X.size(); ++i) X[i] = S[i];
  for (int32_t k = 0; k < K; ++k) {
    double nn = 0.0;
    for (int32_t j = 0; j < d; ++j) {
      const double v = X[(size_t)init[k] * d + j];
      C[(size_t)k * d + j] = v;
      nn += v * v;
    }
    const double inv = nn > 0.0 ? 1.0 / sqrt(nn) : 0.0;
    for (int32_t j = 0; j < d; ++j) C[(size_t)k * d + j] *= inv;
  }
  std::vector<int> prev(N, -1), cur(N);
  int it = 0;
  for (it = 1; it <= max_iters; ++it) {
    for (int32_t i = 0; i < N; ++i)
      for (int32_t k = 0; k < K; ++k) {
        double s = 0.0;
        for (int32_t j = 0; j < d; ++j) s += X[(size_t)i * d + j] * C[(size_t)k * d + j];
        cost[(size_t)i * K + k] = 1.0 - s;
      }
    const std::vector<int> col =
        hungarian(N, K * cap, [&](int i, int j) { return cost[(size_t)i * K + j / cap]; });
    for (int32_t i = 0; i < N; ++i) cur[i] = col[i] / cap;
    for (int32_t k = 0; k < K; ++k) {
      std::vector<double> m(d, 0.0);
      int cnt = 0;
      for (int32_t i = 0; i < N; ++i)
        if (cur[i] == k) {
          ++cnt;
          for (int32_t j = 0; j < d; ++j) m[j] += X[(size_t)i * d + j];
        }
      if (cnt == 0) continue;
      double nn = 0.0;
      for (int32_t j = 0; j < d; ++j) {
        m[j] /= cnt;
        nn += m[j] * m[j];
      }
      if (nn == 0.0) continue;
      const double inv = 1.0 / sqrt(nn);
      for (int32_t j = 0; j < d; ++j) C[(size_t)k * d + j] = m[j] * inv;
    }
    const bool same = cur == prev;
    prev = cur;
    if (same) break;
  }
  if (it > max_iters) it = max_iters;
  for (size_t i = 0; i < C.size(); ++i) centroids[i] = (float)C[i];
  for (int32_t i = 0; i < N; ++i) assign[i] = prev[i];
  *iters = it;
  return MOE_OK;
}

namespace {

int route_one(const float* s, int32_t d, const float* centroids, int32_t K, const int32_t* loads,
              float tau) {
  std::vector<double> a(d), c(d), sims(K);
  for (int32_t j = 0; j < d; ++j) a[j] = s[j];
  double top = -std::numeric_limits<double>::infinity();
  for (int32_t k = 0; k < K; ++k) {
    for (int32_t j = 0; j < d; ++j) c[j] = centroids[(size_t)k * d + j];
    sims[k] = 1.0 - cos_dist(a.data(), c.data(), d);
    top = std::max(top, sims[k]);
  }
  int best = -1;
  for (int32_t k = 0; k < K; ++k) {
    if (!(sims[k] >= top - (double)tau)) continue;
    if (best < 0 || loads[k] < loads[best] || (loads[k] == loads[best] && sims[k] > sims[best]))
      best = k;
  }
  return best;
}

}  // namespace

// The band width is a non-negative finite number (the paper sweeps it over
// [0, 1]); a negative or NaN tau could leave the band empty.
static bool valid_tau(float tau) { return std::isfinite(tau) && tau >= 0.0f; }

extern "C" int eldr_route(const float* s, int32_t d, const float* centroids, int32_t K,
                          const int32_t* loads, float tau, int32_t* worker) {
  if (!s || !centroids || !loads || !worker || d <= 0 || K <= 0 || !valid_tau(tau))
    return MOE_ERR_INVALID;
  const int w = route_one(s, d, centroids, K, loads, tau);
  *worker = w;
  // no worker in the band: a similarity was NaN (a non-finite signature or centroid)
  return w < 0 ? MOE_ERR_INVALID : MOE_OK;
}

extern "C" int eldr_route_batch(const float* S, int32_t R, int32_t d, const float* centroids,
                                int32_t K, int32_t* loads, float tau, int32_t* workers) {
  if (!S || !centroids || !loads || !workers || R < 0 || d <= 0 || K <= 0 || !valid_tau(tau))
    return MOE_ERR_INVALID;
  for (int32_t r = 0; r < R; ++r) {
    const int w = route_one(S + (size_t)r * d, d, centroids, K, loads, tau);
    if (w < 0) {
      // stop at the first request that has no worker; it and the rest stay unrouted
      for (int32_t q = r; q < R; ++q) workers[q] = -1;
      return MOE_ERR_INVALID;
    }
    workers[r] = w;
    loads[w] += 1;
  }
  return MOE_OK;
}
