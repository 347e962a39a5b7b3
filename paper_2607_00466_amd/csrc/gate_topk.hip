// moe_gate_topk: fp32 gate scores, top-k selection and renormalised weights.
//
// Two launches on the caller's stream:
//   gate_scores_kernel  logits[T, E] = x[T, H] . w_gate[E, H]^T
//   gate_select_kernel  one wavefront per token: k rounds of a wave-wide
//                       arg-max (larger logit, then lower id), then the
//                       softmax of the k picks.
#include <math.h>

#include "common.hpp"

namespace eldr {

constexpr int kGateExpertsPerWave = 4;
constexpr int kGateTokens = 8;
constexpr int kGateWaves = 4;
constexpr int kGateExpertsPerBlock = kGateExpertsPerWave * kGateWaves;  // 16
constexpr int kGateOut = kGateExpertsPerWave * kGateTokens;             // 32 sums per wave

// Each wave scores 4 experts for 8 tokens.  Lane l accumulates, for all 32
// (expert, token) pairs, the products at h = 4 * (l + 64 * i) .. + 3, in the
// same order for every expert; the 64 lane partials are then summed by a
// halving butterfly whose tree does not depend on the expert.  So every
// expert's score is the same function of (x, its gate row): experts with
// identical rows get bitwise-identical scores.
__global__ __launch_bounds__(256) void gate_scores_kernel(const float* __restrict__ x,
                                                          const float* __restrict__ wg, int T,
                                                          int H, int E,
                                                          float* __restrict__ logits) {
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int e0 = blockIdx.x * kGateExpertsPerBlock + wave * kGateExpertsPerWave;
  const int t0 = blockIdx.y * kGateTokens;
  const int H4 = H / 4;

  float acc[kGateOut];
#pragma unroll
  for (int i = 0; i < kGateOut; ++i) acc[i] = 0.0f;

  const float4* wrow[kGateExpertsPerWave];
  bool wok[kGateExpertsPerWave];
#pragma unroll
  for (int a = 0; a < kGateExpertsPerWave; ++a) {
    wok[a] = (e0 + a) < E;
    wrow[a] = reinterpret_cast<const float4*>(wg + (size_t)(wok[a] ? e0 + a : 0) * H);
  }
  const float4* xrow[kGateTokens];
  bool xok[kGateTokens];
#pragma unroll
  for (int j = 0; j < kGateTokens; ++j) {
    xok[j] = (t0 + j) < T;
    xrow[j] = reinterpret_cast<const float4*>(x + (size_t)(xok[j] ? t0 + j : 0) * H);
  }

  for (int h4 = lane; h4 < H4; h4 += kWave) {
    float4 w[kGateExpertsPerWave];
#pragma unroll
    for (int a = 0; a < kGateExpertsPerWave; ++a)
      w[a] = wok[a] ? wrow[a][h4] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < kGateTokens; ++j) {
      const float4 xv = xok[j] ? xrow[j][h4] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int a = 0; a < kGateExpertsPerWave; ++a) {
        float s = acc[a * kGateTokens + j];
        s = fmaf(w[a].x, xv.x, s);
        s = fmaf(w[a].y, xv.y, s);
        s = fmaf(w[a].z, xv.z, s);
        s = fmaf(w[a].w, xv.w, s);
        acc[a * kGateTokens + j] = s;
      }
    }
  }

  // Halving butterfly: at each step a lane keeps the half of its sums chosen
  // by one lane bit and adds its partner's copy of that half.  After the
  // masks 32, 16, 8, 4, 2 every lane holds one sum, for output index
  // (lane >> 1) & 31, over all lanes except its bit-0 partner; a final xor-1
  // exchange completes it.  fp32 addition is commutative, so the partner
  // order does not matter; the tree is the same for every output.
#pragma unroll
  for (int step = 0; step < 5; ++step) {
    const int m = 32 >> step;
    const int half = kGateOut >> (step + 1);
    const bool upper = (lane & m) != 0;
#pragma unroll
    for (int i = 0; i < half; ++i) {
      const float mine = upper ? acc[i + half] : acc[i];
      const float other = upper ? acc[i] : acc[i + half];
      acc[i] = mine + __shfl_xor(other, m);
    }
  }
  const float sum = acc[0] + __shfl_xor(acc[0], 1);
  if ((lane & 1) == 0) {
    const int o = lane >> 1;
    const int a = o / kGateTokens;
    const int j = o % kGateTokens;
    if (e0 + a < E && t0 + j < T) logits[(size_t)(t0 + j) * E + e0 + a] = sum;
  }
}

// (value, id) order of the selection: larger value first, then lower id.
// id < 0 means "no candidate".
__device__ __forceinline__ bool better(float v, int e, float bv, int be) {
  if (e < 0) return false;
  if (be < 0) return true;
  return v > bv || (v == bv && e < be);
}

__global__ __launch_bounds__(256) void gate_select_kernel(const float* __restrict__ logits, int T,
                                                          int E, int K, int32_t* __restrict__ ids,
                                                          float* __restrict__ wts) {
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int t = blockIdx.x * (blockDim.x / kWave) + wave;
  if (t >= T) return;
  constexpr int kPer = MOE_MAX_E / kWave;  // 4 candidates per lane
  float v[kPer];
  bool live[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = lane + kWave * i;
    live[i] = e < E;
    v[i] = live[i] ? logits[(size_t)t * E + e] : 0.0f;
  }
  int my_id = -1;
  float my_l = 0.0f;
  for (int j = 0; j < K; ++j) {
    float bv = 0.0f;
    int be = -1;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int e = lane + kWave * i;
      if (live[i] && better(v[i], e, bv, be)) {
        bv = v[i];
        be = e;
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ov = __shfl_xor(bv, m);
      const int oe = __shfl_xor(be, m);
      if (better(ov, oe, bv, be)) {
        bv = ov;
        be = oe;
      }
    }
    // every lane now holds the same winner
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (lane + kWave * i == be) live[i] = false;
    if (lane == j) {
      my_id = be;
      my_l = bv;
    }
  }
  const float lmax = __shfl(my_l, 0);
  const float ex = lane < K ? expf(my_l - lmax) : 0.0f;
  float s = ex;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m);
  if (lane < K) {
    ids[(size_t)t * K + lane] = my_id;
    wts[(size_t)t * K + lane] = ex / s;
  }
}

}  // namespace eldr

extern "C" int moe_gate_topk(const float* x, const float* w_gate, moe_dims d, float* logits,
                             int32_t* topk_ids, float* topk_w, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !w_gate || !logits || !topk_ids || !topk_w) return MOE_ERR_INVALID;
  if (!aligned16(x) || !aligned16(w_gate) || !aligned4(logits) || !aligned4(topk_ids) ||
      !aligned4(topk_w))
    return MOE_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  dim3 g1((d.E + eldr::kGateExpertsPerBlock - 1) / eldr::kGateExpertsPerBlock,
          (d.T + eldr::kGateTokens - 1) / eldr::kGateTokens);
  hipLaunchKernelGGL(eldr::gate_scores_kernel, g1, dim3(256), 0, s, x, w_gate, d.T, d.H, d.E,
                     logits);
  st = launch_status();
  if (st != MOE_OK) return st;
  dim3 g2((d.T + 3) / 4);
  hipLaunchKernelGGL(eldr::gate_select_kernel, g2, dim3(256), 0, s, logits, d.T, d.E, d.K,
                     topk_ids, topk_w);
  return launch_status();
}
