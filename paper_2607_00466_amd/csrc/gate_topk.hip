// moe_gate_topk: fp32 gate scores, top-k selection and renormalised weights.
//
// Two launches on the caller's stream:
//   gate_scores_kernel  logits[T, E] = x[T, H] . w_gate[E, H]^T
//   gate_select_kernel  each token's k best experts by rank, then the
//                       softmax of the k picks.
#include <math.h>

#include "common.hpp"

namespace eldr {

constexpr int kGateWaves = 4;        // the reduction axis H is split over the 4 waves
constexpr int kGateExperts = 4;      // experts per workgroup
constexpr int kGateTokens = 8;       // tokens per workgroup
constexpr int kGateOut = kGateExperts * kGateTokens;  // 32 sums per workgroup

// One step of the halving butterfly over the first 2 * HALF entries of acc:
// a lane keeps the half selected by lane bit M and adds its partner's copy.
template <int HALF, int M>
__device__ __forceinline__ void halving_step(float* acc, int lane) {
  const bool upper = (lane & M) != 0;
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const float mine = upper ? acc[i + HALF] : acc[i];
    const float other = upper ? acc[i] : acc[i + HALF];
    acc[i] = mine + __shfl_xor(other, M);
  }
}

// A workgroup scores 4 experts for 8 tokens.  Wave w covers the w-th quarter
// of H; lane l accumulates, for all 32 (expert, token) pairs, the products at
// float4 positions q = l, l + 64, ... of that quarter, in the same order for
// every expert.  The 64 lane partials are summed by a halving butterfly and
// the 4 wave partials in wave order, so the reduction tree does not depend on
// the expert: experts with identical gate rows get bitwise-identical scores.
__global__ __launch_bounds__(256) void gate_scores_kernel(const float* __restrict__ x,
                                                          const float* __restrict__ wg, int T,
                                                          int H, int E,
                                                          float* __restrict__ logits) {
  __shared__ float part[kGateWaves][kGateOut];
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int e0 = blockIdx.x * kGateExperts;
  const int t0 = blockIdx.y * kGateTokens;
  const int H4 = H / 4;
  const int q_begin = (H4 * wave) / kGateWaves;
  const int q_end = (H4 * (wave + 1)) / kGateWaves;

  const float4* wrow[kGateExperts];
  bool wok[kGateExperts];
#pragma unroll
  for (int a = 0; a < kGateExperts; ++a) {
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

  float acc[kGateOut];
#pragma unroll
  for (int i = 0; i < kGateOut; ++i) acc[i] = 0.0f;

  for (int q = q_begin + lane; q < q_end; q += kWave) {
    float4 w[kGateExperts];
#pragma unroll
    for (int a = 0; a < kGateExperts; ++a)
      w[a] = wok[a] ? wrow[a][q] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < kGateTokens; ++j) {
      const float4 xv = xok[j] ? xrow[j][q] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int a = 0; a < kGateExperts; ++a) {
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
  halving_step<kGateOut / 2, 32>(acc, lane);
  halving_step<kGateOut / 4, 16>(acc, lane);
  halving_step<kGateOut / 8, 8>(acc, lane);
  halving_step<kGateOut / 16, 4>(acc, lane);
  halving_step<kGateOut / 32, 2>(acc, lane);
  const float sum = acc[0] + __shfl_xor(acc[0], 1);
  if ((lane & 1) == 0) part[wave][lane >> 1] = sum;
  __syncthreads();
  if (threadIdx.x < kGateOut) {
    const int o = threadIdx.x;
    const int a = o / kGateTokens;
    const int j = o % kGateTokens;
    const float v = ((part[0][o] + part[1][o]) + part[2][o]) + part[3][o];
    if (e0 + a < E && t0 + j < T) logits[(size_t)(t0 + j) * E + e0 + a] = v;
  }
}

// Selection by rank.  Thread (t, e) counts the experts that precede e in the
// selection order of token t (a larger logit, or an equal logit and a lower
// id); e is selected iff that rank is below K, and the rank is its position
// in topk_ids.  Every comparison is exact, so the result is the oracle's
// order whatever the thread schedule.  Rows are staged in LDS padded with
// -inf to a multiple of 4 (-inf precedes nothing).  The K picks then form
// the softmax over themselves, summed in rank order.
constexpr int kSelectThreads = 256;

__global__ __launch_bounds__(kSelectThreads) void gate_select_kernel(
    const float* __restrict__ logits, int T, int E, int K, int tokens_per_block,
    int32_t* __restrict__ ids, float* __restrict__ wts) {
  extern __shared__ float sl[];                 // [tokens_per_block][Ep] logits, -inf padded
  const int Ep = (E + 3) & ~3;
  float* sel = sl + tokens_per_block * Ep;      // [tokens_per_block][MOE_MAX_K] exp(l - lmax)
  __shared__ float lmax[kSelectThreads];
  const int t0 = blockIdx.x * tokens_per_block;
  const int nt = min(tokens_per_block, T - t0);
  for (int i = threadIdx.x; i < nt * Ep; i += kSelectThreads) {
    const int t = i / Ep;
    const int e = i - t * Ep;
    sl[i] = e < E ? logits[(size_t)(t0 + t) * E + e] : -INFINITY;
  }
  __syncthreads();
  const int p = threadIdx.x;  // one (token, expert) pair per thread
  const bool live = p < nt * E;
  const int t = live ? p / E : 0;
  const int e = p - t * E;
  int rank = K;
  float v = 0.0f;
  if (live) {
    const float4* row = reinterpret_cast<const float4*>(sl + t * Ep);
    v = sl[t * Ep + e];
    int r = 0;
#pragma unroll 8
    for (int f4 = 0; f4 < Ep / 4; ++f4) {
      const float4 u = row[f4];
      const int f = 4 * f4;
      r += (u.x > v || (u.x == v && f + 0 < e)) ? 1 : 0;
      r += (u.y > v || (u.y == v && f + 1 < e)) ? 1 : 0;
      r += (u.z > v || (u.z == v && f + 2 < e)) ? 1 : 0;
      r += (u.w > v || (u.w == v && f + 3 < e)) ? 1 : 0;
    }
    rank = r;
    if (rank == 0) lmax[t] = v;  // rank 0 holds the largest logit
  }
  __syncthreads();
  if (live && rank < K) {
    sel[t * MOE_MAX_K + rank] = expf(v - lmax[t]);
    ids[(size_t)(t0 + t) * K + rank] = e;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nt * K; i += kSelectThreads) {
    const int tt = i / K;
    const int j = i - tt * K;
    float sum = 0.0f;
    for (int q = 0; q < K; ++q) sum += sel[tt * MOE_MAX_K + q];
    wts[(size_t)(t0 + tt) * K + j] = sel[tt * MOE_MAX_K + j] / sum;
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
  dim3 g1((d.E + eldr::kGateExperts - 1) / eldr::kGateExperts,
          (d.T + eldr::kGateTokens - 1) / eldr::kGateTokens);
  hipLaunchKernelGGL(eldr::gate_scores_kernel, g1, dim3(256), 0, s, x, w_gate, d.T, d.H, d.E,
                     logits);
  st = launch_status();
  if (st != MOE_OK) return st;
  // As many tokens per workgroup as give every thread one (token, expert)
  // pair (E <= 256, so at least one token).
  const int tpb = eldr::kSelectThreads / d.E;
  const size_t lds = (size_t)tpb * (((d.E + 3) & ~3) + MOE_MAX_K) * sizeof(float);
  dim3 g2((d.T + tpb - 1) / tpb);
  hipLaunchKernelGGL(eldr::gate_select_kernel, g2, dim3(eldr::kSelectThreads), lds, s, logits, d.T,
                     d.E, d.K, tpb, topk_ids, topk_w);
  return launch_status();
}
