// moe_gate_topk: fp32 gate scores, top-k selection and renormalised weights.
//
// Two launches on the caller's stream:
//   gate_scores_kernel  logits[T, E] = x[T, H] . w_gate[E, H]^T
//   gate_select_kernel  each token's k best experts by rank, then the
//                       softmax of the k picks.
#include <math.h>

#include "common.hpp"

namespace eldr {

#ifndef ELDR_GATE_WAVES
#define ELDR_GATE_WAVES 8
#endif
constexpr int kGateWaves = ELDR_GATE_WAVES;  // the reduction axis H is split over the waves
constexpr int kGateThreads = kGateWaves * 64;
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

// A workgroup scores 4 experts for 8 tokens.  Wave w covers the w-th of
// kGateWaves slices of H; lane l accumulates, for all 32 (expert, token)
// pairs, the products at float4 positions q = l, l + 64, ... of that slice,
// in the same order for every expert.  The 64 lane partials are summed by a
// halving butterfly and the wave partials in wave order, so the reduction
// tree does not depend on the expert: experts with identical gate rows get
// bitwise-identical scores.  With 8 waves a lane takes one float4 of each
// row at H = 2048, so the loads cost a single memory round trip.
__global__ __launch_bounds__(kGateThreads) void gate_scores_kernel(const float* __restrict__ x,
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
    float v = part[0][o];
#pragma unroll
    for (int w = 1; w < kGateWaves; ++w) v += part[w][o];
    if (e0 + a < E && t0 + j < T) logits[(size_t)(t0 + j) * E + e0 + a] = v;
  }
}

// Selection by rank.  Thread (t, e) counts the experts that precede e in the
// selection order of token t (a larger logit, or an equal logit and a lower
// id); e is selected iff that rank is below K, and the rank is its position
// in topk_ids.  The order is folded into one 64-bit key per expert -- the
// logit's bits mapped to an unsigned integer of the same order (with -0 taken
// as +0, so equal logits get equal high words), then the complement of the
// id -- so that "precedes" is a single unsigned comparison of keys, and keys
// are distinct.  Every comparison is exact, so the result is the oracle's
// order whatever the thread schedule.  Rows of keys are staged in LDS, padded
// with 0 (below every key) to an even length.  The K picks then form the
// softmax over themselves, summed in rank order.
constexpr int kSelectThreads = 256;

__device__ __forceinline__ uint64_t select_key(float v, int e) {
  uint32_t b = __float_as_uint(v + 0.0f);  // -0 -> +0
  b = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)b << 32) | (uint32_t)~(uint32_t)e;
}

typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));

__global__ __launch_bounds__(kSelectThreads) void gate_select_kernel(
    const float* __restrict__ logits, int T, int E, int K, int tokens_per_block,
    int32_t* __restrict__ ids, float* __restrict__ wts) {
  extern __shared__ uint64_t skey[];            // [tokens_per_block][Ep] keys, 0 padded
  const int Ep = (E + 1) & ~1;
  float* sel = reinterpret_cast<float*>(skey + tokens_per_block * Ep);  // [tpb][MOE_MAX_K] exp
  __shared__ float lmax[kSelectThreads];
  const int t0 = blockIdx.x * tokens_per_block;
  const int nt = min(tokens_per_block, T - t0);
  const int p = threadIdx.x;  // one (token, expert) pair per thread
  const bool live = p < nt * E;
  const int t = live ? p / E : 0;
  const int e = p - t * E;
  const float v = live ? logits[(size_t)(t0 + t) * E + e] : 0.0f;
  const uint64_t mine = select_key(v, e);
  if (live) skey[t * Ep + e] = mine;
  if (p < nt && (E & 1)) skey[p * Ep + E] = 0;
  __syncthreads();
  int rank = K;
  if (live) {
    const u64x2* row = reinterpret_cast<const u64x2*>(skey + t * Ep);
    int r0 = 0, r1 = 0;
#pragma unroll 8
    for (int f2 = 0; f2 < Ep / 2; ++f2) {
      const u64x2 k = row[f2];
      r0 += k.x > mine ? 1 : 0;
      r1 += k.y > mine ? 1 : 0;
    }
    rank = r0 + r1;
    if (rank == 0) lmax[t] = v;  // rank 0 holds the largest logit
  }
  __syncthreads();
  if (live && rank < K) {
    sel[t * MOE_MAX_K + rank] = expf(v - lmax[t]);
    ids[(size_t)(t0 + t) * K + rank] = e;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nt * K; i += blockDim.x) {
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
  hipLaunchKernelGGL(eldr::gate_scores_kernel, g1, dim3(eldr::kGateThreads), 0, s, x, w_gate, d.T, d.H, d.E,
                     logits);
  st = launch_status();
  if (st != MOE_OK) return st;
  // One token per workgroup, one (token, expert) pair per thread, E rounded
  // up to whole waves (E <= 256 = kSelectThreads): decode batches then spread
  // the rank loops' LDS reads over T CUs.  Measured about 2% shorter than
  // packing 256 / E tokens into 256 threads.
  const int tpb = 1;
  const int sel_threads = (d.E + eldr::kWave - 1) / eldr::kWave * eldr::kWave;
  const size_t lds = (size_t)tpb * (((d.E + 1) & ~1) * sizeof(uint64_t) + MOE_MAX_K * sizeof(float));
  dim3 g2((d.T + tpb - 1) / tpb);
  hipLaunchKernelGGL(eldr::gate_select_kernel, g2, dim3(sel_threads), lds, s, logits, d.T,
                     d.E, d.K, tpb, topk_ids, topk_w);
  return launch_status();
}
