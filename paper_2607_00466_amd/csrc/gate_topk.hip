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
#define ELDR_GATE_WAVES 4
#endif
constexpr int kGateWaves = ELDR_GATE_WAVES;  // the reduction axis H is split over the waves
constexpr int kGateThreads = kGateWaves * 64;

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

// The lane reduction over masks M, M/2, .., 1 of COUNT sums a lane: halving
// steps while a lane holds two or more, then plain exchanges.  Either way the
// sum of each output pairs the lanes by bit 5 first and bit 0 last, and fp32
// addition is commutative, so the tree is the same for every output and every
// tile shape.
template <int COUNT, int M>
__device__ __forceinline__ void lane_reduce(float* acc, int lane) {
  if constexpr (COUNT >= 2) {
    halving_step<COUNT / 2, M>(acc, lane);
  } else {
    acc[0] += __shfl_xor(acc[0], M);
  }
  if constexpr (M > 1) lane_reduce<(COUNT >= 2 ? COUNT / 2 : 1), M / 2>(acc, lane);
}

// A workgroup scores TE experts for TT tokens.  Wave w covers the w-th of
// kGateWaves slices of H; lane l accumulates, for all TT * TE (expert, token)
// pairs, the products at float4 positions q = l, l + 64, ... of that slice,
// in the same order for every pair.  The 64 lane partials are summed by the
// butterfly above and the wave partials in wave order.  So the reduction tree
// of a score depends on H alone: experts with identical gate rows get
// bitwise-identical scores, and a token's scores do not depend on the tile
// shape or on the other tokens of the batch.
template <int TT, int TE>
__global__ __launch_bounds__(kGateThreads) void gate_scores_kernel(const float* __restrict__ x,
                                                          const float* __restrict__ wg, int T,
                                                          int H, int E,
                                                          float* __restrict__ logits) {
  constexpr int kOut = TT * TE;
  static_assert(kOut <= kGateThreads && (kOut & (kOut - 1)) == 0, "a power of two, one thread each");
  __shared__ float part[kGateWaves][kOut];
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int e0 = blockIdx.x * TE;
  const int t0 = blockIdx.y * TT;
  const int H4 = H / 4;
  const int q_begin = (H4 * wave) / kGateWaves;
  const int q_end = (H4 * (wave + 1)) / kGateWaves;

  const float4* wrow[TE];
  bool wok[TE];
#pragma unroll
  for (int a = 0; a < TE; ++a) {
    wok[a] = (e0 + a) < E;
    wrow[a] = reinterpret_cast<const float4*>(wg + (size_t)(wok[a] ? e0 + a : 0) * H);
  }
  const float4* xrow[TT];
  bool xok[TT];
#pragma unroll
  for (int j = 0; j < TT; ++j) {
    xok[j] = (t0 + j) < T;
    xrow[j] = reinterpret_cast<const float4*>(x + (size_t)(xok[j] ? t0 + j : 0) * H);
  }

  float acc[kOut];
#pragma unroll
  for (int i = 0; i < kOut; ++i) acc[i] = 0.0f;

  for (int q = q_begin + lane; q < q_end; q += kWave) {
    float4 w[TE];
#pragma unroll
    for (int a = 0; a < TE; ++a)
      w[a] = wok[a] ? wrow[a][q] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < TT; ++j) {
      const float4 xv = xok[j] ? xrow[j][q] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int a = 0; a < TE; ++a) {
        float s = acc[a * TT + j];
        s = fmaf(w[a].x, xv.x, s);
        s = fmaf(w[a].y, xv.y, s);
        s = fmaf(w[a].z, xv.z, s);
        s = fmaf(w[a].w, xv.w, s);
        acc[a * TT + j] = s;
      }
    }
  }

  // After the lane reduction a lane holds complete sums: outputs
  // l * (kOut / 64) + i for kOut >= 64, else output l / (64 / kOut), which
  // the 64 / kOut lanes of a group hold alike.
  lane_reduce<kOut, 32>(acc, lane);
  if constexpr (kOut >= kWave) {
#pragma unroll
    for (int i = 0; i < kOut / kWave; ++i) part[wave][lane * (kOut / kWave) + i] = acc[i];
  } else {
    if (lane % (kWave / kOut) == 0) part[wave][lane / (kWave / kOut)] = acc[0];
  }
  __syncthreads();
  if (threadIdx.x < kOut) {
    const int o = threadIdx.x;
    const int a = o / TT;
    const int j = o % TT;
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
  // Tiles of 4 tokens x 4 experts up to 128 tokens: the most workgroups for a
  // reduction that is one or two loads a lane long.  Above that 8 x 8: half
  // the L2 reads of x and of the gate rows per product (measured on MI355X at
  // H = 2880: 11.1 -> 8.2 us at T = 256 against 8 x 4 tiles on 8 waves, and
  // 3.9 us at T = 64 against 4.1).  The scores are the same bits either way.
  if (d.T <= 128) {
    dim3 g1((d.E + 3) / 4, (d.T + 3) / 4);
    hipLaunchKernelGGL((eldr::gate_scores_kernel<4, 4>), g1, dim3(eldr::kGateThreads), 0, s, x, w_gate,
                       d.T, d.H, d.E, logits);
  } else {
    dim3 g1((d.E + 7) / 8, (d.T + 7) / 8);
    hipLaunchKernelGGL((eldr::gate_scores_kernel<8, 8>), g1, dim3(eldr::kGateThreads), 0, s, x, w_gate,
                       d.T, d.H, d.E, logits);
  }
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
