// moe_expert_ffn: SwiGLU FFN of every expert in the distinct-expert union.
//
// Cost model (Motivation, "Active Expert Count Drives MoE Decode Latency"):
// a decode step must fetch the weights of every expert its batch activates;
// each expert has only a few tokens, so the work is a skinny product that is
// bound by HBM bandwidth.  The design follows from that:
//
// * Two launches.  "up" computes h = silu(W1 x) * (W3 x) for every slot into
//   the workspace (as bf16 pairs, see below); "down" computes y = W2 h.
//   Within each launch a workgroup owns one expert and a band of output rows
//   and streams that band's bf16 weights from HBM exactly once (128-bit loads
//   straight into the MFMA A operand), for all of the expert's tokens at once.
//   Weights come packed by moe_pack_weights, so each load instruction reads
//   one contiguous 1 KB MFMA fragment.
// * The expert's tokens (at most 64 per pass) are gathered, carried as a pair
//   of bf16 values (high part + rounded remainder) and staged in LDS in
//   k-chunks, double-buffered, shared by the workgroup's four waves; each
//   wave reads them as the MFMA B operand.  Tokens are padded to a multiple
//   of 16 only in registers (lanes past the bucket repeat its last token and
//   their output columns are not stored).
// * Each wave keeps a ring of weight fragments for the next k-steps in
//   flight; a refill is issued right after the MFMAs that consumed its slot.
// * The grid is sized for E experts; a workgroup reads the union size on the
//   device and returns at once if its slot is past it, so inactive experts
//   cost one scalar load and no host synchronisation is needed.
// * Workgroups of one expert are placed on one XCD (the dispatcher deals
//   workgroups round-robin over the 8 XCDs), so the expert's activations are
//   read into a single L2.
#include "common.hpp"

namespace eldr {

#ifndef ELDR_FFN_RING_SMALL
#define ELDR_FFN_RING_SMALL 4
#endif
#ifndef ELDR_FFN_RING_LARGE
#define ELDR_FFN_RING_LARGE 4
#endif

constexpr int kFfnThreads = 256;  // 4 waves
constexpr int kFfnWaves = kFfnThreads / kWave;
constexpr int kKStep = 32;        // k per MFMA
constexpr int kFragElems = 512;   // bf16 values in one packed 16 x 32 weight fragment (1 KB)
constexpr int kMaxTiles = 4;      // token tiles of 16 per pass: at most 64 tokens per pass

// k-steps of weights in flight per wave (the prefetch depth of the ring).
template <int NT>
__host__ __device__ constexpr int ring_depth() {
  return NT <= 2 ? ELDR_FFN_RING_SMALL : ELDR_FFN_RING_LARGE;
}

// Bytes of one LDS staging buffer (two are used, double-buffered): at least
// a base size, and always room for a chunk of ring_depth k-steps of the
// largest pass (NT * 16 tokens, 128 bytes per k-step, 16 bytes of padding).
template <int NT>
__host__ __device__ constexpr int lds_buf_bytes() {
  constexpr int base = NT == 1 ? 16 * 1024 : NT == 2 ? 24 * 1024 : 34 * 1024;
  constexpr int need = NT * 16 * (128 * ring_depth<NT>() + 16);
  return base > need ? base : ((need + 1023) / 1024) * 1024;
}

enum FfnMode { kUp = 0, kDown = 1 };

struct FfnArgs {
  const uint4* src;            // up: x [T, H] fp32; down: h [T*K, I] as bf16 pairs
  const uint16_t* wa;          // up: W1 [E, I, H]; down: W2 [E, H, I]
  const uint16_t* wb;          // up: W3 [E, I, H]; down: unused
  const int32_t* offsets;      // [E+1]
  const int32_t* perm_token;   // [T*K]
  const int32_t* union_ids;    // [E]
  const int32_t* union_size;   // [1]
  void* dst;                   // up: h [T*K, I] as bf16 pairs; down: y_perm [T*K, H] fp32
  int rows;                    // output rows per expert: up I, down H
  int kdim;                    // reduction length: up H, down I
  int tiles;                   // workgroups per expert
};

// Rows per workgroup: up -> 4 waves x 16 rows (each wave reads the same 16
// rows of W1 and of W3); down -> 4 waves x 32 rows of W2 (two 16-row tiles).
template <int MODE>
__host__ __device__ constexpr int rows_per_block() {
  return MODE == kUp ? kFfnWaves * 16 : kFfnWaves * 32;
}

// LDS layout of one staged chunk: per token a row of kcs k-steps; each
// k-step holds 4 groups of 8 k-values; each group is 8 bf16 high parts then
// 8 bf16 low parts (32 bytes).  Row stride = 128 * kcs + 16 bytes, an odd
// multiple of 16, so the 16 lanes that read 16 tokens hit distinct banks.
__device__ __forceinline__ int lds_stride(int kcs) { return 128 * kcs + 16; }

template <int N>
struct Int {
  static constexpr int value = N;
};

// Calls f(Int<0>{}), ..., f(Int<N-1>{}) -- a loop whose index is a constant.
template <int N, typename F, int I = 0>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(Int<I>{});
    static_for<N, F, I + 1>(static_cast<F&&>(f));
  }
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Split two fp32 values into bf16 high parts and rounded remainders with the
// packed round-to-nearest-even convert: hi = rne(v), lo = rne(v - hi).
__device__ __forceinline__ void split2(uint32_t a, uint32_t b, uint32_t& hi, uint32_t& lo) {
  const f32x2 v = {__uint_as_float(a), __uint_as_float(b)};
  const bf16x2 h = __builtin_convertvector(v, bf16x2);
  const f32x2 r = v - __builtin_convertvector(h, f32x2);
  hi = __builtin_bit_cast(uint32_t, h);
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
}

// 8 fp32 values (as raw bits) -> 8 bf16 high parts and 8 bf16 low parts.
__device__ __forceinline__ void split8_pk(const u32x4& a, const u32x4& b, u32x4& hi, u32x4& lo) {
  uint32_t h0, h1, h2, h3, l0, l1, l2, l3;
  split2(a.x, a.y, h0, l0);
  split2(a.z, a.w, h1, l1);
  split2(b.x, b.y, h2, l2);
  split2(b.z, b.w, h3, l3);
  hi = u32x4{h0, h1, h2, h3};
  lo = u32x4{l0, l1, l2, l3};
}

// Activations enter the MFMA B operand as a pair of bf16 numbers (high
// part, rounded remainder).  In LDS, and for h in the workspace, a row of K
// values is K / 8 groups of 32 bytes: 8 bf16 high parts, then the 8 matching
// low parts -- the same 4 bytes per value as fp32.  The up kernel stages x
// from fp32 and splits it on the way into LDS; its epilogue writes h already
// split, so the down kernel stages h with a plain copy.

template <int MODE, int NT>
__global__ __launch_bounds__(kFfnThreads) void ffn_kernel(FfnArgs a) {
  constexpr int kBuf = lds_buf_bytes<NT>();
  constexpr int kRing = ring_depth<NT>();
  static_assert(kBuf >= NT * 16 * (128 * kRing + 16), "a chunk of kRing k-steps must fit");
  constexpr int kGroups = (kBuf / 32 + kFfnThreads - 1) / kFfnThreads;  // staged groups per thread
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][kBuf];
  __shared__ int tok[NT * 16];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;

  // ---- which (expert, row band) this workgroup owns -----------------------
  const int bid = blockIdx.x;
  const int xcd = bid % kNumXcd;
  const int slot = bid / kNumXcd;
  const int u = (slot / a.tiles) * kNumXcd + xcd;
  const int tile = slot % a.tiles;
  const int U = *a.union_size;
  if (u >= U) return;  // also covers U < 0 (invalid routing)
  const int e = a.union_ids[u];
  const int s_begin = a.offsets[e];
  const int c_total = a.offsets[e + 1] - s_begin;
  if (c_total <= 0) return;

  const int K = a.kdim;
  const int nk = K / kKStep;
  const int r0 = tile * rows_per_block<MODE>() + wave * (MODE == kUp ? 16 : 32);
  const bool ok0 = r0 < a.rows;
  const bool ok1 = MODE == kUp ? ok0 : (r0 + 16 < a.rows);
  // A 16-row tile past the end of the matrix (only when rows is not a
  // multiple of the band) re-reads the band's first tile and is not stored.
  const int ra0 = ok0 ? r0 : tile * rows_per_block<MODE>();
  const int ra1 = MODE == kUp ? ra0 : (ok1 ? r0 + 16 : tile * rows_per_block<MODE>());

  // A operand: lane holds row (lane % 16) of its 16-row tile, k-group
  // (lane / 16).  Weights are packed (moe_pack_weights): the 64 lane pieces of
  // one tile and k-step are a contiguous 1 KB fragment, and a tile's k-steps
  // follow each other, so step s of a tile is at tile_base + s * 512 values.
  const int arow = lane & 15;
  const int kgrp = lane >> 4;
  const size_t tiles_per_expert = (size_t)(a.rows / 16);
  const uint16_t* pa0 =
      a.wa + ((e * tiles_per_expert + ra0 / 16) * nk) * kFragElems + lane * 8;
  const uint16_t* pa1 = (MODE == kUp ? a.wb : a.wa) +
                        ((e * tiles_per_expert + ra1 / 16) * nk) * kFragElems + lane * 8;

  // Weight ring: slot i holds the fragments of the k-step congruent to i
  // mod kRing.  Loads past the last k-step re-read the last one (always
  // issued, never used), which keeps the loop free of branches.
  u32x4 ring0[kRing], ring1[kRing];
  auto ring_prologue = [&]() {
#pragma unroll
    for (int i = 0; i < kRing; ++i) {
      const int si = min(i, nk - 1);
      ring0[i] = *reinterpret_cast<const u32x4*>(pa0 + (size_t)si * kFragElems);
      ring1[i] = *reinterpret_cast<const u32x4*>(pa1 + (size_t)si * kFragElems);
    }
  };

  for (int p0 = 0; p0 < c_total; p0 += NT * 16) {
    const int c = min(NT * 16, c_total - p0);
    const int nt = (c + 15) / 16;
    // k-steps per staged chunk: a multiple of kRing that fits c token rows.
    const int kcs = max(kRing, (((kBuf / c - 16) / 128) / kRing) * kRing);
    const int stride = lds_stride(kcs);

    __syncthreads();  // the previous pass has finished with LDS
    if (tid < c) tok[tid] = (MODE == kUp) ? a.perm_token[s_begin + p0 + tid] : s_begin + p0 + tid;
    __syncthreads();

    // Fetch this thread's share of chunk [ks, ks + klen) k-steps into
    // registers.  Every thread issues the same loads (a thread with no group
    // left re-reads group 0), so the number of loads in flight is the same on
    // every path and the compiler never has to drain the weight ring.
    const size_t row_groups = (size_t)K / 8;  // 32-byte groups per activation row
    u32x4 stg[kGroups][2];
    auto fetch = [&](int ks, int klen) {
      const int gpr = 4 * klen;
      const int ng = c * gpr;
#pragma unroll
      for (int j = 0; j < kGroups; ++j) {
        int q = tid + kFfnThreads * j;
        q = q < ng ? q : 0;
        const int n = q / gpr;
        const int gi = q - n * gpr;
        const u32x4* p =
            reinterpret_cast<const u32x4*>(a.src) + 2 * ((size_t)tok[n] * row_groups + ks * 4 + gi);
        stg[j][0] = p[0];
        stg[j][1] = p[1];
      }
    };
    auto publish = [&](int buf, int klen) {
      const int gpr = 4 * klen;
      const int ng = c * gpr;
#pragma unroll
      for (int j = 0; j < kGroups; ++j) {
        const int q = tid + kFfnThreads * j;
        if (q < ng) {
          const int n = q / gpr;
          const int gi = q - n * gpr;
          u32x4* d = reinterpret_cast<u32x4*>(&lds[buf][n * stride + gi * 32]);
          if (MODE == kUp) {
            u32x4 hi, lo;
            split8_pk(stg[j][0], stg[j][1], hi, lo);
            d[0] = hi;
            d[1] = lo;
          } else {
            d[0] = stg[j][0];
            d[1] = stg[j][1];
          }
        }
      }
    };

    f32x4 acc0[NT], acc1[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      acc0[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      acc1[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    ring_prologue();

    // One k-step: multiply ring slot I against the staged tokens of
    // chunk-relative step s - ks, then refill the slot with step s + kRing.
    // The refill is issued after the MFMAs that read the slot, into the same
    // registers, and a scheduling barrier keeps it there, so each slot stays
    // in place and kRing steps of loads are always in flight.
    auto kstep = [&](auto I, int s, const unsigned char* bb, int ks) {
      constexpr int i = decltype(I)::value;
      const unsigned char* bs = bb + (s - ks) * 128;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t < nt) {
          // Column n of the product depends only on column n of B, so lanes
          // past the bucket read its last token and their columns are
          // simply not stored.
          const int n = min(t * 16 + arow, c - 1);
          const u32x4* bp = reinterpret_cast<const u32x4*>(bs + n * stride);
          const u32x4 bh = bp[0];
          const u32x4 bl = bp[1];
          acc0[t] = mfma16x16x32(ring0[i], bh, acc0[t]);
          acc0[t] = mfma16x16x32(ring0[i], bl, acc0[t]);
          acc1[t] = mfma16x16x32(ring1[i], bh, acc1[t]);
          acc1[t] = mfma16x16x32(ring1[i], bl, acc1[t]);
        }
      }
      const int sn = min(s + kRing, nk - 1);
      ring0[i] = *reinterpret_cast<const u32x4*>(pa0 + (size_t)sn * kFragElems);
      ring1[i] = *reinterpret_cast<const u32x4*>(pa1 + (size_t)sn * kFragElems);
      __builtin_amdgcn_sched_barrier(0);
    };

    fetch(0, min(kcs, nk));
    for (int ks = 0, chunk = 0; ks < nk; ks += kcs, ++chunk) {
      const int ke = min(nk, ks + kcs);
      const int buf = chunk & 1;
      // Buffer `buf` was last read two chunks ago; every wave has passed the
      // barrier of the previous chunk since, so it is free to overwrite.
      publish(buf, ke - ks);
      __syncthreads();
      if (ke < nk) fetch(ke, min(kcs, nk - ke));

      const unsigned char* bb = &lds[buf][kgrp * 32];
      // ks is a multiple of kRing, so slot i always holds step sb + i.
      const int kfull = ks + ((ke - ks) / kRing) * kRing;
      for (int sb = ks; sb < kfull; sb += kRing) {
        static_for<kRing>([&](auto I) { kstep(I, sb + decltype(I)::value, bb, ks); });
      }
      // Tail (only in the last chunk, when nk is not a multiple of kRing).
      if (kfull < ke) {
        static_for<kRing>([&](auto I) {
          if (kfull + decltype(I)::value < ke) kstep(I, kfull + decltype(I)::value, bb, ks);
        });
      }
    }

    // ---- epilogue: lane holds rows r0 + 4 * (lane / 16) + i of token lane % 16
    const int rsub = 4 * kgrp;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int n = t * 16 + arow;
      if (t < nt && n < c) {
        const size_t sl = (size_t)(s_begin + p0 + n);
        if (MODE == kUp) {
          if (ok0) {
            // h for rows r0 + rsub .. + 3: half of one 8-value group of the
            // split layout (high parts at +0, low parts at +16 bytes).
            uint32_t hi[4], lo[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) split_bf16(silu(acc0[t][i]) * acc1[t][i], hi[i], lo[i]);
            const int col = r0 + rsub;
            unsigned char* row = static_cast<unsigned char*>(a.dst) + sl * (size_t)a.rows * 4;
            unsigned char* grp = row + (col / 8) * 32 + (col % 8) * 2;
            *reinterpret_cast<uint2*>(grp) = make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16));
            *reinterpret_cast<uint2*>(grp + 16) = make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16));
          }
        } else {
          float* y = static_cast<float*>(a.dst) + sl * a.rows;
          if (ok0)
            *reinterpret_cast<float4*>(y + r0 + rsub) =
                make_float4(acc0[t][0], acc0[t][1], acc0[t][2], acc0[t][3]);
          if (ok1)
            *reinterpret_cast<float4*>(y + r0 + 16 + rsub) =
                make_float4(acc1[t][0], acc1[t][1], acc1[t][2], acc1[t][3]);
        }
      }
    }
  }
}

template <int MODE, int NT>
static void launch_ffn(const FfnArgs& a, int E, hipStream_t s) {
  const int groups = (E + kNumXcd - 1) / kNumXcd;
  const dim3 grid(kNumXcd * a.tiles * groups);
  hipLaunchKernelGGL((ffn_kernel<MODE, NT>), grid, dim3(kFfnThreads), 0, s, a);
}

// Token tiles held per pass: enough for every bucket when T is small (a
// bucket never exceeds T tokens), at most kMaxTiles.
template <int MODE>
static void launch_ffn_nt(const FfnArgs& a, int T, int E, hipStream_t s) {
#ifdef ELDR_FFN_FORCE_NT
  T = 16 * ELDR_FFN_FORCE_NT;
#endif
  if (T <= 16)
    launch_ffn<MODE, 1>(a, E, s);
  else if (T <= 32)
    launch_ffn<MODE, 2>(a, E, s);
  else
    launch_ffn<MODE, kMaxTiles>(a, E, s);
}

}  // namespace eldr

// Workspace: h of every slot as bf16 pairs (4 bytes a value).
extern "C" size_t moe_ffn_workspace_bytes(moe_dims d) {
  if (eldr_host::check_dims(d) != MOE_OK) return 0;
  return (size_t)d.T * d.K * d.I * 4;
}

namespace {

int check_ffn_common(const moe_dims& d, const int32_t* offsets, const int32_t* perm_token,
                     const int32_t* union_ids, const int32_t* union_size) {
  using namespace eldr_host;
  if (!offsets || !perm_token || !union_ids || !union_size) return MOE_ERR_INVALID;
  if (!aligned4(offsets) || !aligned4(perm_token) || !aligned4(union_ids) || !aligned4(union_size))
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

}  // namespace

extern "C" int moe_expert_ffn_up(const float* x, const uint16_t* w1, const uint16_t* w3,
                                 const int32_t* offsets, const int32_t* perm_token,
                                 const int32_t* union_ids, const int32_t* union_size, moe_dims d,
                                 void* ws, size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !w1 || !w3 || !ws) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(w1) || !aligned16(w3) || !aligned16(ws)) return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  eldr::FfnArgs up{reinterpret_cast<const uint4*>(x), w1, w3, offsets, perm_token, union_ids,
                   union_size, ws, d.I, d.H, 0};
  up.tiles = (d.I + eldr::rows_per_block<eldr::kUp>() - 1) / eldr::rows_per_block<eldr::kUp>();
  eldr::launch_ffn_nt<eldr::kUp>(up, d.T, d.E, s);
  return launch_status();
}

extern "C" int moe_expert_ffn_down(const void* ws, const uint16_t* w2, const int32_t* offsets,
                                   const int32_t* perm_token, const int32_t* union_ids,
                                   const int32_t* union_size, moe_dims d, size_t ws_bytes,
                                   float* y_perm, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!ws || !w2 || !y_perm) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(ws) || !aligned16(w2) || !aligned16(y_perm)) return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs down{reinterpret_cast<const uint4*>(ws), w2, nullptr, offsets, perm_token,
                     union_ids, union_size, y_perm, d.H, d.I, 0};
  down.tiles =
      (d.H + eldr::rows_per_block<eldr::kDown>() - 1) / eldr::rows_per_block<eldr::kDown>();
  eldr::launch_ffn_nt<eldr::kDown>(down, d.T, d.E, reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}

extern "C" int moe_expert_ffn(const float* x, const uint16_t* w1, const uint16_t* w3,
                              const uint16_t* w2, const int32_t* offsets,
                              const int32_t* perm_token, const int32_t* union_ids,
                              const int32_t* union_size, moe_dims d, float* y_perm, void* ws,
                              size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !w1 || !w3 || !w2 || !y_perm || !ws) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(w1) || !aligned16(w3) || !aligned16(w2) || !aligned16(y_perm) ||
      !aligned16(ws))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  float* h = static_cast<float*>(ws);
  st = moe_expert_ffn_up(x, w1, w3, offsets, perm_token, union_ids, union_size, d, h, ws_bytes,
                         stream);
  if (st != MOE_OK) return st;
  return moe_expert_ffn_down(h, w2, offsets, perm_token, union_ids, union_size, d, ws_bytes,
                             y_perm, stream);
}
