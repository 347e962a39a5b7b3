// moe_expert_ffn: SwiGLU FFN of every expert in the distinct-expert union.
//
// Cost model (Motivation, "Active Expert Count Drives MoE Decode Latency"):
// a decode step must fetch the weights of every expert its batch activates;
// each expert has only a few tokens, so the work is a skinny product that is
// bound by HBM bandwidth.  The design follows from that:
//
// * Two launches.  "up" computes h = silu(W1 x) * (W3 x) for every slot into
//   a small fp32 workspace; "down" computes y = W2 h.  Within each launch a
//   workgroup owns one expert and a band of output rows, and streams that
//   band's bf16 weights from HBM exactly once (128-bit loads straight into
//   the MFMA A operand), for all of the expert's tokens at once.
// * The expert's tokens (at most 128 per pass) are gathered, split into a
//   pair of bf16 values (high part + rounded remainder) and staged in LDS in
//   k-chunks, double-buffered, shared by the workgroup's four waves; each
//   wave reads them as the MFMA B operand.  Tokens are padded to a multiple
//   of 16 only in registers (lanes beyond the bucket feed zeros).
// * The grid is sized for E experts; a workgroup reads the union size on the
//   device and returns at once if its slot is past it, so inactive experts
//   cost one scalar load and no host synchronisation is needed.
// * Workgroups of one expert are placed on one XCD (the dispatcher deals
//   workgroups round-robin over the 8 XCDs), so the expert's activations are
//   read into a single L2.
#include "common.hpp"

namespace eldr {

constexpr int kFfnThreads = 256;  // 4 waves
constexpr int kFfnWaves = kFfnThreads / kWave;
constexpr int kKStep = 32;        // k per MFMA
constexpr int kRing = 4;          // k-steps of weights in flight per wave (prefetch depth)
constexpr int kMaxTiles = 4;      // token tiles of 16 per pass: at most 64 tokens per pass

// Bytes of one LDS staging buffer (two are used, double-buffered).  Large
// enough that a chunk of kRing k-steps fits for the largest pass.
template <int NT>
__host__ __device__ constexpr int lds_buf_bytes() {
  return NT == 1 ? 16 * 1024 : NT == 2 ? 24 * 1024 : 34 * 1024;
}

enum FfnMode { kUp = 0, kDown = 1 };

struct FfnArgs {
  const float* src;            // up: x [T, H]; down: h workspace [T*K, I]
  const uint16_t* wa;          // up: W1 [E, I, H]; down: W2 [E, H, I]
  const uint16_t* wb;          // up: W3 [E, I, H]; down: unused
  const int32_t* offsets;      // [E+1]
  const int32_t* perm_token;   // [T*K]
  const int32_t* union_ids;    // [E]
  const int32_t* union_size;   // [1]
  float* dst;                  // up: h workspace [T*K, I]; down: y_perm [T*K, H]
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

// Pack 8 fp32 values as 8 bf16 high parts and 8 bf16 low parts.
__device__ __forceinline__ void split8(const float4& a, const float4& b, uint4& hi, uint4& lo) {
  const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  uint32_t h[8], l[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) split_bf16(v[i], h[i], l[i]);
  hi = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
  lo = make_uint4(l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16));
}

template <int MODE, int NT>
__global__ __launch_bounds__(kFfnThreads) void ffn_kernel(FfnArgs a) {
  constexpr int kBuf = lds_buf_bytes<NT>();
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

  // A operand: lane reads row (lane % 16) of its tile, k-group (lane / 16).
  const size_t expert_w = (size_t)a.rows * K;
  const int arow = lane & 15;
  const int kgrp = lane >> 4;
  const uint16_t* pa0 = a.wa + (size_t)e * expert_w + (size_t)(ra0 + arow) * K + kgrp * 8;
  const uint16_t* pa1 = (MODE == kUp ? a.wb : a.wa) + (size_t)e * expert_w +
                        (size_t)(ra1 + arow) * K + kgrp * 8;

  for (int p0 = 0; p0 < c_total; p0 += NT * 16) {
    const int c = min(NT * 16, c_total - p0);
    const int nt = (c + 15) / 16;
    // k-steps per staged chunk: a multiple of kRing that fits c token rows.
    const int kcs = max(kRing, (((kBuf / c - 16) / 128) / kRing) * kRing);
    const int stride = lds_stride(kcs);

    __syncthreads();  // the previous pass has finished with LDS
    if (tid < c) tok[tid] = (MODE == kUp) ? a.perm_token[s_begin + p0 + tid] : s_begin + p0 + tid;
    __syncthreads();

    // Fetch this thread's share of chunk [ks, ks + klen) k-steps into registers.
    float4 stg[kGroups][2];
    auto fetch = [&](int ks, int klen) {
      const int gpr = 4 * klen;
      const int ng = c * gpr;
#pragma unroll
      for (int j = 0; j < kGroups; ++j) {
        const int q = tid + kFfnThreads * j;
        if (q < ng) {
          const int n = q / gpr;
          const int gi = q - n * gpr;
          const float4* p =
              reinterpret_cast<const float4*>(a.src + (size_t)tok[n] * K + ks * kKStep + gi * 8);
          stg[j][0] = p[0];
          stg[j][1] = p[1];
        }
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
          uint4 hi, lo;
          split8(stg[j][0], stg[j][1], hi, lo);
          uint4* d = reinterpret_cast<uint4*>(&lds[buf][n * stride + gi * 32]);
          d[0] = hi;
          d[1] = lo;
        }
      }
    };

    f32x4 acc0[NT], acc1[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      acc0[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      acc1[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // Weight ring: slot i holds the fragments of the k-step congruent to i mod kRing.
    uint4 ring0[kRing], ring1[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) {
      if (i < nk) {
        ring0[i] = *reinterpret_cast<const uint4*>(pa0 + i * kKStep);
        ring1[i] = *reinterpret_cast<const uint4*>(pa1 + i * kKStep);
      }
    }

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
      for (int sb = ks; sb < ke; sb += kRing) {  // ks is a multiple of kRing
#pragma unroll
        for (int i = 0; i < kRing; ++i) {
          const int s = sb + i;
          if (s < ke) {
            const uint4 w0 = ring0[i];
            const uint4 w1 = ring1[i];
            if (s + kRing < nk) {
              ring0[i] = *reinterpret_cast<const uint4*>(pa0 + (s + kRing) * kKStep);
              ring1[i] = *reinterpret_cast<const uint4*>(pa1 + (s + kRing) * kKStep);
            }
            const unsigned char* bs = bb + (s - ks) * 128;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              if (t < nt) {
                // Column n of the product depends only on column n of B, so
                // lanes past the bucket read its last token and their
                // columns are simply not stored.
                const int n = min(t * 16 + arow, c - 1);
                const uint4* bp = reinterpret_cast<const uint4*>(bs + n * stride);
                const uint4 bh = bp[0];
                const uint4 bl = bp[1];
                acc0[t] = mfma16x16x32(w0, bh, acc0[t]);
                acc0[t] = mfma16x16x32(w0, bl, acc0[t]);
                acc1[t] = mfma16x16x32(w1, bh, acc1[t]);
                acc1[t] = mfma16x16x32(w1, bl, acc1[t]);
              }
            }
          }
        }
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
            float4 h;
            h.x = silu(acc0[t][0]) * acc1[t][0];
            h.y = silu(acc0[t][1]) * acc1[t][1];
            h.z = silu(acc0[t][2]) * acc1[t][2];
            h.w = silu(acc0[t][3]) * acc1[t][3];
            *reinterpret_cast<float4*>(a.dst + sl * a.rows + r0 + rsub) = h;
          }
        } else {
          if (ok0)
            *reinterpret_cast<float4*>(a.dst + sl * a.rows + r0 + rsub) =
                make_float4(acc0[t][0], acc0[t][1], acc0[t][2], acc0[t][3]);
          if (ok1)
            *reinterpret_cast<float4*>(a.dst + sl * a.rows + r0 + 16 + rsub) =
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
  if (T <= 16)
    launch_ffn<MODE, 1>(a, E, s);
  else if (T <= 32)
    launch_ffn<MODE, 2>(a, E, s);
  else
    launch_ffn<MODE, kMaxTiles>(a, E, s);
}

}  // namespace eldr

extern "C" size_t moe_ffn_workspace_bytes(moe_dims d) {
  if (eldr_host::check_dims(d) != MOE_OK) return 0;
  return (size_t)d.T * d.K * d.I * sizeof(float);
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
                                 float* ws, size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !w1 || !w3 || !ws) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(w1) || !aligned16(w3) || !aligned16(ws)) return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs up{x, w1, w3, offsets, perm_token, union_ids, union_size, ws, d.I, d.H, 0};
  up.tiles = (d.I + eldr::rows_per_block<eldr::kUp>() - 1) / eldr::rows_per_block<eldr::kUp>();
  eldr::launch_ffn_nt<eldr::kUp>(up, d.T, d.E, reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}

extern "C" int moe_expert_ffn_down(const float* ws, const uint16_t* w2, const int32_t* offsets,
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
  eldr::FfnArgs down{ws, w2, nullptr, offsets, perm_token, union_ids, union_size, y_perm, d.H, d.I,
                     0};
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
