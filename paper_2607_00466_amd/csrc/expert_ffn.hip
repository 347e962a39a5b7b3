// moe_expert_ffn: SwiGLU FFN of every expert in the distinct-expert union.
//
// Cost model (Motivation, "Active Expert Count Drives MoE Decode Latency"):
// a decode step must fetch the weights of every expert its batch activates;
// each expert has only a few tokens, so the work is a skinny product that is
// bound by HBM bandwidth.  The design follows from that:
//
// * Two launches.  "up" computes h = silu(W1 x) * (W3 x) for every slot into
//   the workspace (as bf16 pairs, see below); "down" computes y = W2 h.
//   Within each launch a workgroup item is one expert, one band of output
//   rows and up to 64 of the expert's tokens; it streams the band's bf16
//   weights from HBM (128-bit loads straight into the MFMA A operand).
//   Weights come packed by band (moe_pack_up_weights, moe_pack_down_weights):
//   each load instruction reads one contiguous 1 KB MFMA fragment, and a
//   workgroup's loads of one k-step are adjacent, so an item is one
//   contiguous stream.
// * An expert with at most 64 tokens has one item per band, so its weights
//   are read once, with non-temporal loads.  A bigger bucket is split into
//   token groups of 64 whose items for one band get adjacent workgroup slots
//   on one XCD: they run side by side, read the band with ordinary (cacheable)
//   loads, and the second read is served mostly by that XCD's L2 rather than
//   HBM.
// * The item's tokens are gathered, carried as a pair of bf16 values (high
//   part + rounded remainder) and staged in LDS in fixed-shape chunks,
//   double-buffered, shared by the workgroup's four waves; each wave reads
//   them as the MFMA B operand.  Tokens are padded to a multiple of 16 only
//   in registers (lanes past the bucket repeat its last token and their
//   output columns are not stored).
// * Each wave keeps a ring of weight fragments for the next k-steps in
//   flight; a refill is issued right after the MFMAs that consumed its slot,
//   and staging is arranged so that the compiler never has to drain the ring.
// * The grid is sized from E (and T) alone; a workgroup reads the union size
//   on the device and returns at once if it has no item, so inactive experts
//   cost one scalar load and no host synchronisation is needed.
// * Work is dealt to XCDs by hand (the dispatcher deals workgroups
//   round-robin over the 8 XCDs, so workgroup b runs on XCD b % 8), in the
//   union's order, which moe_bucket makes the dispatch order: buckets with
//   more 16-token tiles first, equal ones by ascending id.  With at most 64
//   tokens an expert, the union's experts go round-robin, all of an
//   expert's bands on one XCD (sharing its L2 for the expert's
//   activations).  With more, whole experts are still dealt while every
//   bucket fits one token group; once one does not, bucket sizes are skewed,
//   and the union's (expert, band) units go round-robin instead, so every XCD
//   gets an equal share of every expert; a band's token groups stay on one
//   XCD, next to each other, so their shared weight reads meet in its L2.
//   Either way an XCD runs its largest buckets first.
// * Weights come in one of two formats (a template parameter): bf16, or
//   MXFP4 (FP4 E2M1 codes with one E8M0 scale per 32 values along the
//   reduction axis, the format the paper serves GPT-OSS-120B in), whose
//   codes are expanded to bf16 in registers by the gfx950 scaled convert
//   right before the same MFMAs -- the products are those of the bf16 path
//   on the dequantized weights, for about a quarter of the bytes.
#include <mutex>

#include "common.hpp"

namespace eldr {

#ifndef ELDR_FFN_RING_SMALL
#define ELDR_FFN_RING_SMALL 4
#endif
#ifndef ELDR_FFN_RING_LARGE
#define ELDR_FFN_RING_LARGE 4
#endif

#ifndef ELDR_FFN_UP_WAVES
#define ELDR_FFN_UP_WAVES 4
#endif
#ifndef ELDR_FFN_DOWN_WAVES
#define ELDR_FFN_DOWN_WAVES 4
#endif
#ifndef ELDR_FFN_FP4_RING
#define ELDR_FFN_FP4_RING 8
#endif
#ifndef ELDR_FFN_FP4_CHUNK
#define ELDR_FFN_FP4_CHUNK 4
#endif
#ifndef ELDR_FFN_FP4_MAX_CHUNK
#define ELDR_FFN_FP4_MAX_CHUNK 16
#endif
constexpr int kKStep = 32;        // k per MFMA
constexpr int kFragElems = 512;   // bf16 values in one packed 16 x 32 weight fragment (1 KB)

// Weight formats.
//   kBf16:  packed by moe_pack_up_weights / moe_pack_down_weights; a ring
//           slot is one k-step of the wave's two 16-row tiles, two adjacent
//           1 KB loads.
//   kMxfp4: packed by moe_pack_mxfp4_up / _down; a ring slot is two k-steps
//           of the wave's two 16-row tiles: one 1 KB load of FP4 codes (a
//           lane's 16 bytes are its 8 codes of tile 0 step 0, tile 0 step 1,
//           tile 1 step 0, tile 1 step 1) and one 64-byte load of their E8M0
//           scales (a dword per row, its bytes in the same order).  For up the
//           two tiles are W1's and W3's rows of the band, for down two
//           adjacent 16-row tiles of W2.
enum WeightFmt { kBf16 = 0, kMxfp4 = 1 };

template <int FMT>
__host__ __device__ constexpr int slot_steps() {
  return FMT == kBf16 ? 1 : 2;
}

// Token tiles of 16 per item: at most 128 tokens of an expert for bf16 (32
// for MXFP4 in batches over 64 tokens, so that the large-batch MXFP4 kernel
// fits four workgroups a CU); a larger bucket takes more token groups,
// served from L2.
template <int FMT>
__host__ __device__ constexpr int max_tiles() {
#ifndef ELDR_FFN_FP4_MAX_TILES
#define ELDR_FFN_FP4_MAX_TILES 2
#endif
  return FMT == kBf16 ? 8 : ELDR_FFN_FP4_MAX_TILES;
}

// Ring slots of weights in flight per wave (the prefetch depth of the ring;
// for MXFP4 the most a pass shape uses: a pass never keeps more than one
// staged chunk of slots in flight).
template <int FMT, int NT>
__host__ __device__ constexpr int ring_depth() {
  return FMT == kMxfp4 ? ELDR_FFN_FP4_RING : NT <= 2 ? ELDR_FFN_RING_SMALL : ELDR_FFN_RING_LARGE;
}

// k-steps per staged chunk: a whole number of ring cycles, as many as keep
// one chunk of NT * 16 tokens within about 34 KB of LDS -- except for 128
// tokens, whose chunks are half a ring cycle (2 k-steps) and are run in pairs.
#ifndef ELDR_FFN_CYCLES1
#define ELDR_FFN_CYCLES1 2
#endif
#ifndef ELDR_FFN_CYCLES2
#define ELDR_FFN_CYCLES2 1
#endif
// MXFP4 moves a quarter of bf16's bytes per k-step; its chunks fill a 17 KB
// buffer: 16 token rows of 8 k-steps, 32 of 4, or 64 of 2 (a pass with fewer
// tiles than its kernel lengthens its chunks, up to 16 k-steps).  Half the
// LDS of bf16's chunks, so that more MXFP4 workgroups share a CU and cover
// each other's item starts: measured, more workgroups a CU beat longer
// chunks and deeper rings for these short items.
template <int FMT, int NT>
__host__ __device__ constexpr int chunk_steps() {
  return FMT == kMxfp4
             ? (NT == 1   ? 2 * ELDR_FFN_FP4_CHUNK
                : NT == 2 ? ELDR_FFN_FP4_CHUNK
                          : ELDR_FFN_FP4_CHUNK / 2)
             : NT == 8 ? ring_depth<FMT, NT>() / 2
                       : ring_depth<FMT, NT>() * (NT == 1 ? ELDR_FFN_CYCLES1 : NT == 2 ? ELDR_FFN_CYCLES2 : 1);
}

#ifndef ELDR_FFN_MAX_CHUNK
#define ELDR_FFN_MAX_CHUNK 8
#endif
// Longest chunk of any pass shape (a chunk's k-steps are unrolled).
template <int FMT>
__host__ __device__ constexpr int max_chunk() {
  return FMT == kBf16 ? ELDR_FFN_MAX_CHUNK : ELDR_FFN_FP4_MAX_CHUNK;
}
__host__ __device__ constexpr int min_c(int a, int b) { return a < b ? a : b; }
__host__ __device__ constexpr int pow2_floor(int v) { return v >= 2 ? 2 * pow2_floor(v / 2) : 1; }

// Bytes of one LDS staging buffer (two are used, double-buffered): NT * 16
// token rows of chunk_steps k-steps (128 bytes each) plus 16 bytes of padding.
template <int FMT, int NT>
__host__ __device__ constexpr int lds_buf_bytes() {
  return NT * 16 * (128 * chunk_steps<FMT, NT>() + 16);
}

enum FfnMode { kUp = 0, kDown = 1 };

// Waves per workgroup: each wave owns 16 output rows (up: of W1 and of W3)
// or 32 (down: two 16-row tiles of W2), and all of them share the staged
// activations.
#ifndef ELDR_FFN_FP4_UP_WAVES
#define ELDR_FFN_FP4_UP_WAVES 4
#endif
#ifndef ELDR_FFN_FP4_DOWN_WAVES
#define ELDR_FFN_FP4_DOWN_WAVES 4
#endif
template <int MODE, int FMT>
__host__ __device__ constexpr int ffn_waves() {
  return FMT == kBf16 ? (MODE == kUp ? ELDR_FFN_UP_WAVES : ELDR_FFN_DOWN_WAVES)
                      : (MODE == kUp ? ELDR_FFN_FP4_UP_WAVES : ELDR_FFN_FP4_DOWN_WAVES);
}
template <int MODE, int FMT>
__host__ __device__ constexpr int ffn_threads() {
  return ffn_waves<MODE, FMT>() * kWave;
}

struct FfnArgs {
  const uint4* src;            // up: x [T, H] fp32; down: h [T*K, I] as bf16 pairs
  const uint16_t* wa;          // bf16, packed by band: up W1 and W3; down W2
  const int32_t* offsets;      // [E+1]
  const int32_t* perm_token;   // [T*K]
  const int32_t* union_ids;    // [E]: the union in dispatch order (moe_bucket's second half)
  const int32_t* union_size;   // [1]
  void* dst;                   // up: h [T*K, I] as bf16 pairs; down: y_perm [T*K, H] fp32
  int rows;                    // output rows per expert: up I, down H
  int kdim;                    // reduction length: up H, down I
  int tiles;                   // row bands per expert
  int experts;                 // E
  const u32x4* qcodes;         // MXFP4: packed FP4 codes (up: W1 and W3; down: W2)
  const uint32_t* qscales;     // MXFP4: packed E8M0 scales
  // Routed up launches (the buckets built in the kernel from the routing):
  const int32_t* ids;          // [T, K] each token's experts
  int T, K;
  int32_t* b_counts;           // moe_bucket's outputs, written by workgroup 0
  int32_t* b_offsets;
  int32_t* b_perm_token;
  int32_t* b_pair_pos;
  int32_t* b_union_ids;
  int32_t* b_union_size;
};

// Rows per workgroup: up -> 16 rows per wave (each wave reads the same 16
// rows of W1 and of W3); down -> 32 rows of W2 per wave (two 16-row tiles).
template <int MODE, int FMT>
__host__ __device__ constexpr int rows_per_block() {
  return MODE == kUp ? ffn_waves<MODE, FMT>() * 16 : ffn_waves<MODE, FMT>() * 32;
}

// LDS layout of one staged chunk: per token a row of the chunk's k-steps;
// each k-step holds 4 groups of 8 k-values; each group is 8 bf16 high parts
// then 8 bf16 low parts (32 bytes).  The row stride is 128 bytes per k-step
// plus 16, an odd multiple of 16, so the 16 lanes that read 16 tokens hit
// distinct banks.

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

// 8 FP4 E2M1 codes (a dword, the first in the low nibble) times the E8M0
// scale in the low byte of sc, as the 8 bf16 values of an MFMA operand.  The
// scaled convert multiplies exactly (an E2M1 value has two significant bits)
// for scale codes 1 .. 252.
__device__ __forceinline__ u32x4 expand_fp4(uint32_t w, uint32_t sc) {
  const float x = __uint_as_float((sc & 0xffu) << 23);
  return u32x4{__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, x, 0)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, x, 1)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, x, 2)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, x, 3))};
}

// Activations enter the MFMA B operand as a pair of bf16 numbers (high
// part, rounded remainder).  In LDS, and for h in the workspace, a row of K
// values is K / 8 groups of 32 bytes: 8 bf16 high parts, then the 8 matching
// low parts -- the same 4 bytes per value as fp32.  The up kernel stages x
// from fp32 and splits it on the way into LDS; its epilogue writes h already
// split, so the down kernel stages h with a plain copy.

// Inclusive prefix sum over the 64 lanes of a wave: shifts within rows of 16
// lanes (lanes shifted in from outside the row read 0), then the totals of
// rows 0 and 2 broadcast into rows 1 and 3, then that of rows 0-1 into 2-3.
__device__ __forceinline__ int wave_inclusive_sum(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// LDS of one workgroup: the two activation chunk buffers and the item's
// token list.
template <int FMT, int NT>
struct FfnLds {
  unsigned char buf[2][lds_buf_bytes<FMT, NT>()];
  int tok[NT * 16];
};

struct NoHook {
  __device__ __forceinline__ void operator()() const {}
};

// One item: the token group of up to NT * 16 tokens starting at slot
// s_begin + p0 of expert e's bucket, against row band `tile`.
// EARLY: the prologue's load order (below).  LISTED: L.tok already holds the
// item's tokens (a routed launch lists them from its buckets).
// SHARED: the band is read by more than one token group of the expert; those
// items run side by side on one XCD, so their weight loads are ordinary
// (cacheable) loads and the repeated reads are served by the XCD's L2.
// Every other band is read once, with non-temporal loads.
// before_acts runs (in every thread) once the weight ring is in flight and
// before the first activations are read; after_store once the item's outputs
// are stored.  The fused launch waits for h in the first and publishes h in
// the second; the separate launches pass NoHook.  WT (up): h is stored with
// device-scope stores, written through to memory (the fused launch).
template <int MODE, int NT, int FMT, bool EARLY, bool LISTED, bool SHARED, bool WT, class Before,
          class After>
__device__ __forceinline__ void ffn_item(const FfnArgs& a, FfnLds<FMT, NT>& L, const int e, const int tile,
                                         const int s_begin, const int p0, const int c, Before&& before_acts,
                                         After&& after_store) {
    constexpr int kFfnThreads = ffn_threads<MODE, FMT>();
    constexpr int kBuf = lds_buf_bytes<FMT, NT>();
    constexpr int kRing = ring_depth<FMT, NT>();
    constexpr int kSlot = slot_steps<FMT>();  // k-steps per ring slot
    static_assert(ffn_waves<MODE, FMT>() == 4,
                  "the packed weight layouts put 4 waves' fragments side by side per band");
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int K = a.kdim;
    const int nk = K / kKStep;
    const int nslot = nk / kSlot;  // ring slots of a row band
    const int arow = lane & 15;
    const int kgrp = lane >> 4;
    auto& lds = L.buf;
    auto& tok = L.tok;
    constexpr bool kShared = SHARED;
    const int nt = (c + 15) / 16;

    const int r0 = tile * rows_per_block<MODE, FMT>() + wave * (MODE == kUp ? 16 : 32);
    const bool ok0 = r0 < a.rows;
    const bool ok1 = MODE == kUp ? ok0 : (r0 + 16 < a.rows);

    // A operand: lane holds row (lane % 16) of its 16-row tile, k-group
    // (lane / 16).  bf16 weights are packed by band (moe_pack_up_weights,
    // moe_pack_down_weights): for each k-step the band's waves' two 1 KB
    // fragments lie side by side (up: W1 then W3 of the wave's 16 rows; down:
    // the wave's two 16-row tiles of W2), so the workgroup streams one
    // contiguous stretch.  A wave past a short last band re-reads the band's
    // last wave and stores nothing.
    constexpr int kWaveRows = MODE == kUp ? 16 : 32;
    constexpr int kMats = MODE == kUp ? 2 : 1;  // matrices a band interleaves
    const int waves_b = min(rows_per_block<MODE, FMT>(), a.rows - tile * rows_per_block<MODE, FMT>()) /
                        kWaveRows;
    const int wc = min(wave, waves_b - 1);
    const size_t step_elems = (size_t)waves_b * 2 * kFragElems;
    const uint16_t* pa0 = a.wa +
                          ((size_t)e * a.rows + (size_t)tile * rows_per_block<MODE, FMT>()) *
                              (size_t)K * kMats +
                          (size_t)(2 * wc) * kFragElems + lane * 8;
    const uint16_t* pa1 = pa0 + kFragElems;
    // MXFP4: the wave's two tiles are one wave band (up: 16 rows of W1 and
    // W3; down: 32 rows of W2), 64 code pieces and 16 scale dwords a slot;
    // the workgroup band's wave bands lie side by side slot by slot
    // (moe_pack_mxfp4_up / _down), and a wave past a short last band re-reads
    // the band's last wave band.
    constexpr int kBandRows = MODE == kUp ? 16 : 32;
    const int nwb = a.rows / kBandRows;
    const int wb_q = min(rows_per_block<MODE, FMT>() / kBandRows, nwb - tile * (rows_per_block<MODE, FMT>() / kBandRows));
    const size_t q0 = ((size_t)e * nwb + (size_t)tile * (rows_per_block<MODE, FMT>() / kBandRows)) * nslot +
                      (size_t)min(wave, wb_q - 1);
    const u32x4* pq = a.qcodes + q0 * 64 + lane;
    const uint32_t* ps = a.qscales + q0 * 16 + arow;

    // Weight ring: slot i holds the weights of the ring slot congruent to i
    // mod kRing.  Loads past the last slot re-read the last one (always
    // issued, never used), which keeps the loop free of branches.
    u32x4 ring0[kRing], ring1[kRing];  // MXFP4: ring0 holds the codes
    uint32_t rsc[kRing];               // MXFP4: the scales
    // Weights are read once per call, so the loads are non-temporal: they
    // stream past the caches instead of displacing the activations there
    // (a plain streaming read reaches about 7.0 TB/s this way, 6.2 without).
    auto ring_load = [&](const int i, const int si) {
      if constexpr (FMT == kBf16) {
        const u32x4* q0 = reinterpret_cast<const u32x4*>(pa0 + (size_t)si * step_elems);
        const u32x4* q1 = reinterpret_cast<const u32x4*>(pa1 + (size_t)si * step_elems);
        if constexpr (kShared) {
          ring0[i] = *q0;
          ring1[i] = *q1;
        } else {
          ring0[i] = __builtin_nontemporal_load(q0);
          ring1[i] = __builtin_nontemporal_load(q1);
        }
      } else {
        const u32x4* q = &pq[(size_t)si * wb_q * 64];
        const uint32_t* r = &ps[(size_t)si * wb_q * 16];
        if constexpr (kShared) {
          ring0[i] = *q;
          rsc[i] = *r;
        } else {
          ring0[i] = __builtin_nontemporal_load(q);
          rsc[i] = __builtin_nontemporal_load(r);
        }
      }
    };
    // Ring slots [FROM, TO) of the prologue.  A CU keeps only so many loads
    // in flight.  When every item starts with the launch (batches of at most
    // 64 tokens) and its tokens are known without a load (a routed launch, or
    // the down projection, whose tokens are its slots), the loads go out in
    // the order the first k-step needs them: ring slot 0, the first chunk of
    // activations, then the rest of the ring, and the first publish waits
    // for the activations and slot 0 alone.  Otherwise (a token list to load
    // first, or items that start behind others on a busy CU) the whole ring
    // goes out first (measured: 2% on the mixed 48-layer step at T=128).
    constexpr bool kEarlyActs = EARLY;
    auto ring_prologue = [&](auto FROM_, auto TO_) {
#pragma unroll
      for (int i = decltype(FROM_)::value; i < decltype(TO_)::value; ++i) ring_load(i, min(i, nslot - 1));
    };
    auto stage_tokens = [&]() {
      __syncthreads();  // the previous item has finished with LDS
      // (a routed launch has listed the tokens already)
      if (!LISTED && tid < c)
        tok[tid] = (MODE == kUp) ? a.perm_token[s_begin + p0 + tid] : s_begin + p0 + tid;
      __syncthreads();
    };

    // bf16 issues the ring (or its slot 0) before the pass shape is chosen;
    // MXFP4's ring depth depends on the pass shape, so each pass fills its own.
    if constexpr (FMT == kBf16) {
      ring_prologue(Int<0>{}, Int<kEarlyActs ? 1 : kRing>{});
      stage_tokens();
    }

    // Pass shape: NTB token tiles, the LDS buffer split into token rows of
    // kChunk k-steps -- fewer tokens, longer chunks, so every shape fills the
    // same buffer and a small bucket crosses as few barriers as a large one.
    auto run_pass = [&](auto NTB_) {
      constexpr int NTB = decltype(NTB_)::value;
      // (a power of two, so that it divides the ring cycle or a multiple of it)
      constexpr int kChunk = pow2_floor(min_c(chunk_steps<FMT, NT>() * NT / NTB, max_chunk<FMT>()));
      constexpr int kStride = 128 * kChunk + 16;  // bytes per staged token row: an odd multiple of 16
      // ring slots this pass keeps in flight
      constexpr int kRingP = FMT == kBf16 ? kRing : min_c(kRing, kChunk / kSlot);
      // A chunk is a whole number of ring cycles, or (128 token rows) half of
      // one: then chunks run in kPhases consecutive phases, chunk c in phase
      // c % kPhases, whose ring slots start kChunk k-steps further round.
      constexpr int kPhases = kChunk >= kRingP * kSlot ? 1 : kRingP * kSlot / kChunk;
      static_assert(kPhases == 1 ? kChunk % (kRingP * kSlot) == 0 : kPhases * kChunk == kRingP * kSlot,
                    "a chunk is a whole number of ring cycles, or an exact fraction of one");
      static_assert(NTB * 16 * kStride <= kBuf, "a chunk fits its buffer");
      constexpr int kGroups = NTB * 16 * 4 * kChunk / kFfnThreads;  // staged 32-byte groups per thread
      static_assert(kGroups * kFfnThreads == NTB * 16 * 4 * kChunk, "groups divide evenly");
      if constexpr (FMT == kMxfp4) {
        ring_prologue(Int<0>{}, Int<kEarlyActs ? 1 : kRingP>{});
        stage_tokens();
      }

      // Activations are staged in chunks of kChunk k-steps.  Every chunk has
      // the same shape, so the groups a thread moves, their LDS places and the
      // number of loads issued between a chunk's fetch and its publish are
      // compile-time constants: the compiler then waits only for the staged
      // groups at a publish, never for the weights in flight behind them.
      // Group q of a chunk is token row q / (4 kChunk), 32-byte group
      // q % (4 kChunk); groups past the bucket or past the last k-step re-read
      // group 0 of the chunk.
      const size_t row_groups = (size_t)K / 8;  // 32-byte groups per activation row
      u32x4 stg[kGroups][2];
      auto group_ok = [&](int j, int ks) {
        const int q = tid + kFfnThreads * j;
        return q / (4 * kChunk) < c && ks * 4 + q % (4 * kChunk) < 4 * nk;
      };
      auto fetch = [&](int ks) {
  #pragma unroll
        for (int j = 0; j < kGroups; ++j) {
          const int q = tid + kFfnThreads * j;
          const bool ok = group_ok(j, ks);
          const int n = ok ? q / (4 * kChunk) : 0;
          const int gi = ok ? q % (4 * kChunk) : 0;
          const u32x4* p =
              reinterpret_cast<const u32x4*>(a.src) + 2 * ((size_t)tok[n] * row_groups + ks * 4 + gi);
          stg[j][0] = p[0];
          stg[j][1] = p[1];
        }
      };
      // Every group is written, valid or not: the places of invalid groups
      // (token rows >= c, k-steps past the end) lie inside the buffer and are
      // never read, and unconditional stores keep every path's wait the same.
      auto publish = [&](int buf) {
  #pragma unroll
        for (int j = 0; j < kGroups; ++j) {
          const int q = tid + kFfnThreads * j;
          const int n = q / (4 * kChunk);
          const int gi = q % (4 * kChunk);
          u32x4* d = reinterpret_cast<u32x4*>(&lds[buf][n * kStride + gi * 32]);
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
      };

      f32x4 acc0[NTB], acc1[NTB];
  #pragma unroll
      for (int t = 0; t < NTB; ++t) {
        acc0[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc1[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      }

      // One k-step: multiply the weights of chunk-relative step I (ring slot
      // (I / kSlot) mod kRingP) against the staged tokens of step s, and after
      // a slot's last k-step refill it with the slot kRingP ahead.  The refill
      // is issued after the MFMAs that read the slot, into the same
      // registers, and a scheduling barrier keeps it there, so each slot
      // stays in place and kRingP slots of loads are always in flight.
      auto kstep = [&](auto PH, auto I, int s, const unsigned char* bb, int ks) {
        constexpr int i = ((decltype(PH)::value * kChunk + decltype(I)::value) / kSlot) % kRingP;
        constexpr int j = decltype(I)::value % kSlot;
        const unsigned char* bs = bb + (s - ks) * 128;
        u32x4 a0, a1;
        if constexpr (FMT == kBf16) {
          a0 = ring0[i];
          a1 = ring1[i];
        } else {
          a0 = expand_fp4(ring0[i][j], rsc[i] >> (8 * j));
          a1 = expand_fp4(ring0[i][2 + j], rsc[i] >> (8 * (2 + j)));
        }
        if constexpr (NTB == 8) {
          // The widest pass runs tile by tile and only over the bucket's
          // tiles: the grouped form below needs more registers than two
          // waves a SIMD leave it.  Lanes past the bucket read its last
          // token; their columns are not stored.
#pragma unroll
          for (int t = 0; t < NTB; ++t) {
            if (t < nt) {
              const int n = min(t * 16 + arow, c - 1);
              const u32x4* bp = reinterpret_cast<const u32x4*>(bs + n * kStride);
              const u32x4 bh = bp[0];
              const u32x4 bl = bp[1];
              acc0[t] = mfma16x16x32(a0, bh, acc0[t]);
              acc0[t] = mfma16x16x32(a0, bl, acc0[t]);
              acc1[t] = mfma16x16x32(a1, bh, acc1[t]);
              acc1[t] = mfma16x16x32(a1, bl, acc1[t]);
            }
          }
        } else {
          // Token tiles in groups of up to 4: the group's B operands are read
          // from LDS first, then its high-part products, then its low-part
          // ones (the two products into one accumulator are a group apart).
          // Every tile of the pass is multiplied: column n of the product
          // depends only on column n of B, so lanes past the bucket read its
          // last token, and tiles and columns past it are simply not stored.
          constexpr int kGrp = NTB <= 4 ? NTB : 2;
          static_assert(NTB % kGrp == 0, "whole tile groups");
          static_for<NTB / kGrp>([&](auto G) {
            constexpr int t0 = decltype(G)::value * kGrp;
            u32x4 bh[kGrp], bl[kGrp];
#pragma unroll
            for (int q = 0; q < kGrp; ++q) {
              const int n = min((t0 + q) * 16 + arow, c - 1);
              const u32x4* bp = reinterpret_cast<const u32x4*>(bs + n * kStride);
              bh[q] = bp[0];
              bl[q] = bp[1];
            }
#pragma unroll
            for (int q = 0; q < kGrp; ++q) {
              acc0[t0 + q] = mfma16x16x32(a0, bh[q], acc0[t0 + q]);
              acc1[t0 + q] = mfma16x16x32(a1, bh[q], acc1[t0 + q]);
            }
#pragma unroll
            for (int q = 0; q < kGrp; ++q) {
              acc0[t0 + q] = mfma16x16x32(a0, bl[q], acc0[t0 + q]);
              acc1[t0 + q] = mfma16x16x32(a1, bl[q], acc1[t0 + q]);
            }
          });
        }
        if constexpr (j == kSlot - 1) ring_load(i, min(s / kSlot + kRingP, nslot - 1));
        __builtin_amdgcn_sched_barrier(0);
      };

      // Chunk 0 is staged before the loop.  Each chunk then fetches the next
      // one (always issued: the last full chunk fetches the tail chunk, or
      // itself again), runs kChunk k-steps, unrolled, and publishes the next
      // chunk into the other buffer.  In steady state the staged groups are
      // older than the weight loads behind them, so a publish waits for them
      // alone.  Chunk c starts at k-step c * kChunk, a multiple of the ring
      // cycle plus kChunk * (c % kPhases), so its step I sits in ring slot
      // (kChunk * (c % kPhases) + I) / kSlot mod kRingP, a constant of the
      // phase.  The buffer published at the end of chunk c was last read in
      // chunk c - 1, before the previous barrier.
      const int nfull = nk / kChunk;
      const int last_start = ((nk - 1) / kChunk) * kChunk;
      auto chunk = [&](auto PH, const int ch) {
        const int ks = ch * kChunk;
        const int next = min(ks + kChunk, last_start);
        fetch(next);
        const unsigned char* bb = &lds[ch & 1][kgrp * 32];
        static_for<kChunk>([&](auto I) { kstep(PH, I, ks + decltype(I)::value, bb, ks); });
        publish((ch + 1) & 1);
        __syncthreads();
      };
      before_acts();
      fetch(0);
      if constexpr (kEarlyActs) ring_prologue(Int<1>{}, Int<kRingP>{});
      publish(0);
      __syncthreads();
      const int nround = nfull - nfull % kPhases;
      for (int ch = 0; ch < nround; ch += kPhases)
        static_for<kPhases>([&](auto PH) { chunk(PH, ch + decltype(PH)::value); });
      if constexpr (kPhases > 1) {
        static_for<kPhases - 1>([&](auto PH) {
          if (decltype(PH)::value < nfull - nround) chunk(PH, nround + decltype(PH)::value);
        });
      }
      // Tail chunk (when nk is not a multiple of kChunk), already staged.
      if (nfull * kChunk < nk) {
        const int ks = nfull * kChunk;
        const unsigned char* bb = &lds[nfull & 1][kgrp * 32];
        static_for<kPhases>([&](auto PH) {
          if (nfull % kPhases == decltype(PH)::value) {
            static_for<kChunk>([&](auto I) {
              if (ks + decltype(I)::value < nk) kstep(PH, I, ks + decltype(I)::value, bb, ks);
            });
          }
        });
      }

      // ---- epilogue: lane holds rows r0 + 4 * (lane / 16) + i of token lane % 16
      const int rsub = 4 * kgrp;
  #pragma unroll
      for (int t = 0; t < NTB; ++t) {
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
              if constexpr (WT) {
                const uint64_t h64 = (uint64_t)(hi[0] | (hi[1] << 16)) | ((uint64_t)(hi[2] | (hi[3] << 16)) << 32);
                const uint64_t l64 = (uint64_t)(lo[0] | (lo[1] << 16)) | ((uint64_t)(lo[2] | (lo[3] << 16)) << 32);
                __hip_atomic_store(reinterpret_cast<uint64_t*>(grp), h64, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(reinterpret_cast<uint64_t*>(grp + 16), l64, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
              } else {
                *reinterpret_cast<uint2*>(grp) = make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16));
                *reinterpret_cast<uint2*>(grp + 16) = make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16));
              }
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
      after_store();
    };
    if constexpr (NT == 1) {
      run_pass(Int<1>{});
    } else if constexpr (NT == 2) {
      if (nt == 1) run_pass(Int<1>{});
      else run_pass(Int<2>{});
    } else if constexpr (NT == 4) {
      if (nt == 1) run_pass(Int<1>{});
      else if (nt == 2) run_pass(Int<2>{});
      else run_pass(Int<4>{});
    } else {
      static_assert(NT == 8, "token tiles per item: 1, 2, 4 or 8");
      if (nt == 1) run_pass(Int<1>{});
      else if (nt == 2) run_pass(Int<2>{});
      else if (nt <= 4) run_pass(Int<4>{});
      else run_pass(Int<8>{});
    }
}

// The buckets of moe_bucket, built in LDS by a workgroup of a routed launch.
struct RouteLds {
  uint32_t mask[2 * MOE_MAX_E];       // token bitmaps: bit t of word t / 32
  int off[MOE_MAX_E];                 // bucket offsets
  unsigned long long cls[4][4];       // [wave][class - 1] ballots
  int wn[4], wp[4];                   // per-wave totals: pairs, experts
  int bad, e;
};

// Builds the buckets of moe_bucket in LDS from the routing ids [T, K] (T <= 64,
// so a token bitmap is two words): counts, offsets, the union in dispatch
// order, and the expert at the union position pick(U) returns for this
// workgroup (-1: none); workgroup 0 also writes them out for the later calls
// (the down projection, the combine).  Same results as moe_bucket, bit for
// bit.  Returns whether the workgroup has an item: R.e is its expert.  Every
// branch is uniform over the workgroup.
template <int kThreads, class Pick>
__device__ __forceinline__ bool route_buckets(const FfnArgs& a, RouteLds& R, Pick&& pick) {
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int K = a.K, E = a.experts, P = a.T * a.K;
  constexpr int kIdsPerThread = 64 * MOE_MAX_K / kThreads;
  int idv[kIdsPerThread];
#pragma unroll
  for (int j = 0; j < kIdsPerThread; ++j) {
    const int p = tid + kThreads * j;
    idv[j] = p < P ? a.ids[p] : 0;
  }
  for (int i = tid; i < 2 * E; i += kThreads) R.mask[i] = 0u;
  if (tid == 0) {
    R.bad = 0;
    R.e = -1;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kIdsPerThread; ++j) {
    const int p = tid + kThreads * j;
    if (p < P) {
      const int t = p / K;
      const int e = idv[j];
      if (e < 0 || e >= E) {
        R.bad = 1;
      } else {
        const uint32_t bit = 1u << (t & 31);
        if (atomicOr(&R.mask[2 * e + (t >> 5)], bit) & bit) R.bad = 1;  // an expert twice
      }
    }
  }
  __syncthreads();
  // One expert a thread.  Its count n, and its class: the 16-token tiles of
  // its bucket (1 .. 4 here, T <= 64; 0 when absent).  The dispatch order
  // (more tiles first, equal tiles by ascending id) ranks an expert by the
  // experts of higher classes plus those of its class with lower ids, which
  // per-wave ballots of each class give directly.  Offsets and ascending
  // union positions are prefix sums: within a wave by DPP, across the
  // four waves from their totals.
  static_assert(MOE_MAX_E <= kThreads && kThreads == 4 * kWave, "one expert a thread");
  const int me = tid;
  const int n = me < E ? __popc(R.mask[2 * me]) + __popc(R.mask[2 * me + 1]) : 0;
  const int cls = (n + 15) / 16;
  const int incl_n = wave_inclusive_sum(n);
  const int incl_p = wave_inclusive_sum(n > 0 ? 1 : 0);
#pragma unroll
  for (int c = 1; c <= 4; ++c) {
    const unsigned long long b = __ballot(cls == c);
    if (lane == 0) R.cls[wave][c - 1] = b;
  }
  if (lane == kWave - 1) {
    R.wn[wave] = incl_n;
    R.wp[wave] = incl_p;
  }
  __syncthreads();
  int U = 0, before_n = 0, before_p = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    U += R.wp[w];
    before_n += w < wave ? R.wn[w] : 0;
    before_p += w < wave ? R.wp[w] : 0;
  }
  const int pairs = R.wn[0] + R.wn[1] + R.wn[2] + R.wn[3];
  const int u = pick(U);  // this workgroup's union position
  // Workgroups without an item leave here (the grid is sized from E); the
  // first stays, to write the buckets out.
  if (u < 0 && blockIdx.x != 0) return false;
  const int off = before_n + incl_n - n;
  int rank = 0;
  if (cls > 0) {
#pragma unroll
    for (int c = 4; c >= 1; --c) {
      if (c > cls) {
#pragma unroll
        for (int w = 0; w < 4; ++w) rank += __popcll(R.cls[w][c - 1]);
      }
    }
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const unsigned long long b = R.cls[w][cls - 1];
      rank += w < wave ? __popcll(b) : w == wave ? __popcll(b & ((1ull << lane) - 1ull)) : 0;
    }
  }
  if (me < E) R.off[me] = off;
  if (cls > 0 && rank == u) R.e = me;
  const bool ok = R.bad == 0 && pairs == P;
  if (blockIdx.x == 0) {
    if (me < E) {
      a.b_counts[me] = n;
      a.b_offsets[me] = off;
      if (n > 0) {
        a.b_union_ids[before_p + incl_p - 1] = me;
        a.b_union_ids[E + rank] = me;
      }
      if (me >= U) {
        a.b_union_ids[me] = -1;
        a.b_union_ids[E + me] = -1;
      }
    }
    if (tid == 0) {
      a.b_offsets[E] = pairs;
      *a.b_union_size = ok ? U : -1;
    }
    __syncthreads();  // R.off complete (uniform: the whole of workgroup 0)
    if (ok) {
#pragma unroll
      for (int j = 0; j < kIdsPerThread; ++j) {
        const int p = tid + kThreads * j;
        if (p < P) {
          const int t = p / K;
          const int e = idv[j];
          const int w = t >> 5;
          const int below = (w ? __popc(R.mask[2 * e]) : 0) +
                            __popc(R.mask[2 * e + w] & ((1u << (t & 31)) - 1u));
          const int sl = R.off[e] + below;
          a.b_perm_token[sl] = t;
          a.b_pair_pos[p] = sl;
        }
      }
    }
  }
  __syncthreads();
  return ok && R.e >= 0;  // invalid routing, or no expert at this position: nothing
}

// Lists expert e's tokens of a routed launch in ascending order into tok: the
// rank of token tid's bit.  Returns the count.
__device__ __forceinline__ int route_tokens(const FfnArgs& a, const RouteLds& R, const int e, int* tok) {
  const int tid = threadIdx.x;
  if (tid < a.T) {
    const uint64_t m = (uint64_t)R.mask[2 * e] | ((uint64_t)R.mask[2 * e + 1] << 32);
    if ((m >> tid) & 1u) tok[__popcll(m & ((1ull << tid) - 1ull))] = tid;
  }
  return __popc(R.mask[2 * e]) + __popc(R.mask[2 * e + 1]);
}

template <int MODE, int NT, bool MULTI, int FMT, bool ROUTED>
// (128-token passes: held to two waves a SIMD, the LDS limit, so registers
// never lower it; the large-batch MXFP4 kernel: at least three, so that its
// registers leave room for three or four workgroups a CU)
__global__ __launch_bounds__((ffn_threads<MODE, FMT>()))
__attribute__((amdgpu_waves_per_eu(NT == 8 ? 2 : (FMT == kMxfp4 && MULTI ? 3 : 1))))
void ffn_kernel(FfnArgs a) {
  constexpr int kGroupTokens = NT * 16;  // tokens of one expert one workgroup item takes
  __shared__ __attribute__((aligned(16))) FfnLds<FMT, NT> L;
  // The prologue's load order: the first activations early when every item
  // starts with the launch and its tokens are known without a load.
  constexpr bool kEarly = ROUTED || (MODE == kDown && !MULTI);

  // ---- work items -----------------------------------------------------------
  // Workgroups are dealt to the XCDs round-robin, so workgroup b runs on XCD
  // b % 8 and is that XCD's slot b / 8.  An item is (expert, row band, token
  // group of up to kGroupTokens tokens); an XCD's items are numbered expert
  // by expert, and within an expert band by band with the band's token
  // groups adjacent, so the workgroups that read one band's weights for
  // different tokens run side by side and share the XCD's L2.  A slot takes
  // items slot, slot + slots, ... .  Without MULTI (batches of at most
  // kGroupTokens tokens) every expert has one group and the expert at union
  // position u belongs to XCD u % 8; with it, the same holds while every
  // bucket fits one group, and otherwise the union's (expert, band) units are
  // dealt round-robin.
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int xcd = blockIdx.x % kNumXcd;
  const int slot = blockIdx.x / kNumXcd;
  const int slots = gridDim.x / kNumXcd;

  if constexpr (ROUTED) {
    static_assert(!MULTI && MODE == kUp, "routed launches: up projection, batches of <= 64 tokens");
    __shared__ RouteLds R;
    auto pick = [&](const int U) {
      const int u = (slot / a.tiles) * kNumXcd + xcd;
      return u < U ? u : -1;
    };
    if (!route_buckets<ffn_threads<MODE, FMT>()>(a, R, pick)) return;
    const int e = R.e;
    const int c = route_tokens(a, R, e, L.tok);
    ffn_item<MODE, NT, FMT, kEarly, true, false, false>(a, L, e, slot % a.tiles, R.off[e], 0, c, NoHook{},
                                                 NoHook{});
  } else if constexpr (!MULTI) {
    // At most kGroupTokens tokens per expert: slot = (expert / 8) * tiles + band.
    const int u = (slot / a.tiles) * kNumXcd + xcd;
    const int U = *a.union_size;
    if (u >= U) return;  // also covers U < 0 (invalid routing)
    const int e = a.union_ids[u];
    if (e < 0 || e >= a.experts) return;  // not reached for a union member
    const int s_begin = a.offsets[e];
    const int c = a.offsets[e + 1] - s_begin;
    if (c > 0)
      ffn_item<MODE, NT, FMT, kEarly, false, false, false>(a, L, e, slot % a.tiles, s_begin, 0,
                                                    min(c, kGroupTokens), NoHook{}, NoHook{});
  } else {
    // The union lists its experts in dispatch order (moe_bucket: more
    // 16-token tiles first).  A projection's units are (expert, row band)
    // pairs in that order, band by band: unit tiles * u + t is band t of the
    // expert at union position u, and unit k goes to XCD k % 8.  So every XCD gets an
    // equal share of every expert's bands (exactly equal when the band count
    // is a multiple of 8, within one band otherwise) and the XCDs' loads match
    // however skewed the buckets are; an XCD's items follow the union order,
    // so the largest buckets start first; and an expert's items there are its
    // bands in order with each band's token groups adjacent, reading the same
    // weights side by side through the XCD's L2.
    //
    // Every wave holds the whole union, four positions a lane (4 * lane + j;
    // union_ids is -1 past the union and is read together with union_size):
    // id, bucket start and size, and the first item and number of items of
    // the expert on this XCD.  Loads are issued unconditionally (from clamped
    // indices), so the wave waits for two round trips rather than one a slot.
    static_assert(MOE_MAX_E <= 4 * kWave, "four union positions a lane");
    int e_j[4], sb_j[4], hi_j[4], c_j[4], n_j[4], first_j[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) e_j[j] = a.union_ids[min(4 * lane + j, a.experts - 1)];
    const int U = *a.union_size;  // U <= 0 (empty or invalid routing): no items
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int ec = e_j[j] >= 0 && e_j[j] < a.experts ? e_j[j] : 0;
      sb_j[j] = a.offsets[ec];
      hi_j[j] = a.offsets[ec + 1];
    }
    // (keeps the compiler from sinking a load into the branch that uses it)
#pragma unroll
    for (int j = 0; j < 4; ++j) asm volatile("" : "+v"(sb_j[j]), "+v"(hi_j[j]));
    int lane_n = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int u = 4 * lane + j;
      const bool member = u < min(U, a.experts) && e_j[j] >= 0 && e_j[j] < a.experts;
      c_j[j] = member ? max(hi_j[j] - sb_j[j], 0) : 0;
      const int g = (c_j[j] + kGroupTokens - 1) / kGroupTokens;
      const int band0 = (xcd - a.tiles * u) & (kNumXcd - 1);  // first band on this XCD
      const int nb = band0 < a.tiles ? (a.tiles - 1 - band0) / kNumXcd + 1 : 0;
      n_j[j] = nb * g;
      first_j[j] = lane_n;
      lane_n += n_j[j];
    }
    // When every bucket fits one token group, the batch is not skewed enough
    // to need the band dealing: whole experts go round-robin over the XCDs as
    // for small batches, so that an expert's activations (x rows for up, h
    // for down) are fetched into one XCD's L2 rather than into all eight.
    int cmax = max(max(c_j[0], c_j[1]), max(c_j[2], c_j[3]));
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) cmax = max(cmax, __shfl_xor(cmax, off));
    if (__builtin_amdgcn_readfirstlane(cmax) <= kGroupTokens) {
      const int u = (slot / a.tiles) * kNumXcd + xcd;
      if (u >= U || u >= a.experts) return;  // also covers U < 0 (invalid routing)
      // union position u: its entries, from the lane that holds them
      const int ls = u / 4, js = u % 4;
      int ie = 0, isb = 0, ic = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (j == js) {
          ie = __builtin_amdgcn_readlane(e_j[j], ls);
          isb = __builtin_amdgcn_readlane(sb_j[j], ls);
          ic = __builtin_amdgcn_readlane(c_j[j], ls);
        }
      }
      if (ic > 0)
        ffn_item<MODE, NT, FMT, MODE == kDown, false, false, false>(a, L, ie, slot % a.tiles, isb, 0, ic,
                                                                   NoHook{}, NoHook{});
      return;
    }
    const int incl = wave_inclusive_sum(lane_n);
    const int total = __builtin_amdgcn_readlane(incl, kWave - 1);
    if (slot >= total) return;
    // The table moves to LDS for the item loop: held in registers it would
    // stay live across every item and crowd the 128-token passes.
    __shared__ int4 lk_first[kWave], lk_n[kWave], lk_c[kWave], lk_e[kWave], lk_sb[kWave];
    if (wave == 0) {
      const int f0 = incl - lane_n;
      lk_first[lane] = make_int4(first_j[0] + f0, first_j[1] + f0, first_j[2] + f0, first_j[3] + f0);
      lk_n[lane] = make_int4(n_j[0], n_j[1], n_j[2], n_j[3]);
      lk_c[lane] = make_int4(c_j[0], c_j[1], c_j[2], c_j[3]);
      lk_e[lane] = make_int4(e_j[0], e_j[1], e_j[2], e_j[3]);
      lk_sb[lane] = make_int4(sb_j[0], sb_j[1], sb_j[2], sb_j[3]);
    }
    __syncthreads();
    for (int item = slot; item < total; item += slots) {
      // the union position whose items cover this one
      const int4 f4 = lk_first[lane];
      const int4 n4 = lk_n[lane];
      const int fj[4] = {f4.x, f4.y, f4.z, f4.w};
      const int nj[4] = {n4.x, n4.y, n4.z, n4.w};
      int js = -1, ls = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const unsigned long long hit = __ballot(nj[j] > 0 && fj[j] <= item && item < fj[j] + nj[j]);
        if (hit != 0) {
          js = j;
          ls = __ffsll(hit) - 1;
        }
      }
      if (js < 0) break;  // not reached: the ranges cover [0, total)
      js = __builtin_amdgcn_readfirstlane(js);
      ls = __builtin_amdgcn_readfirstlane(ls);
      // union position 4 * ls + js: its entries, read at a uniform address
      auto pick = [&](const int4* v) { return reinterpret_cast<const int*>(v)[4 * ls + js]; };
      const int cu = pick(lk_c);
      const int g = (cu + kGroupTokens - 1) / kGroupTokens;
      const int r = item - pick(lk_first);
      const int band = r / g;
      const int group = r - band * g;
      const int tile = ((xcd - a.tiles * (4 * ls + js)) & (kNumXcd - 1)) + kNumXcd * band;
      const int p0 = group * kGroupTokens;
      const int c = min(kGroupTokens, cu - p0);
      if (c > 0) {
        const int ie = pick(lk_e);
        const int isb = pick(lk_sb);
        if (g > 1)
          ffn_item<MODE, NT, FMT, kEarly, false, true, false>(a, L, ie, tile, isb, p0, c, NoHook{}, NoHook{});
        else
          ffn_item<MODE, NT, FMT, kEarly, false, false, false>(a, L, ie, tile, isb, p0, c, NoHook{}, NoHook{});
      }
    }
  }
}

// int32 words between the counters of consecutive union positions in the
// fused launch's sync buffer (one 256-byte line each).
constexpr int kSyncStride = 64;

// Spins of a fused down item's wait for its expert's h before it gives up and
// raises the error word (never in a correct run: see ffn_fused_kernel).
#ifndef ELDR_FFN_SPIN_LIMIT
#define ELDR_FFN_SPIN_LIMIT (1 << 18)
#endif

// Buckets, up projection and down projection in one launch (batches of at
// most 64 tokens, every expert one token group).  Each workgroup builds the
// buckets (route_buckets), then takes one item by its XCD slot: an XCD's items
// are the up bands of its union experts (positions u = xcd, xcd + 8, ...),
// expert by expert, then their down bands, then nothing.  A down item streams
// its first W2 weights, then waits until every up band of its expert has
// stored h, then reads h.
//
// Synchronisation, over `sync` (int32 [64 E + 1], zero before the first call),
// without cache write-backs or invalidations (each costs a pass over an XCD's
// L2; one per up item tripled the layer's time):
// * an up item stores its h with device-scope stores, which write through to
//   memory, waits in every wave until its stores are acknowledged, passes a
//   barrier, and adds 1 to its position's up counter (an atomic at device
//   scope);
// * a down item's thread 0 polls that counter with device-scope loads until it
//   reads the up band count, then the workgroup reads h with ordinary loads.
//   No CU of the device can hold a stale copy of those lines: the launch
//   starts with the caches invalidated, h rows are whole 128-byte lines (the
//   entry points require a 128-byte aligned workspace, and a row is 4 I
//   bytes with I % 32 == 0), and only the expert's own down items read its rows,
//   after the wait;
// * each down item then counts itself in the position's down counter, and
//   the expert's last one sets both back to 0, so every call leaves `sync` as
//   it found it.
// Progress: the dispatcher starts an XCD's workgroups in index order, and
// every up item comes before every down item of its XCD (and before every
// down item of its expert in index order, whatever XCD runs it), so an up
// item never waits behind a down item.  A wait that outlasts
// ELDR_FFN_SPIN_LIMIT polls (not reached in a correct run) sets sync[64 E]
// to 1 and goes on, so every wave ends.
template <int NT, int FMT>
__global__ __launch_bounds__((ffn_threads<kUp, FMT>())) void ffn_fused_kernel(FfnArgs up, FfnArgs dn,
                                                                              int32_t* sync) {
  static_assert(ffn_threads<kUp, FMT>() == ffn_threads<kDown, FMT>(), "one workgroup shape");
  __shared__ __attribute__((aligned(16))) FfnLds<FMT, NT> L;
  __shared__ RouteLds R;
  const int xcd = blockIdx.x % kNumXcd;
  const int slot = blockIdx.x / kNumXcd;
  int is_down = 0, band = 0;
  auto pick = [&](const int U) {
    const int ux = U > xcd ? (U - xcd + kNumXcd - 1) / kNumXcd : 0;  // union experts on this XCD
    const int n_up = up.tiles * ux;
    if (slot < n_up) {
      band = slot % up.tiles;
      return (slot / up.tiles) * kNumXcd + xcd;
    }
    const int s2 = slot - n_up;
    if (s2 < dn.tiles * ux) {
      is_down = 1;
      band = s2 % dn.tiles;
      return (s2 / dn.tiles) * kNumXcd + xcd;
    }
    return -1;
  };
  int u = -1;
  auto pick_u = [&](const int U) {
    u = pick(U);
    return u;
  };
  if (!route_buckets<ffn_threads<kUp, FMT>()>(up, R, pick_u)) return;
  const int e = __builtin_amdgcn_readfirstlane(R.e);
  u = __builtin_amdgcn_readfirstlane(u);
  band = __builtin_amdgcn_readfirstlane(band);
  // One 256-byte line per union position: word 0 counts the up items that
  // stored h, word 1 the down items past their wait.  Polled counters packed
  // into a few lines put every poll on one memory channel, and the weight
  // streams queued behind them (measured: 85 -> 67 us at U = 32, T = 64).
  const int E = up.experts;
  int32_t* up_done = sync + kSyncStride * u;
  int32_t* dn_seen = up_done + 1;
  int32_t* err = sync + kSyncStride * E;  // a wait gave up
  if (__builtin_amdgcn_readfirstlane(is_down) == 0) {
    const int c = route_tokens(up, R, e, L.tok);
    auto publish_h = [&] {
      __builtin_amdgcn_s_waitcnt(0);  // this wave's h stores are acknowledged
      __syncthreads();
      if (threadIdx.x == 0)
        __hip_atomic_fetch_add(up_done, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    ffn_item<kUp, NT, FMT, true, true, false, true>(up, L, e, band, R.off[e], 0, c, NoHook{}, publish_h);
  } else {
    const int c = __popc(R.mask[2 * e]) + __popc(R.mask[2 * e + 1]);
    auto wait_h = [&] {
      if (threadIdx.x == 0) {
        int n = 0;
        while (__hip_atomic_load(up_done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < up.tiles) {
          __builtin_amdgcn_s_sleep(2);
          if (++n == ELDR_FFN_SPIN_LIMIT) {
            __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
        }
        if (__hip_atomic_fetch_add(dn_seen, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
            dn.tiles - 1) {
          // the expert's last down item: nobody reads either counter again in this call
          __hip_atomic_store(up_done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(dn_seen, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      __syncthreads();
    };
    ffn_item<kDown, NT, FMT, false, false, false, false>(dn, L, e, band, R.off[e], 0, c, wait_h, NoHook{});
  }
}

// Token tiles of 16 per item: enough for every bucket when T is small (a
// bucket never exceeds T tokens), at most max_tiles.
template <int FMT>
static int ffn_nt(int T) {
  int nt_T = T;
#ifdef ELDR_FFN_FORCE_NT
  nt_T = 16 * ELDR_FFN_FORCE_NT;
#endif
  return nt_T <= 16 ? 1 : nt_T <= 32 ? 2 : nt_T <= 64 ? 4 : max_tiles<FMT>();
}

// Slots per XCD: one item per (expert, band) of an XCD's share of the
// experts; batches with more tokens than one item takes also get room for an
// XCD's share of the extra token groups (T*K / (NT*16) at most in all), and
// slots loop over any items beyond that.
template <int MODE, int FMT, int NT>
static void launch_ffn(FfnArgs a, int T, int K, int E, hipStream_t s) {
  const int per_xcd = (E + kNumXcd - 1) / kNumXcd;
  // Batches of up to 64 tokens (never the 128-token kernel) deal whole
  // experts; larger ones deal (expert, band) units, balancing skewed buckets.
  if constexpr (NT <= 4) {
    if (T <= NT * 16) {
      hipLaunchKernelGGL((ffn_kernel<MODE, NT, false, FMT, false>), dim3(kNumXcd * a.tiles * per_xcd),
                         dim3(ffn_threads<MODE, FMT>()), 0, s, a);
      return;
    }
  }
  const int extra = (T * K / (NT * 16) + kNumXcd - 1) / kNumXcd;
  hipLaunchKernelGGL((ffn_kernel<MODE, NT, true, FMT, false>), dim3(kNumXcd * a.tiles * (per_xcd + extra)),
                     dim3(ffn_threads<MODE, FMT>()), 0, s, a);
}

// The routed up launch (batches of at most 64 tokens): the grid of the
// whole-expert dealing, each workgroup building the buckets itself.
template <int FMT>
static void launch_ffn_routed(const FfnArgs& a, int T, int E, hipStream_t s) {
  const int per_xcd = (E + kNumXcd - 1) / kNumXcd;
  const dim3 grid(kNumXcd * a.tiles * per_xcd), block(ffn_threads<kUp, FMT>());
  if (T <= 16)
    hipLaunchKernelGGL((ffn_kernel<kUp, 1, false, FMT, true>), grid, block, 0, s, a);
  else if (T <= 32)
    hipLaunchKernelGGL((ffn_kernel<kUp, 2, false, FMT, true>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((ffn_kernel<kUp, 4, false, FMT, true>), grid, block, 0, s, a);
}

// The fused launch: every XCD gets room for the up and down bands of its
// share of E experts; workgroups past the union's items return at once.
template <int FMT>
static void launch_ffn_fused(const FfnArgs& up, const FfnArgs& dn, int32_t* sync, int T, int E,
                             hipStream_t s) {
  const int per_xcd = (E + kNumXcd - 1) / kNumXcd;
  const dim3 grid(kNumXcd * per_xcd * (up.tiles + dn.tiles)), block(ffn_threads<kUp, FMT>());
  if (T <= 16)
    hipLaunchKernelGGL((ffn_fused_kernel<1, FMT>), grid, block, 0, s, up, dn, sync);
  else if (T <= 32)
    hipLaunchKernelGGL((ffn_fused_kernel<2, FMT>), grid, block, 0, s, up, dn, sync);
  else
    hipLaunchKernelGGL((ffn_fused_kernel<4, FMT>), grid, block, 0, s, up, dn, sync);
}

template <int MODE, int FMT>
static void launch_ffn_nt(const FfnArgs& a, int T, int K, int E, hipStream_t s) {
  const int nt = ffn_nt<FMT>(T);
  if (nt == 1)
    launch_ffn<MODE, FMT, 1>(a, T, K, E, s);
  else if (nt == 2)
    launch_ffn<MODE, FMT, 2>(a, T, K, E, s);
  else if (nt == 4 || max_tiles<FMT>() == 4)
    launch_ffn<MODE, FMT, 4>(a, T, K, E, s);
  else
    launch_ffn<MODE, FMT, max_tiles<FMT>()>(a, T, K, E, s);
}

// Row bands of a projection.
template <int MODE, int FMT>
static int ffn_tiles(const moe_dims& d) {
  const int rows = MODE == kUp ? d.I : d.H;
  return (rows + rows_per_block<MODE, FMT>() - 1) / rows_per_block<MODE, FMT>();
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

extern "C" int moe_expert_ffn_up(const float* x, const uint16_t* w13, const int32_t* offsets,
                                 const int32_t* perm_token,
                                 const int32_t* union_ids, const int32_t* union_size, moe_dims d,
                                 void* ws, size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !w13 || !ws) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(w13) || !aligned16(ws)) return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  eldr::FfnArgs up{reinterpret_cast<const uint4*>(x), w13, offsets, perm_token, union_ids + d.E,
                   union_size, ws, d.I, d.H, 0, d.E, nullptr, nullptr};
  up.tiles = eldr::ffn_tiles<eldr::kUp, eldr::kBf16>(d);
  eldr::launch_ffn_nt<eldr::kUp, eldr::kBf16>(up, d.T, d.K, d.E, s);
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
  eldr::FfnArgs down{reinterpret_cast<const uint4*>(ws), w2, offsets, perm_token,
                     union_ids + d.E, union_size, y_perm, d.H, d.I, 0, d.E, nullptr, nullptr};
  down.tiles = eldr::ffn_tiles<eldr::kDown, eldr::kBf16>(d);
  eldr::launch_ffn_nt<eldr::kDown, eldr::kBf16>(down, d.T, d.K, d.E,
                                               reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}

extern "C" int moe_expert_ffn(const float* x, const uint16_t* w13, const uint16_t* w2,
                              const int32_t* offsets,
                              const int32_t* perm_token, const int32_t* union_ids,
                              const int32_t* union_size, moe_dims d, float* y_perm, void* ws,
                              size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !w13 || !w2 || !y_perm || !ws) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(w13) || !aligned16(w2) || !aligned16(y_perm) || !aligned16(ws))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  float* h = static_cast<float*>(ws);
  st = moe_expert_ffn_up(x, w13, offsets, perm_token, union_ids, union_size, d, h, ws_bytes, stream);
  if (st != MOE_OK) return st;
  return moe_expert_ffn_down(h, w2, offsets, perm_token, union_ids, union_size, d, ws_bytes,
                             y_perm, stream);
}

// ---- the allocation-free expert FFN ---------------------------------------------

// The workspace of moe_expert_ffn_noalloc: h of every slot, in a file-scope
// device array of fixed size that each GPU the library runs on holds until the
// process ends.  Host code never passes `scratch` itself (in host code it is
// a stand-in, not a device address): the device address comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kNoallocScratchBytes = size_t(32) << 20;  // 32 MiB
__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device.
int scratch_on_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return MOE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MOE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MOE_OK;
}

}  // namespace

extern "C" size_t moe_expert_ffn_noalloc_max_bytes(void) { return kNoallocScratchBytes; }

extern "C" int moe_expert_ffn_noalloc(const float* x, const uint16_t* w13, const uint16_t* w2,
                                      const int32_t* offsets, const int32_t* perm_token,
                                      const int32_t* union_ids, const int32_t* union_size,
                                      moe_dims d, float* y_perm, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (moe_ffn_workspace_bytes(d) > kNoallocScratchBytes) return MOE_ERR_WORKSPACE;
  void* ws = nullptr;
  st = scratch_on_current_device(&ws);
  if (st != MOE_OK) return st;
  return moe_expert_ffn(x, w13, w2, offsets, perm_token, union_ids, union_size, d, y_perm, ws,
                        kNoallocScratchBytes, stream);
}

// ---- routed up launches: moe_bucket and the up projection in one launch ------

namespace {

// Checks shared by the routed entry points; on success the bucket outputs
// are valid, non-null, 4-byte aligned buffers.
int check_routed(const moe_dims& d, const int32_t* topk_ids, const int32_t* counts,
                 const int32_t* offsets, const int32_t* perm_token, const int32_t* pair_pos,
                 const int32_t* union_ids, const int32_t* union_size) {
  using namespace eldr_host;
  if (!counts || !offsets || !perm_token || !pair_pos || !union_ids || !union_size || !topk_ids)
    return MOE_ERR_INVALID;
  if (!aligned4(topk_ids) || !aligned4(counts) || !aligned4(offsets) || !aligned4(perm_token) ||
      !aligned4(pair_pos) || !aligned4(union_ids) || !aligned4(union_size))
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

}  // namespace

extern "C" int moe_expert_ffn_up_routed(const float* x, const uint16_t* w13,
                                        const int32_t* topk_ids, moe_dims d, int32_t* counts,
                                        int32_t* offsets, int32_t* perm_token, int32_t* pair_pos,
                                        int32_t* union_ids, int32_t* union_size, void* ws,
                                        size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0 || d.T > 64) {
    // nothing to multiply (moe_bucket writes the empty buckets), or too many
    // tokens for the in-kernel buckets: the two calls
    st = moe_bucket(topk_ids, d, counts, offsets, perm_token, pair_pos, union_ids, union_size,
                    stream);
    if (st != MOE_OK || d.T == 0) return st;
    return moe_expert_ffn_up(x, w13, offsets, perm_token, union_ids, union_size, d, ws, ws_bytes,
                             stream);
  }
  if (!x || !w13 || !ws) return MOE_ERR_INVALID;
  st = check_routed(d, topk_ids, counts, offsets, perm_token, pair_pos, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(w13) || !aligned16(ws)) return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs up{reinterpret_cast<const uint4*>(x), w13, offsets, perm_token, union_ids + d.E,
                   union_size, ws, d.I, d.H, 0, d.E, nullptr, nullptr,
                   topk_ids, d.T, d.K, counts, offsets, perm_token, pair_pos, union_ids,
                   union_size};
  up.tiles = eldr::ffn_tiles<eldr::kUp, eldr::kBf16>(d);
  eldr::launch_ffn_routed<eldr::kBf16>(up, d.T, d.E, reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}

// ---- MXFP4 expert weights ----------------------------------------------------

namespace {

int check_mxfp4_dims(const moe_dims& d) {
  const int st = eldr_host::check_dims(d);
  if (st != MOE_OK) return st;
  // a ring slot is two k-steps (64 values) of both reductions
  if (d.H % 64 != 0 || d.I % 64 != 0) return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

}  // namespace

extern "C" int moe_expert_ffn_mxfp4_up(const float* x, const uint8_t* up_codes,
                                       const uint8_t* up_scales, const int32_t* offsets,
                                       const int32_t* perm_token, const int32_t* union_ids,
                                       const int32_t* union_size, moe_dims d, void* ws,
                                       size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_mxfp4_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !up_codes || !up_scales || !ws) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(up_codes) || !aligned4(up_scales) || !aligned16(ws))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs up{reinterpret_cast<const uint4*>(x), nullptr, offsets, perm_token,
                   union_ids + d.E, union_size, ws, d.I, d.H, 0, d.E,
                   reinterpret_cast<const eldr::u32x4*>(up_codes),
                   reinterpret_cast<const uint32_t*>(up_scales)};
  up.tiles = eldr::ffn_tiles<eldr::kUp, eldr::kMxfp4>(d);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  eldr::launch_ffn_nt<eldr::kUp, eldr::kMxfp4>(up, d.T, d.K, d.E, s);
  return launch_status();
}

extern "C" int moe_expert_ffn_mxfp4_down(const void* ws, const uint8_t* down_codes,
                                         const uint8_t* down_scales, const int32_t* offsets,
                                         const int32_t* perm_token, const int32_t* union_ids,
                                         const int32_t* union_size, moe_dims d, size_t ws_bytes,
                                         float* y_perm, void* stream) {
  using namespace eldr_host;
  int st = check_mxfp4_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!ws || !down_codes || !down_scales || !y_perm) return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(ws) || !aligned16(down_codes) || !aligned4(down_scales) || !aligned16(y_perm))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs down{reinterpret_cast<const uint4*>(ws), nullptr, offsets, perm_token,
                     union_ids + d.E, union_size, y_perm, d.H, d.I, 0, d.E,
                     reinterpret_cast<const eldr::u32x4*>(down_codes),
                     reinterpret_cast<const uint32_t*>(down_scales)};
  down.tiles = eldr::ffn_tiles<eldr::kDown, eldr::kMxfp4>(d);
  eldr::launch_ffn_nt<eldr::kDown, eldr::kMxfp4>(down, d.T, d.K, d.E,
                                                reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}

extern "C" int moe_expert_ffn_mxfp4(const float* x, const uint8_t* up_codes,
                                    const uint8_t* up_scales, const uint8_t* down_codes,
                                    const uint8_t* down_scales, const int32_t* offsets,
                                    const int32_t* perm_token, const int32_t* union_ids,
                                    const int32_t* union_size, moe_dims d, float* y_perm, void* ws,
                                    size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_mxfp4_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!x || !up_codes || !up_scales || !down_codes || !down_scales || !y_perm || !ws)
    return MOE_ERR_INVALID;
  st = check_ffn_common(d, offsets, perm_token, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(up_codes) || !aligned4(up_scales) || !aligned16(down_codes) ||
      !aligned4(down_scales) || !aligned16(y_perm) || !aligned16(ws))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  st = moe_expert_ffn_mxfp4_up(x, up_codes, up_scales, offsets, perm_token, union_ids, union_size,
                               d, ws, ws_bytes, stream);
  if (st != MOE_OK) return st;
  return moe_expert_ffn_mxfp4_down(ws, down_codes, down_scales, offsets, perm_token, union_ids,
                                   union_size, d, ws_bytes, y_perm, stream);
}

extern "C" int moe_expert_ffn_mxfp4_up_routed(const float* x, const uint8_t* up_codes,
                                              const uint8_t* up_scales, const int32_t* topk_ids,
                                              moe_dims d, int32_t* counts, int32_t* offsets,
                                              int32_t* perm_token, int32_t* pair_pos,
                                              int32_t* union_ids, int32_t* union_size, void* ws,
                                              size_t ws_bytes, void* stream) {
  using namespace eldr_host;
  int st = check_mxfp4_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0 || d.T > 64) {
    st = moe_bucket(topk_ids, d, counts, offsets, perm_token, pair_pos, union_ids, union_size,
                    stream);
    if (st != MOE_OK || d.T == 0) return st;
    return moe_expert_ffn_mxfp4_up(x, up_codes, up_scales, offsets, perm_token, union_ids,
                                   union_size, d, ws, ws_bytes, stream);
  }
  if (!x || !up_codes || !up_scales || !ws) return MOE_ERR_INVALID;
  st = check_routed(d, topk_ids, counts, offsets, perm_token, pair_pos, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(up_codes) || !aligned4(up_scales) || !aligned16(ws))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs up{reinterpret_cast<const uint4*>(x), nullptr, offsets, perm_token,
                   union_ids + d.E, union_size, ws, d.I, d.H, 0, d.E,
                   reinterpret_cast<const eldr::u32x4*>(up_codes),
                   reinterpret_cast<const uint32_t*>(up_scales),
                   topk_ids, d.T, d.K, counts, offsets, perm_token, pair_pos, union_ids,
                   union_size};
  up.tiles = eldr::ffn_tiles<eldr::kUp, eldr::kMxfp4>(d);
  eldr::launch_ffn_routed<eldr::kMxfp4>(up, d.T, d.E, reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}

// ---- fused launches: buckets, up and down projections in one launch ---------

extern "C" size_t moe_ffn_sync_bytes(moe_dims d) {
  if (eldr_host::check_dims(d) != MOE_OK) return 0;
  return (size_t)(eldr::kSyncStride * d.E + 1) * 4;
}

extern "C" int moe_expert_ffn_routed(const float* x, const uint16_t* w13, const uint16_t* w2,
                                     const int32_t* topk_ids, moe_dims d, int32_t* counts,
                                     int32_t* offsets, int32_t* perm_token, int32_t* pair_pos,
                                     int32_t* union_ids, int32_t* union_size, float* y_perm,
                                     void* ws, size_t ws_bytes, int32_t* sync, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (!sync) return MOE_ERR_INVALID;
  if (!aligned4(sync)) return MOE_ERR_UNSUPPORTED;
  if (d.T == 0 || d.T > 64) {
    // nothing to multiply (moe_bucket writes the empty buckets), or too many
    // tokens for the in-kernel buckets: the separate calls
    st = moe_bucket(topk_ids, d, counts, offsets, perm_token, pair_pos, union_ids, union_size,
                    stream);
    if (st != MOE_OK || d.T == 0) return st;
    return moe_expert_ffn(x, w13, w2, offsets, perm_token, union_ids, union_size, d, y_perm, ws,
                          ws_bytes, stream);
  }
  if (!x || !w13 || !w2 || !y_perm || !ws) return MOE_ERR_INVALID;
  st = check_routed(d, topk_ids, counts, offsets, perm_token, pair_pos, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(w13) || !aligned16(w2) || !aligned16(y_perm) || !aligned128(ws))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs up{reinterpret_cast<const uint4*>(x), w13, offsets, perm_token, union_ids + d.E,
                   union_size, ws, d.I, d.H, 0, d.E, nullptr, nullptr,
                   topk_ids, d.T, d.K, counts, offsets, perm_token, pair_pos, union_ids,
                   union_size};
  up.tiles = eldr::ffn_tiles<eldr::kUp, eldr::kBf16>(d);
  eldr::FfnArgs dn{reinterpret_cast<const uint4*>(ws), w2, offsets, perm_token, union_ids + d.E,
                   union_size, y_perm, d.H, d.I, 0, d.E, nullptr, nullptr};
  dn.tiles = eldr::ffn_tiles<eldr::kDown, eldr::kBf16>(d);
  eldr::launch_ffn_fused<eldr::kBf16>(up, dn, sync, d.T, d.E, reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}

extern "C" int moe_expert_ffn_mxfp4_routed(const float* x, const uint8_t* up_codes,
                                           const uint8_t* up_scales, const uint8_t* down_codes,
                                           const uint8_t* down_scales, const int32_t* topk_ids,
                                           moe_dims d, int32_t* counts, int32_t* offsets,
                                           int32_t* perm_token, int32_t* pair_pos,
                                           int32_t* union_ids, int32_t* union_size, float* y_perm,
                                           void* ws, size_t ws_bytes, int32_t* sync,
                                           void* stream) {
  using namespace eldr_host;
  int st = check_mxfp4_dims(d);
  if (st != MOE_OK) return st;
  if (!sync) return MOE_ERR_INVALID;
  if (!aligned4(sync)) return MOE_ERR_UNSUPPORTED;
  if (d.T == 0 || d.T > 64) {
    st = moe_bucket(topk_ids, d, counts, offsets, perm_token, pair_pos, union_ids, union_size,
                    stream);
    if (st != MOE_OK || d.T == 0) return st;
    return moe_expert_ffn_mxfp4(x, up_codes, up_scales, down_codes, down_scales, offsets,
                                perm_token, union_ids, union_size, d, y_perm, ws, ws_bytes, stream);
  }
  if (!x || !up_codes || !up_scales || !down_codes || !down_scales || !y_perm || !ws)
    return MOE_ERR_INVALID;
  st = check_routed(d, topk_ids, counts, offsets, perm_token, pair_pos, union_ids, union_size);
  if (st != MOE_OK) return st;
  if (!aligned16(x) || !aligned16(up_codes) || !aligned4(up_scales) || !aligned16(down_codes) ||
      !aligned4(down_scales) || !aligned16(y_perm) || !aligned128(ws))
    return MOE_ERR_UNSUPPORTED;
  if (ws_bytes < moe_ffn_workspace_bytes(d)) return MOE_ERR_WORKSPACE;
  eldr::FfnArgs up{reinterpret_cast<const uint4*>(x), nullptr, offsets, perm_token,
                   union_ids + d.E, union_size, ws, d.I, d.H, 0, d.E,
                   reinterpret_cast<const eldr::u32x4*>(up_codes),
                   reinterpret_cast<const uint32_t*>(up_scales),
                   topk_ids, d.T, d.K, counts, offsets, perm_token, pair_pos, union_ids,
                   union_size};
  up.tiles = eldr::ffn_tiles<eldr::kUp, eldr::kMxfp4>(d);
  eldr::FfnArgs dn{reinterpret_cast<const uint4*>(ws), nullptr, offsets, perm_token,
                   union_ids + d.E, union_size, y_perm, d.H, d.I, 0, d.E,
                   reinterpret_cast<const eldr::u32x4*>(down_codes),
                   reinterpret_cast<const uint32_t*>(down_scales)};
  dn.tiles = eldr::ffn_tiles<eldr::kDown, eldr::kMxfp4>(d);
  eldr::launch_ffn_fused<eldr::kMxfp4>(up, dn, sync, d.T, d.E,
                                       reinterpret_cast<hipStream_t>(stream));
  return launch_status();
}
