// The block-granular expert-signature cache (Design, Prefix Cache Coherence):
// capture of a prefill forward's picks into int8 per-block rows, block reset,
// and per-request sums over a block table.
//
// capture: one thread per (layer, token, pick).  Four int8 cells share one
// 32-bit word, so a pick adds 1 << (8 * (cell % 4)) to its word.  A cell
// never exceeds 127 (a block holds at most 127 tokens and a token picks an
// expert at most once per layer), so no carry crosses into the neighbouring
// cell.  A workgroup first sums its picks' increments per word in an LDS hash
// table (its 256 picks are a few tokens of one or two blocks, and popular
// experts repeat), then adds each word's sum with one 32-bit device atomic.
// Integer addition makes the result independent of the order and grouping
// of the picks.
//
// request counts: a workgroup per (request, 1 KB stretch of the [L, E] row).
// Its four waves split the request's blocks, 16 at a time a wave; a lane
// reads 16 cells of each block (one 16-byte load), all 16 blocks' loads in
// flight before the first is used, and keeps 16 int32 sums.  The four waves'
// sums then meet in LDS, and each thread writes four of the stretch's counts.
#include "common.hpp"
#include "eldr_signature.h"

namespace eldr {

constexpr int kSigThreads = 256;

// LDS hash slots of the capture: twice the most distinct words a workgroup
// can touch (one a pick), so a probe always finds its word or a free slot.
constexpr int kCapSlots = 2 * kSigThreads;
constexpr uint64_t kCapFree = ~0ull;

__global__ __launch_bounds__(kSigThreads) void sig_capture_kernel(
    const int32_t* __restrict__ ids, const int32_t* __restrict__ token_block, int64_t picks,
    int T, int K, int layer0, int L, int E, int num_blocks, uint32_t* __restrict__ sig_words,
    int32_t* __restrict__ rejected) {
  __shared__ uint64_t key[kCapSlots];  // word index, or kCapFree
  __shared__ uint32_t sum[kCapSlots];  // summed increments of the word
  for (int i = threadIdx.x; i < kCapSlots; i += kSigThreads) {
    key[i] = kCapFree;
    sum[i] = 0u;
  }
  __syncthreads();
  const int64_t p = (int64_t)blockIdx.x * kSigThreads + threadIdx.x;  // (l * T + t) * K + j
  bool bad = false;
  if (p < picks) {
    const int64_t lt = p / K;
    const int t = (int)(lt % T);
    const int l = (int)(lt / T);
    const int b = token_block[t];
    if (b >= 0) {
      const int e = ids[p];
      if (b >= num_blocks || e < 0 || e >= E) {
        bad = true;
      } else {
        const int64_t cell = ((int64_t)b * L + layer0 + l) * E + e;
        const uint64_t word = (uint64_t)(cell >> 2);
        const uint32_t inc = 1u << (8 * (int)(cell & 3));
        // linear probing from a multiplicative hash of the word
        uint32_t h = ((uint32_t)word ^ (uint32_t)(word >> 32)) * 0x9e3779b1u >> 23;
        for (int probe = 0; probe < kCapSlots; ++probe) {
          const uint64_t k = atomicCAS(reinterpret_cast<unsigned long long*>(&key[h]),
                                       (unsigned long long)kCapFree, (unsigned long long)word);
          if (k == kCapFree || k == word) {
            atomicAdd(&sum[h], inc);
            break;
          }
          h = (h + 1) & (kCapSlots - 1);
        }
      }
    }
  }
  if (rejected) {
    // one atomic per wave that saw a rejected pick
    const uint64_t m = __ballot(bad);
    if (m && (threadIdx.x % kWave) == 0) atomicAdd(rejected, (int)__popcll(m));
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kCapSlots; i += kSigThreads) {
    const uint64_t w = key[i];
    if (w != kCapFree) atomicAdd(&sig_words[w], sum[i]);
  }
}

__global__ __launch_bounds__(kSigThreads) void sig_reset_kernel(const int32_t* __restrict__ blocks,
                                                               int row_words, int num_blocks,
                                                               uint32_t* __restrict__ sig_words) {
  const int b = blocks[blockIdx.y];
  if (b < 0 || b >= num_blocks) return;
  const int w = blockIdx.x * kSigThreads + threadIdx.x;
  if (w < row_words) sig_words[(int64_t)b * row_words + w] = 0u;
}

constexpr int kReqWaves = 4;
constexpr int kReqWords = 4 * kWave;  // row words a workgroup covers: 4 a lane (1 KB)
constexpr int kReqUnroll = 16;        // blocks a wave has in flight

// VEC: every row starts 16-byte aligned and holds a whole number of 16-byte
// pieces (row_words % 4 == 0), so a lane reads its 4 words with one load;
// otherwise word by word, each within the row.
template <bool VEC>
__global__ __launch_bounds__(kReqWaves * kWave) void sig_request_kernel(
    const uint32_t* __restrict__ sig_words, const int32_t* __restrict__ block_table,
    const int32_t* __restrict__ n_blocks, int max_blocks, int row_words, int num_blocks,
    int4* __restrict__ out) {
  __shared__ int4 part[kReqWaves][kWave][4];
  const int r = blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int w0 = blockIdx.x * kReqWords + 4 * lane;  // the lane's first word
  int acc[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) acc[c] = 0;
  // Group g holds blocks [g * 64, g * 64 + 64); wave w takes 16 consecutive
  // ones.  The first group is issued before n is known: its table entries
  // are read up to max_blocks (in the table), so that the table and n arrive
  // together.  Entries past n, and invalid block ids, read block 0's words
  // and add nothing.  An empty cache (num_blocks == 0, sig may be null)
  // contributes nothing and is not read.
  if (num_blocks > 0) {
    const int n = min(max(n_blocks[r], 0), max_blocks);
    const int32_t* table = block_table + (int64_t)r * max_blocks;
    int i0 = wave * kReqUnroll;
    do {
      u32x4 v[kReqUnroll];
#pragma unroll
      for (int k = 0; k < kReqUnroll; ++k) {
        const int i = i0 + k;
        const int b = i < max_blocks ? table[i] : -1;
        const bool ok = i < n && b >= 0 && b < num_blocks;
        const uint32_t* row = sig_words + (int64_t)(ok ? b : 0) * row_words;
        const uint32_t m = ok ? 0xffffffffu : 0u;
        if constexpr (VEC) {
          const u32x4 x = w0 < row_words ? *reinterpret_cast<const u32x4*>(row + w0) : u32x4{0u, 0u, 0u, 0u};
          v[k] = x & m;
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) v[k][q] = (w0 + q < row_words ? row[w0 + q] : 0u) & m;
        }
      }
#pragma unroll
      for (int k = 0; k < kReqUnroll; ++k) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // the four int8 cells of the word, sign-extended (cell 0 is the low byte)
          const uint32_t x = v[k][q];
          acc[4 * q + 0] += (int)(int8_t)(x & 0xffu);
          acc[4 * q + 1] += (int)(int8_t)((x >> 8) & 0xffu);
          acc[4 * q + 2] += (int)(int8_t)((x >> 16) & 0xffu);
          acc[4 * q + 3] += (int)(int8_t)(x >> 24);
        }
      }
      i0 += kReqWaves * kReqUnroll;
    } while (i0 < n);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q)
    part[wave][lane][q] = make_int4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
  __syncthreads();
  // thread t: word 4 * (t / 4) + t % 4 of the stretch, i.e. word blockIdx.x * kReqWords + t
  const int t = threadIdx.x;
  const int w = blockIdx.x * kReqWords + t;
  if (w < row_words) {
    int4 sum = make_int4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < kReqWaves; ++j) {
      const int4 p = part[j][t / 4][t % 4];
      sum.x += p.x;
      sum.y += p.y;
      sum.z += p.z;
      sum.w += p.w;
    }
    out[(int64_t)r * row_words + w] = sum;
  }
}

}  // namespace eldr

namespace {

int check_sig_shape(int32_t L, int32_t E, int32_t num_blocks) {
  if (L <= 0 || E <= 0 || num_blocks < 0) return MOE_ERR_INVALID;
  if (L > MOE_SIG_MAX_LAYERS || E > MOE_MAX_E) return MOE_ERR_UNSUPPORTED;
  if (((int64_t)L * E) % 4 != 0) return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

}  // namespace

extern "C" int moe_sig_capture(const int32_t* ids, const int32_t* token_block, int32_t n_layers,
                               int32_t T, int32_t K, int32_t layer0, int32_t L, int32_t E,
                               int32_t num_blocks, int8_t* sig, int32_t* rejected, void* stream) {
  using namespace eldr_host;
  int st = check_sig_shape(L, E, num_blocks);
  if (st != MOE_OK) return st;
  if (n_layers < 0 || T < 0 || K <= 0 || K > E || layer0 < 0 || layer0 + n_layers > L)
    return MOE_ERR_INVALID;
  if (T > MOE_SIG_MAX_TOKENS) return MOE_ERR_UNSUPPORTED;
  const int64_t picks = (int64_t)n_layers * T * K;
  if (picks == 0 || num_blocks == 0) return MOE_OK;
  if (!ids || !token_block || !sig) return MOE_ERR_INVALID;
  if (!aligned4(ids) || !aligned4(token_block) || !aligned4(sig) || (rejected && !aligned4(rejected)))
    return MOE_ERR_UNSUPPORTED;
  const int64_t blocks = (picks + eldr::kSigThreads - 1) / eldr::kSigThreads;
  if (blocks > 0x7fffffffLL) return MOE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(eldr::sig_capture_kernel, dim3((unsigned)blocks), dim3(eldr::kSigThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), ids, token_block, picks, T, K, layer0,
                     L, E, num_blocks, reinterpret_cast<uint32_t*>(sig), rejected);
  return launch_status();
}

extern "C" int moe_sig_reset(const int32_t* blocks, int32_t n, int32_t L, int32_t E,
                             int32_t num_blocks, int8_t* sig, void* stream) {
  using namespace eldr_host;
  int st = check_sig_shape(L, E, num_blocks);
  if (st != MOE_OK) return st;
  if (n < 0) return MOE_ERR_INVALID;
  if (n == 0 || num_blocks == 0) return MOE_OK;
  if (n > 65535) return MOE_ERR_UNSUPPORTED;
  if (!blocks || !sig) return MOE_ERR_INVALID;
  if (!aligned4(blocks) || !aligned4(sig)) return MOE_ERR_UNSUPPORTED;
  const int row_words = L * E / 4;
  dim3 grid((row_words + eldr::kSigThreads - 1) / eldr::kSigThreads, n);
  hipLaunchKernelGGL(eldr::sig_reset_kernel, grid, dim3(eldr::kSigThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), blocks, row_words, num_blocks,
                     reinterpret_cast<uint32_t*>(sig));
  return launch_status();
}

extern "C" int moe_sig_request_counts(const int8_t* sig, const int32_t* block_table,
                                      const int32_t* n_blocks, int32_t R, int32_t max_blocks,
                                      int32_t L, int32_t E, int32_t num_blocks, int32_t* out,
                                      void* stream) {
  using namespace eldr_host;
  int st = check_sig_shape(L, E, num_blocks);
  if (st != MOE_OK) return st;
  if (R < 0 || max_blocks < 0) return MOE_ERR_INVALID;
  if (R == 0) return MOE_OK;
  if (R > 65535) return MOE_ERR_UNSUPPORTED;
  if (!n_blocks || !out || (max_blocks > 0 && !block_table) || (num_blocks > 0 && !sig))
    return MOE_ERR_INVALID;
  if (!aligned16(out) || !aligned4(n_blocks) || (block_table && !aligned4(block_table)) ||
      (sig && !aligned4(sig)))
    return MOE_ERR_UNSUPPORTED;
  const int row_words = L * E / 4;
  const dim3 grid((row_words + eldr::kReqWords - 1) / eldr::kReqWords, R);
  const dim3 block(eldr::kReqWaves * eldr::kWave);
  const bool vec = row_words % 4 == 0 && (!sig || aligned16(sig));
  if (vec)
    hipLaunchKernelGGL(eldr::sig_request_kernel<true>, grid, block, 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const uint32_t*>(sig), block_table, n_blocks, max_blocks, row_words,
                       num_blocks, reinterpret_cast<int4*>(out));
  else
    hipLaunchKernelGGL(eldr::sig_request_kernel<false>, grid, block, 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const uint32_t*>(sig), block_table, n_blocks, max_blocks, row_words,
                       num_blocks, reinterpret_cast<int4*>(out));
  return launch_status();
}
