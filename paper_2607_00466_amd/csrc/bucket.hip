// moe_bucket: per-expert buckets of (token, expert) pairs and the union of
// distinct experts, in one workgroup.
//
// Each expert gets a bitmap over tokens in LDS (bit t set when token t picked
// it).  A slot's rank inside its bucket is the number of set bits below t,
// so buckets list their tokens in ascending order without any sort, and the
// result does not depend on the order in which threads ran.  The union is
// listed twice: in ascending id, then in dispatch order -- experts with more
// 16-token tiles (the expert FFN's unit of work per item) first, equal ones
// by ascending id -- so the FFN starts its longest items first while batches
// of small buckets stream the experts in address order.  An expert's
// dispatch position is the number of experts with a larger (tiles, -id) key.
#include "common.hpp"

namespace eldr {

constexpr int kBucketThreads = 1024;
constexpr int kBucketMaxWords = 16384;  // E * ceil(T / 32) limit (64 KiB of bitmaps)
constexpr int kOrderTokens = 16;        // union order: buckets compared in tiles of 16 tokens

__global__ __launch_bounds__(kBucketThreads) void bucket_kernel(
    const int32_t* __restrict__ ids, int T, int E, int K, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ perm_token, int32_t* __restrict__ pair_pos,
    int32_t* __restrict__ union_ids, int32_t* __restrict__ union_size) {
  extern __shared__ uint32_t smem[];
  // union order keys, larger first: 16-token tiles (<= 256) above 255 - e
  // (e < 256); 0 past E, below every expert with tokens
  __shared__ __attribute__((aligned(16))) int key_s[MOE_MAX_E];
  __shared__ int bad;
  __shared__ int total_pairs, total_union;
  const int W = (T + 31) / 32;
  const int EW = E * W;
  uint32_t* mask = smem;                                          // [E][W] token bitmaps
  uint16_t* pre = reinterpret_cast<uint16_t*>(mask + EW);         // [E][W] bits before word w
  int32_t* cnt = reinterpret_cast<int32_t*>(pre + ((EW + 1) & ~1));  // [E]
  int32_t* off = cnt + E;                                         // [E]
  int32_t* usc = off + E;                                         // [E] position, ascending union
  int32_t* rnk = usc + E;                                         // [E] position, dispatch order
  const int tid = threadIdx.x;
  const int P = T * K;

  for (int i = tid; i < EW; i += kBucketThreads) mask[i] = 0u;
  if (tid == 0) bad = 0;
  __syncthreads();

  for (int p = tid; p < P; p += kBucketThreads) {
    const int t = p / K;
    const int e = ids[p];
    if (e < 0 || e >= E) {
      bad = 1;
      continue;
    }
    const uint32_t bit = 1u << (t & 31);
    const uint32_t old = atomicOr(&mask[e * W + (t >> 5)], bit);
    if (old & bit) bad = 1;  // the same expert twice for one token
  }
  __syncthreads();

  for (int e = tid; e < E; e += kBucketThreads) {
    int run = 0;
    for (int w = 0; w < W; ++w) {
      pre[e * W + w] = (uint16_t)run;
      run += __popc(mask[e * W + w]);
    }
    cnt[e] = run;
    key_s[e] = (((run + kOrderTokens - 1) / kOrderTokens) << 8) | (MOE_MAX_E - 1 - e);
  }
  for (int e = E + tid; e < MOE_MAX_E; e += kBucketThreads) key_s[e] = 0;
  __syncthreads();

  // Exclusive scans of counts and of (counts > 0) over E <= 256 experts by
  // wave 0: 4 consecutive experts per lane, then a shuffle scan over lanes.
  // Meanwhile the other waves rank each expert: R adjacent threads split the
  // keys (in runs of 4, read 16 bytes at a time) and sum their counts.
  static_assert(kBucketThreads >= kWave + 2 * MOE_MAX_E, "two ranking threads an expert");
  if (tid >= kWave) {
    const int R = E <= (kBucketThreads - kWave) / 4 ? 4 : 2;
    const int q = tid - kWave;
    const int e = q / R;
    const int quads = (E + 3) / 4;
    const int per = (quads + R - 1) / R;
    const int q0 = (q % R) * per;
    const int q1 = min(quads, q0 + per);
    int above = 0;
    if (e < E) {
      const int key = key_s[e];
      const int4* k4 = reinterpret_cast<const int4*>(key_s);
      for (int i = q0; i < q1; ++i) {
        const int4 k = k4[i];
        above += (k.x > key) + (k.y > key) + (k.z > key) + (k.w > key);
      }
    }
    above += __shfl_xor(above, 1);
    if (R == 4) above += __shfl_xor(above, 2);
    if (e < E && q % R == 0) rnk[e] = above;
  } else {
    const int lane = tid;
    int c[4], f[4], sc = 0, sf = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane * 4 + i;
      c[i] = e < E ? cnt[e] : 0;
      f[i] = c[i] > 0 ? 1 : 0;
      sc += c[i];
      sf += f[i];
    }
    int ic = sc, jf = sf;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int nc = __shfl_up(ic, o);
      const int nf = __shfl_up(jf, o);
      if (lane >= o) {
        ic += nc;
        jf += nf;
      }
    }
    int bc = ic - sc, bf = jf - sf;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane * 4 + i;
      if (e < E) {
        off[e] = bc;
        usc[e] = bf;
      }
      bc += c[i];
      bf += f[i];
    }
    if (lane == kWave - 1) {
      total_pairs = ic;
      total_union = jf;
    }
  }
  __syncthreads();

  const bool ok = (bad == 0) && (total_pairs == P);
  if (ok) {
    for (int p = tid; p < P; p += kBucketThreads) {
      const int t = p / K;
      const int e = ids[p];
      const int w = t >> 5;
      const uint32_t below = mask[e * W + w] & ((1u << (t & 31)) - 1u);
      const int slot = off[e] + pre[e * W + w] + __popc(below);
      perm_token[slot] = t;
      pair_pos[p] = slot;
    }
  }
  const int U = total_union;
  for (int e = tid; e < E; e += kBucketThreads) {
    counts[e] = cnt[e];
    offsets[e] = off[e];
    if (cnt[e] > 0) {
      union_ids[usc[e]] = e;
      union_ids[E + rnk[e]] = e;
    }
  }
  for (int u = tid; u < E; u += kBucketThreads)
    if (u >= U) {
      union_ids[u] = -1;
      union_ids[E + u] = -1;
    }
  if (tid == 0) {
    offsets[E] = total_pairs;
    *union_size = ok ? U : -1;
  }
}

size_t bucket_lds_bytes(int T, int E) {
  const size_t W = (size_t)(T + 31) / 32;
  const size_t EW = (size_t)E * W;
  return EW * 4 + ((EW + 1) & ~(size_t)1) * 2 + (size_t)E * 4 * 4;
}

}  // namespace eldr

extern "C" int moe_bucket(const int32_t* topk_ids, moe_dims d, int32_t* counts, int32_t* offsets,
                          int32_t* perm_token, int32_t* pair_pos, int32_t* union_ids,
                          int32_t* union_size, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (!counts || !offsets || !union_ids || !union_size) return MOE_ERR_INVALID;
  if (d.T > 0 && (!topk_ids || !perm_token || !pair_pos)) return MOE_ERR_INVALID;
  if (!aligned4(topk_ids) || !aligned4(counts) || !aligned4(offsets) || !aligned4(perm_token) ||
      !aligned4(pair_pos) || !aligned4(union_ids) || !aligned4(union_size))
    return MOE_ERR_UNSUPPORTED;
  if ((long long)d.E * ((d.T + 31) / 32) > eldr::kBucketMaxWords) return MOE_ERR_UNSUPPORTED;
  const size_t lds = eldr::bucket_lds_bytes(d.T, d.E);
  // Bitmaps above 64 KiB (E * ceil(T / 32) > 8192 words) need the kernel's
  // dynamic LDS limit raised, on the current device, before the launch; the
  // call is cheap and shapes that need it are prefill-sized, so it is made on
  // every such call rather than cached.
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(reinterpret_cast<const void*>(eldr::bucket_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return MOE_ERR_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(eldr::bucket_kernel, dim3(1), dim3(eldr::kBucketThreads), lds, s, topk_ids,
                     d.T, d.E, d.K, counts, offsets, perm_token, pair_pos, union_ids, union_size);
  return launch_status();
}
