// moe_pack_weights: lay expert weights out as MFMA fragments, once, off the
// decode path.
//
// The expert FFN reads each 16-row x 32-column tile of a weight matrix as one
// MFMA A operand: lane l takes row (l % 16) and the 8 columns starting at
// 8 * (l / 16).  In the row-major [out, in] layout those 64 lane pieces are 16
// rows apart; packed, the 64 pieces of one tile are one contiguous 1 KB block
// in lane order, and a 16-row band's tiles follow each other along the
// reduction axis, so every load instruction of the FFN reads 1 KB of
// consecutive memory.  Packing permutes bf16 values; it changes no value and
// no byte count.
#include "common.hpp"

namespace eldr {

// One thread moves one 16-byte piece (8 bf16): piece index p enumerates the
// packed array in order, and its source is computed from (tile, lane).
__global__ __launch_bounds__(256) void pack_kernel(const u32x4* __restrict__ src, int64_t pieces,
                                                   int R, int K, u32x4* __restrict__ dst) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= pieces) return;
  const int lane = (int)(p & 63);
  const int64_t tile = p >> 6;             // ((e * R/16) + band) * K/32 + step
  const int nk = K / 32;
  const int step = (int)(tile % nk);
  const int64_t band = tile / nk;          // e * R/16 + row band
  const int64_t row = band * 16 + (lane & 15);
  const int64_t col = (int64_t)step * 32 + 8 * (lane >> 4);
  dst[p] = src[(row * K + col) / 8];
}

}  // namespace eldr

extern "C" int moe_pack_weights(const uint16_t* src, int32_t E, int32_t R, int32_t K,
                                uint16_t* dst, void* stream) {
  using namespace eldr_host;
  if (E < 0 || R < 0 || K < 0) return MOE_ERR_INVALID;
  if (R % 16 != 0 || K % 32 != 0) return MOE_ERR_UNSUPPORTED;
  const int64_t pieces = (int64_t)E * R * K / 8;
  if (pieces == 0) return MOE_OK;
  if (!src || !dst) return MOE_ERR_INVALID;
  if (!aligned16(src) || !aligned16(dst)) return MOE_ERR_UNSUPPORTED;
  if (src == dst) return MOE_ERR_INVALID;
  const int64_t blocks = (pieces + 255) / 256;
  if (blocks > 0x7fffffffLL) return MOE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(eldr::pack_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), reinterpret_cast<const eldr::u32x4*>(src),
                     pieces, R, K, reinterpret_cast<eldr::u32x4*>(dst));
  return launch_status();
}
