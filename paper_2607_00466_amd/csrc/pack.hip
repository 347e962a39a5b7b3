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

// ---- MXFP4 ---------------------------------------------------------------------
//
// The MXFP4 FFN reads, per wave and ring slot, two 16-row tiles over two
// k-steps (64 values along the reduction axis) with one 16-byte load per
// lane: lane l takes row l % 16 of each tile and the 8 values starting at
// 8 * (l / 16) of each k-step, whose FP4 codes are 4 consecutive bytes of the
// row.  Its 16 bytes are (tile 0, step 0), (tile 0, step 1), (tile 1, step
// 0), (tile 1, step 1).  The 16 rows' E8M0 scales of the slot follow the same
// order, one dword per row.  Up pairs W1 and W3 rows of a 16-row band; down
// pairs the two 16-row halves of a 32-row band of W2.

namespace eldr {

// One thread moves one lane piece (16 bytes of codes); the threads of lanes
// 0 .. 15 also move their row's scale dword.  p enumerates the packed codes
// as ((band * nslot) + slot) * 64 + lane over all bands of all experts.
__global__ __launch_bounds__(256) void pack_mxfp4_kernel(
    const uint32_t* __restrict__ ca, const uint32_t* __restrict__ cb,
    const uint8_t* __restrict__ sa, const uint8_t* __restrict__ sb, int64_t pieces, int K,
    int band_rows, u32x4* __restrict__ dq, uint32_t* __restrict__ ds) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= pieces) return;
  const int lane = (int)(p & 63);
  const int64_t bs = p >> 6;  // band * nslot + slot
  const int nslot = K / 64;
  const int slot = (int)(bs % nslot);
  const int64_t band = bs / nslot;
  const int r = lane & 15;
  const int g = lane >> 4;
  // source rows of the two tiles, in the flattened [E * R] row order
  const int64_t row0 = band * band_rows + r;
  const int64_t row1 = band_rows == 32 ? row0 + 16 : row0;
  const uint32_t* c1 = band_rows == 32 ? ca : cb;
  const uint8_t* s1 = band_rows == 32 ? sa : sb;
  const int64_t words = K / 8;  // code dwords per row
  const int k0 = 2 * slot;      // first k-step of the slot
  u32x4 v;
  v.x = ca[row0 * words + 4 * k0 + g];
  v.y = ca[row0 * words + 4 * (k0 + 1) + g];
  v.z = c1[row1 * words + 4 * k0 + g];
  v.w = c1[row1 * words + 4 * (k0 + 1) + g];
  dq[p] = v;
  if (lane < 16) {
    const int64_t nb = K / 32;  // scales per row
    const uint32_t b0 = sa[row0 * nb + k0];
    const uint32_t b1 = sa[row0 * nb + k0 + 1];
    const uint32_t b2 = s1[row1 * nb + k0];
    const uint32_t b3 = s1[row1 * nb + k0 + 1];
    ds[bs * 16 + r] = b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
  }
}

}  // namespace eldr

namespace {

int pack_mxfp4(const uint8_t* ca, const uint8_t* sa, const uint8_t* cb, const uint8_t* sb,
               int32_t E, int32_t R, int32_t K, int band_rows, uint8_t* codes, uint8_t* scales,
               void* stream) {
  using namespace eldr_host;
  if (E < 0 || R < 0 || K < 0) return MOE_ERR_INVALID;
  if (R % band_rows != 0 || K % 64 != 0) return MOE_ERR_UNSUPPORTED;
  const int64_t pieces = (int64_t)E * (R / band_rows) * K;  // 64 lanes per slot, K / 64 slots
  if (pieces == 0) return MOE_OK;
  if (!ca || !sa || !cb || !sb || !codes || !scales) return MOE_ERR_INVALID;
  if (!aligned4(ca) || !aligned4(cb) || !aligned16(codes) || !aligned4(scales))
    return MOE_ERR_UNSUPPORTED;
  if (codes == ca || codes == cb || scales == sa || scales == sb) return MOE_ERR_INVALID;
  const int64_t blocks = (pieces + 255) / 256;
  if (blocks > 0x7fffffffLL) return MOE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(eldr::pack_mxfp4_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), reinterpret_cast<const uint32_t*>(ca),
                     reinterpret_cast<const uint32_t*>(cb), sa, sb, pieces, K, band_rows,
                     reinterpret_cast<eldr::u32x4*>(codes), reinterpret_cast<uint32_t*>(scales));
  return launch_status();
}

}  // namespace

extern "C" int moe_pack_mxfp4_up(const uint8_t* w1_codes, const uint8_t* w1_scales,
                                 const uint8_t* w3_codes, const uint8_t* w3_scales, int32_t E,
                                 int32_t I, int32_t H, uint8_t* codes, uint8_t* scales,
                                 void* stream) {
  return pack_mxfp4(w1_codes, w1_scales, w3_codes, w3_scales, E, I, H, 16, codes, scales, stream);
}

extern "C" int moe_pack_mxfp4_down(const uint8_t* w2_codes, const uint8_t* w2_scales, int32_t E,
                                   int32_t H, int32_t I, uint8_t* codes, uint8_t* scales,
                                   void* stream) {
  return pack_mxfp4(w2_codes, w2_scales, w2_codes, w2_scales, E, H, I, 32, codes, scales, stream);
}
