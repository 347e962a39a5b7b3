// moe_pack_up_weights / moe_pack_down_weights: lay the bf16 expert weights out
// as the expert FFN streams them, once, off the decode path.
//
// The FFN reads each 16-row x 32-column tile of a weight matrix as one MFMA A
// operand: lane l takes row (l % 16) and the 8 columns starting at
// 8 * (l / 16); packed, the 64 lane pieces of one tile are one contiguous
// 1 KB fragment in lane order.  A workgroup item covers a band of rows (up:
// 64 rows of W1 and the same 64 rows of W3; down: 128 rows of W2), one wave
// per 16 rows of W1/W3 or per 32 rows of W2, each wave reading two fragments
// per k-step.  The packed band puts, for each k-step, the fragments of all
// its waves side by side -- wave by wave, the wave's two fragments in order
// -- and the k-steps one after the other, so a workgroup streams one
// contiguous stretch of memory per item.  On MI355X that streams markedly
// faster than the same bytes as one stream per wave and matrix (a probe of
// the access pattern: 6.8-6.9 against 4.7-5.2 TB/s at 512-1536 items).
// Packing permutes bf16 values; it changes no value and no byte count.
#include "common.hpp"

namespace eldr {

// One thread moves one 16-byte piece (8 bf16): piece index p enumerates the
// packed array in order.  up: fragment f of wave w is W1 (f = 0) or W3 (f = 1)
// rows 64 b + 16 w + (l % 16); down: rows 128 b + 32 w + 16 f + (l % 16) of
// W2.  A last band with fewer rows holds only its waves' fragments.
__global__ __launch_bounds__(256) void pack_band_kernel(const u32x4* __restrict__ a,
                                                        const u32x4* __restrict__ b,
                                                        int64_t pieces, int R, int K, int up,
                                                        u32x4* __restrict__ dst) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= pieces) return;
  const int lane = (int)(p & 63);
  const int64_t frag = p >> 6;
  const int nk = K / 32;
  const int band_rows = up ? 64 : 128;
  const int wave_rows = up ? 16 : 32;
  const int64_t per_expert = (int64_t)(up ? 2 : 1) * (R / 16) * nk;  // fragments per expert
  const int64_t e = frag / per_expert;
  const int64_t q = frag - e * per_expert;
  const int64_t per_band = 8LL * nk;  // fragments of a full band
  const int band = (int)(q / per_band);
  const int64_t r = q - (int64_t)band * per_band;
  const int rows_b = min(band_rows, R - band * band_rows);
  const int frags_step = 2 * (rows_b / wave_rows);  // fragments of one k-step of this band
  const int step = (int)(r / frags_step);
  const int f2 = (int)(r - (int64_t)step * frags_step);
  const int w = f2 >> 1;
  const int f = f2 & 1;
  const int row = band * band_rows + w * wave_rows + (up ? 0 : 16 * f) + (lane & 15);
  const u32x4* src = (up && f) ? b : a;
  const int64_t col = (int64_t)step * 32 + 8 * (lane >> 4);
  dst[p] = src[((e * R + row) * K + col) / 8];
}

static int pack_band(const uint16_t* a, const uint16_t* b, int32_t E, int32_t R, int32_t K, int up,
                     uint16_t* dst, void* stream) {
  using namespace eldr_host;
  if (E < 0 || R < 0 || K < 0) return MOE_ERR_INVALID;
  if (R % 32 != 0 || K % 32 != 0) return MOE_ERR_UNSUPPORTED;
  const int64_t pieces = (int64_t)(up ? 2 : 1) * E * R * K / 8;
  if (pieces == 0) return MOE_OK;
  if (!a || !b || !dst) return MOE_ERR_INVALID;
  if (!aligned16(a) || !aligned16(b) || !aligned16(dst)) return MOE_ERR_UNSUPPORTED;
  if (a == dst || b == dst) return MOE_ERR_INVALID;
  const int64_t blocks = (pieces + 255) / 256;
  if (blocks > 0x7fffffffLL) return MOE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(pack_band_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), reinterpret_cast<const u32x4*>(a),
                     reinterpret_cast<const u32x4*>(b), pieces, R, K, up,
                     reinterpret_cast<u32x4*>(dst));
  return launch_status();
}

}  // namespace eldr

extern "C" int moe_pack_up_weights(const uint16_t* w1, const uint16_t* w3, int32_t E, int32_t I,
                                   int32_t H, uint16_t* dst, void* stream) {
  return eldr::pack_band(w1, w3, E, I, H, 1, dst, stream);
}

extern "C" int moe_pack_down_weights(const uint16_t* w2, int32_t E, int32_t H, int32_t I,
                                     uint16_t* dst, void* stream) {
  return eldr::pack_band(w2, w2, E, H, I, 0, dst, stream);
}

// ---- MXFP4 ---------------------------------------------------------------------
//
// The MXFP4 FFN reads, per wave and ring slot, two 16-row tiles over two
// k-steps (64 values along the reduction axis) with one 16-byte load per
// lane: lane l takes row l % 16 of each tile and the 8 values starting at
// 8 * (l / 16) of each k-step, whose FP4 codes are 4 consecutive bytes of the
// row.  Its 16 bytes are (tile 0, step 0), (tile 0, step 1), (tile 1, step
// 0), (tile 1, step 1).  The 16 rows' E8M0 scales of the slot follow the same
// order, one dword per row.  Up pairs W1 and W3 rows of a 16-row wave band;
// down pairs the two 16-row halves of a 32-row wave band of W2.  The four
// wave bands of a workgroup band lie side by side slot by slot, as for bf16.

namespace eldr {

// One thread moves one lane piece (16 bytes of codes); the threads of lanes
// 0 .. 15 also move their row's scale dword.  p enumerates the packed codes
// in their packed order: per expert, workgroup band of 4 wave bands (the last
// one may hold fewer), slot, wave band within it, lane.  A wave band is 16
// rows (up) or 32 rows (down), so a workgroup item's codes are one
// contiguous stretch and its scales another.
__global__ __launch_bounds__(256) void pack_mxfp4_kernel(
    const uint32_t* __restrict__ ca, const uint32_t* __restrict__ cb,
    const uint8_t* __restrict__ sa, const uint8_t* __restrict__ sb, int64_t pieces, int R, int K,
    int band_rows, u32x4* __restrict__ dq, uint32_t* __restrict__ ds) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= pieces) return;
  const int lane = (int)(p & 63);
  const int64_t q = p >> 6;  // (slot, wave band) unit in packed order
  const int nslot = K / 64;
  const int nwb = R / band_rows;  // wave bands per expert
  const int64_t e = q / ((int64_t)nwb * nslot);
  const int64_t rq = q - e * nwb * nslot;
  const int j = (int)(rq / (4 * nslot));          // workgroup band
  const int r2 = (int)(rq - (int64_t)j * 4 * nslot);
  const int wb = min(4, nwb - 4 * j);             // wave bands in this workgroup band
  const int slot = r2 / wb;
  const int64_t band = e * nwb + 4 * j + (r2 - slot * wb);  // wave band in [E * R / band_rows]
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
    ds[q * 16 + r] = b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
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
                     reinterpret_cast<const uint32_t*>(cb), sa, sb, pieces, R, K, band_rows,
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
