// Internal helpers shared by the gfx950 kernels of libeldr_moe.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "eldr_moe.h"

namespace eldr {

constexpr int kWave = 64;    // CDNA wavefront width
constexpr int kNumXcd = 8;   // MI355X: 8 XCDs, workgroups dispatched round-robin over them

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
// Native 128-bit vector (HIP's uint4 is a struct the optimiser cannot always
// keep in registers when it is copied whole).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// fp32 -> bf16 bit pattern, round to nearest even (inputs are finite; a NaN
// keeps a quiet-NaN pattern).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Split v into hi + lo, both bf16: hi = rne(v), lo = rne(v - hi).  v - hi is
// exact in fp32, so hi + lo carries about 16 significant bits of v.
__device__ __forceinline__ void split_bf16(float v, uint32_t& hi, uint32_t& lo) {
  hi = f32_to_bf16_bits(v);
  lo = f32_to_bf16_bits(v - bf16_bits_to_f32(hi));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// 16x16x32 bf16 MFMA with fp32 accumulation.  A lane supplies 8 k-values of
// one row of A (row = lane % 16) and 8 k-values of one column of B
// (column = lane % 16), the k-set chosen by lane / 16 identically for A and
// B; the result lane holds D[4 * (lane / 16) + i][lane % 16], i = 0..3.
__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

}  // namespace eldr

// Host-side helpers.
namespace eldr_host {

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
inline bool aligned128(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 127u) == 0; }

// Basic validation of the dims every call shares.
inline int check_dims(const moe_dims& d) {
  if (d.T < 0 || d.H <= 0 || d.E <= 0 || d.K <= 0 || d.I <= 0) return MOE_ERR_INVALID;
  if (d.K > d.E) return MOE_ERR_INVALID;
  if (d.E > MOE_MAX_E || d.K > MOE_MAX_K || d.T > MOE_MAX_T || d.H > MOE_MAX_H || d.I > MOE_MAX_I)
    return MOE_ERR_UNSUPPORTED;
  if (d.H % 32 != 0 || d.I % 32 != 0) return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

inline int launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

}  // namespace eldr_host
