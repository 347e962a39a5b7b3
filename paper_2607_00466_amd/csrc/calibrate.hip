// moe_stream_read_probe: a plain streaming read, for reporting the achievable
// HBM read bandwidth beside the peak (a measurement aid, not the MoE path).
// The loads are non-temporal, as the expert FFN's weight loads are: on
// MI355X that streams at about 7.0 TB/s where ordinary loads reach 6.2.
#include "common.hpp"
#include "eldr_calibration.h"

namespace eldr {

constexpr int kProbeThreads = 256;
constexpr int kProbeBlocks = 2048;
constexpr int kProbeDepth = 8;  // 16-byte loads in flight per thread
constexpr uint32_t kProbeMagic = 0x9e3779b9u;

__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const u32x4* __restrict__ buf,
                                                                   int64_t n16,
                                                                   uint32_t* __restrict__ sink) {
  // Workgroup b reads pieces [begin, end) of the buffer, contiguous.
  const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t begin = (int64_t)blockIdx.x * per;
  const int64_t end = begin + per < n16 ? begin + per : n16;
  uint32_t acc = 0;
  constexpr int64_t step = (int64_t)kProbeThreads * kProbeDepth;
  int64_t i = begin + threadIdx.x;
  for (; i + (kProbeDepth - 1) * kProbeThreads < end; i += step) {
    u32x4 v[kProbeDepth];
#pragma unroll
    for (int d = 0; d < kProbeDepth; ++d) v[d] = __builtin_nontemporal_load(&buf[i + d * kProbeThreads]);
#pragma unroll
    for (int d = 0; d < kProbeDepth; ++d) acc ^= v[d].x ^ v[d].y ^ v[d].z ^ v[d].w;
  }
  for (; i < end; i += kProbeThreads) {
    const u32x4 v = __builtin_nontemporal_load(&buf[i]);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == kProbeMagic) sink[0] = acc;
}

}  // namespace eldr

extern "C" int moe_stream_read_probe(const void* buf, size_t bytes, uint32_t* sink, void* stream) {
  using namespace eldr_host;
  if (bytes == 0) return MOE_OK;
  if (!buf || !sink) return MOE_ERR_INVALID;
  if (!aligned16(buf) || !aligned4(sink) || bytes % 16 != 0) return MOE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(eldr::stream_read_kernel, dim3(eldr::kProbeBlocks), dim3(eldr::kProbeThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), reinterpret_cast<const eldr::u32x4*>(buf),
                     (int64_t)(bytes / 16), sink);
  return launch_status();
}
