// moe_combine: out[t, :] = sum_j topk_w[t, j] * y_perm[pair_pos[t, j], :],
// j ascending, one fp32 fused multiply-add chain per element (deterministic,
// no atomics).  Plus the library's status strings and ABI version.
#include "common.hpp"

namespace eldr {

constexpr int kCombineThreads = 256;

__global__ __launch_bounds__(kCombineThreads) void combine_kernel(
    const float* __restrict__ y, const int32_t* __restrict__ pair_pos,
    const float* __restrict__ w, int T, int H, int K, float* __restrict__ out) {
  const int t = blockIdx.y;
  const int h4 = blockIdx.x * kCombineThreads + threadIdx.x;
  if (h4 * 4 >= H) return;
  const int P = T * K;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < K; ++j) {
    const int p = pair_pos[t * K + j];
    if (p < 0 || p >= P) continue;
    const float wj = w[t * K + j];
    const float4 v = reinterpret_cast<const float4*>(y + (size_t)p * H)[h4];
    acc.x = fmaf(wj, v.x, acc.x);
    acc.y = fmaf(wj, v.y, acc.y);
    acc.z = fmaf(wj, v.z, acc.z);
    acc.w = fmaf(wj, v.w, acc.w);
  }
  reinterpret_cast<float4*>(out + (size_t)t * H)[h4] = acc;
}

}  // namespace eldr

extern "C" int moe_combine(const float* y_perm, const int32_t* pair_pos, const float* topk_w,
                           moe_dims d, float* out, void* stream) {
  using namespace eldr_host;
  int st = check_dims(d);
  if (st != MOE_OK) return st;
  if (d.T == 0) return MOE_OK;
  if (!y_perm || !pair_pos || !topk_w || !out) return MOE_ERR_INVALID;
  if (!aligned16(y_perm) || !aligned16(out) || !aligned4(pair_pos) || !aligned4(topk_w))
    return MOE_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int h4 = d.H / 4;
  dim3 grid((h4 + eldr::kCombineThreads - 1) / eldr::kCombineThreads, d.T);
  hipLaunchKernelGGL(eldr::combine_kernel, grid, dim3(eldr::kCombineThreads), 0, s, y_perm,
                     pair_pos, topk_w, d.T, d.H, d.K, out);
  return launch_status();
}

extern "C" const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK:
      return "MOE_OK";
    case MOE_ERR_INVALID:
      return "MOE_ERR_INVALID: null pointer or inconsistent dimensions";
    case MOE_ERR_UNSUPPORTED:
      return "MOE_ERR_UNSUPPORTED: shape outside the library limits or misaligned pointer";
    case MOE_ERR_WORKSPACE:
      return "MOE_ERR_WORKSPACE: workspace smaller than required";
    case MOE_ERR_HIP:
      return "MOE_ERR_HIP: the HIP runtime rejected a launch";
    default:
      return "unknown status";
  }
}

extern "C" int moe_abi_version(void) { return 1; }
