// Gate-weighted combine (the last step of the MoE layer): y_t = sum_j g_tj o_tj in rank order,
// plus the shared expert's output with weight 1.  A fixed summation order keeps paged and
// resident runs bit-identical.  HBM-bound: reads T (k + shared) d floats, writes T d floats.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace wisp {
namespace {

__global__ void __launch_bounds__(256) combine_kernel(int k, int d, int has_shared, const float* __restrict__ w,
                                                      const float4* __restrict__ buf, float4* __restrict__ y) {
  const int t = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;  // float4 column
  const int d4 = d / 4;
  if (c >= d4) return;
  const int rows = k + 1;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < k; ++j) {
    const float g = w[t * k + j];
    const float4 o = buf[static_cast<size_t>(t * rows + j) * d4 + c];
    acc.x = fmaf(g, o.x, acc.x); acc.y = fmaf(g, o.y, acc.y);
    acc.z = fmaf(g, o.z, acc.z); acc.w = fmaf(g, o.w, acc.w);
  }
  if (has_shared) {
    const float4 o = buf[static_cast<size_t>(t * rows + k) * d4 + c];
    acc.x += o.x; acc.y += o.y; acc.z += o.z; acc.w += o.w;
  }
  y[static_cast<size_t>(t) * d4 + c] = acc;
}

}  // namespace

hipError_t launch_combine(int T, int k, int d, int has_shared, const float* w, const float* buf, float* y,
                          hipStream_t st, const LaunchTiming& tm) {
  if (T <= 0) return hipSuccess;
  if (d % 4 != 0) return hipErrorInvalidValue;
  dim3 grid((d / 4 + 255) / 256, T), block(256);
  hipExtLaunchKernelGGL(combine_kernel, grid, block, 0, st, tm.start, tm.stop, 0, k, d, has_shared, w,
                        reinterpret_cast<const float4*>(buf), reinterpret_cast<float4*>(y));
  return hipGetLastError();
}

}  // namespace wisp
