// Gate-weighted combine (the last step of the MoE layer): y_t = sum_j g_tj o_tj in rank order,
// plus the shared expert's output with weight 1.  A fixed summation order keeps paged and
// resident runs bit-identical.  HBM-bound: reads T (k + shared) d expert outputs (fp32 from the
// GEMV kernels, bf16 from the grouped GEMMs), writes T d floats.
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

// bf16 expert outputs (8 columns per thread): each value widened exactly to fp32, then the same
// fmaf chain in rank order.
__global__ void __launch_bounds__(256) combine_bf16_kernel(int k, int d, const float* __restrict__ w,
                                                           const uint4* __restrict__ buf, float4* __restrict__ y) {
  const int t = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;  // 8-column group
  const int d8 = d / 8;
  if (c >= d8) return;
  const int rows = k + 1;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < k; ++j) {
    const float g = w[t * k + j];
    const uint4 o = buf[static_cast<size_t>(t * rows + j) * d8 + c];
    const uint32_t q[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] = fmaf(g, __uint_as_float(q[i] << 16), acc[2 * i]);
      acc[2 * i + 1] = fmaf(g, __uint_as_float(q[i] & 0xFFFF0000u), acc[2 * i + 1]);
    }
  }
  y[(static_cast<size_t>(t) * d8 + c) * 2] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  y[(static_cast<size_t>(t) * d8 + c) * 2 + 1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
}

}  // namespace

hipError_t launch_combine_bf16(int T, int k, int d, const float* w, const uint16_t* buf, float* y, hipStream_t st,
                               const LaunchTiming& tm) {
  if (T <= 0) return hipSuccess;
  if (d % 8 != 0) return hipErrorInvalidValue;
  dim3 grid((d / 8 + 255) / 256, T), block(256);
  hipExtLaunchKernelGGL(combine_bf16_kernel, grid, block, 0, st, tm.start, tm.stop, 0, k, d, w,
                        reinterpret_cast<const uint4*>(buf), reinterpret_cast<float4*>(y));
  return hipGetLastError();
}

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
