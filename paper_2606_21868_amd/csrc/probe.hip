// Yardsticks: a plain device copy with 16-byte loads and stores (for HBM byte counters, FETCH_SIZE /
// WRITE_SIZE per copied byte, and the achievable copy bandwidth), a plain streaming read (the read
// time of a launch of a given size, the floor of any kernel that must read those bytes), and a
// register-only stream of bf16 matrix-core instructions (the dense bf16 rate the chip sustains).
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace wisp {
namespace {

__global__ void __launch_bounds__(256) hbm_copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                       size_t n) {
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Each thread issues its four 16-byte non-temporal loads before using any; a workgroup covers 16 KB.
// The loaded words are folded into one value that is stored only if it equals an arbitrary constant,
// so the loads cannot be dropped and the kernel writes (almost) nothing.
__global__ void __launch_bounds__(256) hbm_read_kernel(const u32x4_t* __restrict__ src, size_t n, uint32_t* sink) {
  const size_t base = static_cast<size_t>(blockIdx.x) * 1024 + threadIdx.x;
  u32x4_t a[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const size_t i = base + static_cast<size_t>(m) * 256;
    a[m] = i < n ? __builtin_nontemporal_load(src + i) : u32x4_t{0u, 0u, 0u, 0u};
  }
  uint32_t acc = 0;
#pragma unroll
  for (int m = 0; m < 4; ++m) acc ^= a[m].x ^ a[m].y ^ a[m].z ^ a[m].w;
  if (acc == 0x9e3779b9u) sink[0] = acc;
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Every wave runs `iters` rounds of four independent v_mfma_f32_32x32x16_bf16 chains on register
// operands (2 * 32 * 32 * 16 flops each); nothing touches memory but a store that happens only if
// the folded result equals an arbitrary constant.
__global__ void __launch_bounds__(256) mfma_peak_kernel(int iters, float* sink) {
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<__bf16>(static_cast<float>((threadIdx.x + i) & 7) * 0.125f);
    b[i] = static_cast<__bf16>(static_cast<float>((threadIdx.x * 3 + i) & 7) * 0.0625f);
  }
  f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, b, c3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
  if (s == 1234.5f) sink[0] = s;
}

}  // namespace

hipError_t launch_mfma_peak(int wgs, int iters, float* sink, hipStream_t st) {
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(static_cast<unsigned>(wgs)), dim3(256), 0, st, iters, sink);
  return hipGetLastError();
}

hipError_t launch_hbm_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  const size_t n = bytes / 16;
  hipLaunchKernelGGL(hbm_read_kernel, dim3(static_cast<unsigned>((n + 1023) / 1024)), dim3(256), 0, st,
                     static_cast<const u32x4_t*>(src), n, sink);
  return hipGetLastError();
}

hipError_t launch_hbm_copy(const void* src, void* dst, size_t bytes, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  const size_t n = bytes / 16;
  size_t blocks = (n + 255) / 256;
  if (blocks > 256 * 32) blocks = 256 * 32;
  hipLaunchKernelGGL(hbm_copy_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                     static_cast<const uint4*>(src), static_cast<uint4*>(dst), n);
  return hipGetLastError();
}

}  // namespace wisp
