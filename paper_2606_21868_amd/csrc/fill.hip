// Expert fills by the compute units: faulted blobs read straight from their pinned host masters over
// the host link and stored into their HBM slots (WiSP Algorithm 1's fills, as the device pager's
// streaming does).  One launch per fill list on the side stream.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace wisp {
namespace {

// Workgroups of a fill launch: about kFillWgsTotal whatever the number of blobs (each thread holds
// four 16-byte loads in flight, so a few dozen workgroups keep the link busy), between 4 and 32 per
// blob.  Thousands of workgroups each streaming its own part of host memory were measured slower.
constexpr int kFillWgsTotal = 128;

__global__ void __launch_bounds__(256) fill_kernel(const FillList fl, uint64_t bytes, int wgs) {
  const int item = static_cast<int>(blockIdx.x) / wgs, q = static_cast<int>(blockIdx.x) % wgs;
  if (item >= fl.n) return;
  const uint4* src = reinterpret_cast<const uint4*>(fl.src[item]);
  uint4* dst = reinterpret_cast<uint4*>(fl.dst[item]);
  const uint64_t n16 = bytes / 16;
  const uint64_t per = (n16 + wgs - 1) / wgs;
  const uint64_t c0 = static_cast<uint64_t>(q) * per;
  const uint64_t c1 = c0 + per < n16 ? c0 + per : n16;
  uint64_t i = c0 + threadIdx.x;
  for (; i + 768 < c1; i += 1024) {
    const uint4 a = src[i], b = src[i + 256], c = src[i + 512], e = src[i + 768];
    dst[i] = a;
    dst[i + 256] = b;
    dst[i + 512] = c;
    dst[i + 768] = e;
  }
  for (; i < c1; i += 256) dst[i] = src[i];
  if (q == wgs - 1) {
    for (uint64_t b = n16 * 16 + threadIdx.x; b < bytes; b += 256)
      reinterpret_cast<uint8_t*>(fl.dst[item])[b] = fl.src[item][b];
  }
}

}  // namespace

hipError_t launch_fill(const FillList& fl, uint64_t bytes, hipStream_t st, const LaunchTiming& tm) {
  if (fl.n <= 0) return hipSuccess;
  if (fl.n > kMaxFills) return hipErrorInvalidValue;
  int wgs = kFillWgsTotal / fl.n;
  wgs = wgs < 4 ? 4 : wgs > 32 ? 32 : wgs;
  hipExtLaunchKernelGGL(fill_kernel, dim3(static_cast<unsigned>(fl.n * wgs)), dim3(256), 0, st, tm.start, tm.stop, 0,
                        fl, bytes, wgs);
  return hipGetLastError();
}

}  // namespace wisp
