// One router logit row for decode-sized token counts, shared by the router kernel and the device
// pager's fused route-and-page kernel so that both compute every logit with the same operations.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "kernels.hpp"

namespace wisp {

template <int XT>
__device__ __forceinline__ float4 load_x4(const void* x, size_t idx) {
  if constexpr (XT == DT_F32) {
    return *reinterpret_cast<const float4*>(static_cast<const float*>(x) + idx);
  } else {
    const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(x) + idx);
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u));
  }
}

// z = W_r[e] . x[t0 + t] for the ntok <= 4 tokens t, by all 256 threads of the workgroup: 16-byte
// loads of the fp32 row, a shuffle reduction per wave and the four wave sums added in a fixed
// order.  Thread t < ntok returns token t's logit (others return 0); part is a 4x4 LDS scratch.  Ends
// with the threads of the workgroup synchronised.
template <int XT>
__device__ __forceinline__ float router_row(const float* __restrict__ wr, const void* __restrict__ x, int t0, int ntok,
                                            int d, int e, float (*part)[4]) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float4* row = reinterpret_cast<const float4*>(wr + static_cast<size_t>(e) * d);
  const int chunks = d / 4;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  // the thread's chunks c = tid, tid + 256, ... in groups of U whose row loads are all issued before
  // the first FMA (one HBM round trip per group, not per chunk); each acc[t] is still one FMA chain
  // in ascending chunk order.  The first group covers every d up to 256 * U * 4 = 4096; it runs
  // outside the loop so that its row loads also overlap with whatever the caller issued before
  // (inside a loop they would wait for those first).
  constexpr int U = 4;
  auto group = [&](int c0) {
    float4 wv[U], xf[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 256;
      wv[u] = c < chunks ? row[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    // the first token's inputs go out with the row (a chunk past the last reads the last one again:
    // in bounds, never used), so a single-token step waits once
#pragma unroll
    for (int u = 0; u < U; ++u)
      xf[u] = load_x4<XT>(x, static_cast<size_t>(t0) * d + static_cast<size_t>(min(c0 + u * 256, chunks - 1)) * 4);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 256;
      if (c >= chunks) break;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (t >= ntok) break;
        const float4 v =
            t == 0 ? xf[u] : load_x4<XT>(x, static_cast<size_t>(t0 + t) * d + static_cast<size_t>(c) * 4);
        acc[t] = fmaf(wv[u].x, v.x, acc[t]);
        acc[t] = fmaf(wv[u].y, v.y, acc[t]);
        acc[t] = fmaf(wv[u].z, v.z, acc[t]);
        acc[t] = fmaf(wv[u].w, v.w, acc[t]);
      }
    }
  };
  group(threadIdx.x);
  for (int c0 = threadIdx.x + 256 * U; c0 < chunks; c0 += 256 * U) group(c0);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t >= ntok) break;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc[t] += __shfl_xor(acc[t], off, 64);
    if (lane == 0) part[t][wave] = acc[t];
  }
  __syncthreads();
  float z = 0.f;
  if (static_cast<int>(threadIdx.x) < ntok) {
    const int t = threadIdx.x;
    z = (part[t][0] + part[t][1]) + (part[t][2] + part[t][3]);
  }
  __syncthreads();
  return z;
}

}  // namespace wisp
