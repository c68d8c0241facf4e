// Router scoring and top-k for gfx950 (the routing that decides R at each layer, WiSP Sec. 3.1).
//
// router_logits: z[t, e] = W_r[e] . x[t] in fp32.  One wavefront per (expert row, group of up
//   to four tokens); the 64 lanes stream the fp32 row with 16-byte loads and reduce with
//   cross-lane shuffles.
// router_select: one wavefront per token.  Each lane holds the logits of experts lane, lane+64,
//   lane+128, lane+192 (N <= 256).  Selection runs k rounds of a wave-wide argmax on
//   (score desc, expert id asc); the score used for ordering is the logit itself, which ranks
//   experts exactly as softmax or sigmoid do (both are increasing) without creating ties.
//   Group-limited routing first scores each group by its two largest sigmoids and keeps the best
//   groups.  Gates: softmax over the chosen logits (equal to renormalising a softmax over all
//   N), or chosen sigmoids divided by their sum.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>

#include "kernels.hpp"

namespace wisp {
namespace {

enum { R_SOFTMAX_RENORM = 0, R_TOPK_SOFTMAX = 1, R_SIGMOID_GROUP = 2 };

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

template <int XT>
__global__ void __launch_bounds__(256) router_logits_kernel(const float* __restrict__ wr, const void* __restrict__ x,
                                                            int T, int N, int d, float* __restrict__ logits) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int e = blockIdx.x * 4 + wave;
  const int t0 = blockIdx.y * 4;
  if (e >= N) return;
  const int ntok = min(4, T - t0);
  const float4* row = reinterpret_cast<const float4*>(wr + static_cast<size_t>(e) * d);
  const int chunks = d / 4;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int c = lane; c < chunks; c += 64) {
    const float4 w = row[c];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (t >= ntok) break;
      const float4 v = load_x4<XT>(x, static_cast<size_t>(t0 + t) * d + static_cast<size_t>(c) * 4);
      acc[t] = fmaf(w.x, v.x, acc[t]);
      acc[t] = fmaf(w.y, v.y, acc[t]);
      acc[t] = fmaf(w.z, v.z, acc[t]);
      acc[t] = fmaf(w.w, v.w, acc[t]);
    }
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t >= ntok) break;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc[t] += __shfl_xor(acc[t], off, 64);
  }
  if (lane == 0)
    for (int t = 0; t < ntok; ++t) logits[static_cast<size_t>(t0 + t) * N + e] = acc[t];
}

// Wave-wide argmax on (v desc, id asc); every lane returns the winner.
__device__ __forceinline__ void wave_argmax(float& v, int& id) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(v, off, 64);
    const int oid = __shfl_xor(id, off, 64);
    if (ov > v || (ov == v && oid < id)) { v = ov; id = oid; }
  }
}

// Best of this lane's candidates that pass `ok`, then the wave-wide winner.
template <typename Ok>
__device__ __forceinline__ void argmax_masked(const float* z, int lane, Ok ok, float& bv, int& bi) {
  bv = -INFINITY;
  bi = 0x7FFFFFFF;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int e = lane + 64 * m;
    if (ok(m, e) && (z[m] > bv || bi == 0x7FFFFFFF)) { bv = z[m]; bi = e; }
  }
  wave_argmax(bv, bi);
}

__device__ __forceinline__ float sigmoidf(float z) { return 1.0f / (1.0f + __expf(-z)); }

__global__ void __launch_bounds__(256) router_select_kernel(const float* __restrict__ logits, int T, int N, int k,
                                                            int route, int n_groups, int topk_groups,
                                                            int32_t* __restrict__ idx, float* __restrict__ w) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  if (t >= T) return;
  float z[4];
  bool allowed[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int e = lane + 64 * m;
    allowed[m] = e < N;
    z[m] = allowed[m] ? logits[static_cast<size_t>(t) * N + e] : -INFINITY;
  }
  if (route == R_SIGMOID_GROUP) {
    const int gs = N / n_groups;
    uint32_t kept = 0;
    float gscore[32];
    for (int q = 0; q < n_groups && q < 32; ++q) {
      float v1, v2;
      int i1, i2;
      argmax_masked(z, lane, [&](int m, int e) { return allowed[m] && e / gs == q; }, v1, i1);
      argmax_masked(z, lane, [&](int m, int e) { return allowed[m] && e / gs == q && e != i1; }, v2, i2);
      gscore[q] = sigmoidf(v1) + (gs > 1 ? sigmoidf(v2) : 0.f);
    }
    for (int j = 0; j < topk_groups; ++j) {
      int best = -1;
      for (int q = 0; q < n_groups && q < 32; ++q) {
        if (kept & (1u << q)) continue;
        if (best < 0 || gscore[q] > gscore[best]) best = q;
      }
      if (best >= 0) kept |= 1u << best;
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int e = lane + 64 * m;
      allowed[m] = allowed[m] && ((kept >> (e / gs)) & 1u);
    }
  }
  float zs[8];
  int is[8];
  for (int j = 0; j < k; ++j) {
    float bv;
    int bi;
    argmax_masked(z, lane, [&](int m, int e) { return allowed[m]; }, bv, bi);
    zs[j] = bv;
    is[j] = bi;
#pragma unroll
    for (int m = 0; m < 4; ++m)
      if (lane + 64 * m == bi) allowed[m] = false;
  }
  if (lane == 0) {
    float g[8];
    float den = 0.f;
    if (route == R_SIGMOID_GROUP) {
      for (int j = 0; j < k; ++j) { g[j] = sigmoidf(zs[j]); den += g[j]; }
    } else {
      for (int j = 0; j < k; ++j) { g[j] = __expf(zs[j] - zs[0]); den += g[j]; }
    }
    const float inv = 1.0f / den;
    for (int j = 0; j < k; ++j) {
      idx[t * k + j] = is[j];
      w[t * k + j] = g[j] * inv;
    }
  }
}

}  // namespace

hipError_t launch_router_logits(const float* wr, const void* x, int x_dtype, int T, int N, int d, float* logits,
                                hipStream_t st, const LaunchTiming& tm) {
  if (T <= 0) return hipSuccess;
  if (d % 4 != 0) return hipErrorInvalidValue;
  dim3 grid((N + 3) / 4, (T + 3) / 4), block(256);
  if (x_dtype == DT_F32)
    hipExtLaunchKernelGGL(router_logits_kernel<DT_F32>, grid, block, 0, st, tm.start, tm.stop, 0, wr, x, T, N, d,
                          logits);
  else
    hipExtLaunchKernelGGL(router_logits_kernel<DT_BF16>, grid, block, 0, st, tm.start, tm.stop, 0, wr, x, T, N, d,
                          logits);
  return hipGetLastError();
}

hipError_t launch_router_select(const float* logits, int T, int N, int k, int route, int n_groups, int topk_groups,
                                int32_t* idx, float* w, hipStream_t st, const LaunchTiming& tm) {
  if (T <= 0) return hipSuccess;
  if (N > 256 || k > 8 || k < 1 || (route == R_SIGMOID_GROUP && (n_groups > 32 || N % n_groups != 0)))
    return hipErrorInvalidValue;
  dim3 grid((T + 3) / 4), block(256);
  hipExtLaunchKernelGGL(router_select_kernel, grid, block, 0, st, tm.start, tm.stop, 0, logits, T, N, k, route,
                        n_groups, topk_groups, idx, w);
  return hipGetLastError();
}

}  // namespace wisp
