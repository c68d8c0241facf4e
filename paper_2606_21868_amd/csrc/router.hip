// Router scoring and top-k for gfx950 (the routing that decides R at each layer, WiSP Sec. 3.1).
//
// router_logits: z[t, e] = W_r[e] . x[t] in fp32.  Decode sizes (T <= 8): one workgroup per
//   expert row, so the fp32 router matrix is read by N workgroups at once (one HBM round trip);
//   larger T: one wavefront per (expert row, four tokens).
// router_select: one wavefront per token, its N <= 256 scores in LDS.  Every lane computes the
//   rank of its experts (the number of allowed experts that order before it on (score desc,
//   id asc)) and the expert of rank j < k is written to slot j: a parallel selection with no
//   dependent cross-lane chains.  The ordering score is the logit itself, which orders experts
//   exactly as softmax or sigmoid do (both increase) without creating ties by rounding.
//   Group-limited routing first scores each group by the sum of its two largest sigmoids and
//   keeps the topk_groups best groups.  Gates: softmax over the chosen logits (equal to
//   renormalising a softmax over all N), or the chosen sigmoids divided by their sum.  The
//   indices can also be published to host-coherent memory as 64-bit (sequence, id) words, which
//   is how the host pager learns R without a copy, an event or a fence.
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

// Decode-sized logits: one workgroup per expert row; 256 threads split the row (16-byte loads),
// reduce through shuffles and LDS.  Up to four tokens per pass.
template <int XT>
__global__ void __launch_bounds__(256) router_logits_wide_kernel(const float* __restrict__ wr,
                                                                 const void* __restrict__ x, int T, int N, int d,
                                                                 float* __restrict__ logits) {
  __shared__ float part[4][4];
  const int e = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float4* row = reinterpret_cast<const float4*>(wr + static_cast<size_t>(e) * d);
  const int chunks = d / 4;
  for (int t0 = 0; t0 < T; t0 += 4) {
    const int ntok = min(4, T - t0);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c = threadIdx.x; c < chunks; c += 256) {
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
      if (lane == 0) part[t][wave] = acc[t];
    }
    __syncthreads();
    if (threadIdx.x < ntok) {
      const int t = threadIdx.x;
      logits[static_cast<size_t>(t0 + t) * N + e] = (part[t][0] + part[t][1]) + (part[t][2] + part[t][3]);
    }
    __syncthreads();
  }
}

__device__ __forceinline__ float sigmoidf(float z) { return 1.0f / (1.0f + __expf(-z)); }

// Does candidate (va, a) rank before (vb, b)?  Value descending, then id ascending.
__device__ __forceinline__ bool better(float va, int a, float vb, int b) { return va > vb || (va == vb && a < b); }

// Selection by ranks: one wavefront per token, the token's scores in LDS; each lane computes the
// rank of its experts among the allowed ones (count of candidates that rank before it) and the
// expert of rank j < k lands in slot j.  No dependent chains of cross-lane operations.  The
// ordering score is the logit (softmax and sigmoid are increasing, so the order is the same and
// no ties are created by rounding a sigmoid).
__global__ void __launch_bounds__(256) router_select_kernel(const float* __restrict__ logits, int T, int N, int k,
                                                            int route, int n_groups, int topk_groups,
                                                            int32_t* __restrict__ idx, float* __restrict__ w,
                                                            uint64_t* __restrict__ idx_host, uint32_t seq) {
  __shared__ float zs[4][256];
  __shared__ uint8_t ok[4][256];
  __shared__ float gam[4][32];
  __shared__ int sel[4][8];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  const bool active = t < T;
  if (active) {
    for (int e = lane; e < N; e += 64) {
      zs[wave][e] = logits[static_cast<size_t>(t) * N + e];
      ok[wave][e] = 1;
    }
  }
  __syncthreads();
  if (route == R_SIGMOID_GROUP) {
    const int gs = N / n_groups;
    // group score: sum of the sigmoids of the group's two best experts
    if (active && lane < n_groups) {
      const int q = lane;
      int b1 = -1, b2 = -1;
      for (int e = q * gs; e < (q + 1) * gs; ++e) {
        if (b1 < 0 || better(zs[wave][e], e, zs[wave][b1], b1)) { b2 = b1; b1 = e; }
        else if (b2 < 0 || better(zs[wave][e], e, zs[wave][b2], b2)) b2 = e;
      }
      gam[wave][q] = sigmoidf(zs[wave][b1]) + (b2 >= 0 ? sigmoidf(zs[wave][b2]) : 0.f);
    }
    __syncthreads();
    // keep the topk_groups best groups (score desc, group asc)
    if (active) {
      for (int e = lane; e < N; e += 64) {
        const int q = e / gs;
        int grank = 0;
        for (int q2 = 0; q2 < n_groups; ++q2) grank += better(gam[wave][q2], q2, gam[wave][q], q) ? 1 : 0;
        ok[wave][e] = grank < topk_groups;
      }
    }
  }
  __syncthreads();
  if (active) {
    for (int e = lane; e < N; e += 64) {
      if (!ok[wave][e]) continue;
      const float ze = zs[wave][e];
      int rank = 0;
      for (int e2 = 0; e2 < N; ++e2) rank += (ok[wave][e2] && better(zs[wave][e2], e2, ze, e)) ? 1 : 0;
      if (rank < k) sel[wave][rank] = e;
    }
  }
  __syncthreads();
  if (active && lane == 0) {
    float g[8];
    float den = 0.f;
    const float z0 = zs[wave][sel[wave][0]];
    for (int j = 0; j < k; ++j) {
      const float zj = zs[wave][sel[wave][j]];
      g[j] = route == R_SIGMOID_GROUP ? sigmoidf(zj) : __expf(zj - z0);
      den += g[j];
    }
    const float inv = 1.0f / den;
    for (int j = 0; j < k; ++j) {
      idx[t * k + j] = sel[wave][j];
      w[t * k + j] = g[j] * inv;
    }
  }
  // publish to host-coherent memory: every entry is one 64-bit store of (seq << 32 | id), so the
  // host knows an entry is current from its tag alone and no fence is needed
  if (idx_host && active && lane < k)
    __hip_atomic_store(idx_host + t * k + lane, (static_cast<uint64_t>(seq) << 32) | static_cast<uint32_t>(sel[wave][lane]),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace

hipError_t launch_router_logits(const float* wr, const void* x, int x_dtype, int T, int N, int d, float* logits,
                                hipStream_t st, const LaunchTiming& tm) {
  if (T <= 0) return hipSuccess;
  if (d % 4 != 0) return hipErrorInvalidValue;
  if (T <= 8) {
    dim3 grid(N), block(256);
    if (x_dtype == DT_F32)
      hipExtLaunchKernelGGL(router_logits_wide_kernel<DT_F32>, grid, block, 0, st, tm.start, tm.stop, 0, wr, x, T, N,
                            d, logits);
    else
      hipExtLaunchKernelGGL(router_logits_wide_kernel<DT_BF16>, grid, block, 0, st, tm.start, tm.stop, 0, wr, x, T, N,
                            d, logits);
    return hipGetLastError();
  }
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
                                int32_t* idx, float* w, uint64_t* idx_host, uint32_t seq, hipStream_t st,
                                const LaunchTiming& tm) {
  if (T <= 0) return hipSuccess;
  if (N > 256 || k > 8 || k < 1 || (route == R_SIGMOID_GROUP && (n_groups > 32 || N % n_groups != 0)))
    return hipErrorInvalidValue;
  dim3 grid((T + 3) / 4), block(256);
  hipExtLaunchKernelGGL(router_select_kernel, grid, block, 0, st, tm.start, tm.stop, 0, logits, T, N, k, route,
                        n_groups, topk_groups, idx, w, idx_host, seq);
  return hipGetLastError();
}

}  // namespace wisp
