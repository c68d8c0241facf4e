// Router scoring and top-k for gfx950 (the routing that decides R at each layer, WiSP Sec. 3.1).
//
// router_logits: z[t, e] = W_r[e] . x[t] in fp32.  Decode sizes (T <= 8): one workgroup per
//   expert row, so the fp32 router matrix is read by N workgroups at once (one HBM round trip);
//   token batches: fp32 matrix cores (a 16-token x 16-row block per workgroup) when N is a
//   multiple of 16 and d of 64, else a workgroup per 16 tokens with LDS-staged slices of W_r.
// router_select: top-k selection and gates (select.hpp), optionally publishing the ids to the
//   host pager through host-coherent memory.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>

#include "kernels.hpp"
#include "router_row.hpp"
#include "select.hpp"

namespace wisp {
namespace {

// Decode-sized logits: one workgroup per expert row (router_row in router_row.hpp), up to four
// tokens per pass.
template <int XT>
__global__ void __launch_bounds__(256) router_logits_wide_kernel(const float* __restrict__ wr,
                                                                 const void* __restrict__ x, int T, int N, int d,
                                                                 float* __restrict__ logits) {
  __shared__ float part[4][4];
  const int e = blockIdx.x;
  for (int t0 = 0; t0 < T; t0 += 4) {
    const int ntok = min(4, T - t0);
    const float z = router_row<XT>(wr, x, t0, ntok, d, e, part);
    if (threadIdx.x < ntok) logits[static_cast<size_t>(t0 + threadIdx.x) * N + e] = z;
    __syncthreads();
  }
}

// Token-batch logits: a workgroup per 16 tokens computes their logits against all N <= 256 router
// rows, staging 32-column slices of W_r and of the tokens in LDS (fp32; padded rows keep the
// 16-byte reads conflict-free).  Thread e owns router row e (N <= 128: two half-blocks of 8 tokens
// each).  Every logit is one fp32 FMA chain in ascending column order.
template <int XT, int TPT>
__global__ void __launch_bounds__(256) router_logits_tiled_kernel(const float* __restrict__ wr,
                                                                  const void* __restrict__ x, int T, int N, int d,
                                                                  float* __restrict__ logits) {
  constexpr int TT = 16, KS = 32, LD = KS + 4;
  __shared__ __attribute__((aligned(16))) float Ws[256 * LD];
  __shared__ __attribute__((aligned(16))) float Xs[TT * LD];
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * TT;
  const int e = TPT == 16 ? tid : (tid & 127);
  const int tb = TPT == 16 ? 0 : (tid >> 7) * 8;
  float acc[TPT];
#pragma unroll
  for (int t = 0; t < TPT; ++t) acc[t] = 0.f;
  for (int k0 = 0; k0 < d; k0 += KS) {
    for (int i = tid; i < N * (KS / 4); i += 256) {
      const int r = i / (KS / 4), c = (i % (KS / 4)) * 4;
      *reinterpret_cast<float4*>(&Ws[r * LD + c]) =
          *reinterpret_cast<const float4*>(wr + static_cast<size_t>(r) * d + k0 + c);
    }
    if (tid < TT * (KS / 4)) {
      const int r = tid / (KS / 4), c = (tid % (KS / 4)) * 4;
      *reinterpret_cast<float4*>(&Xs[r * LD + c]) =
          t0 + r < T ? load_x4<XT>(x, static_cast<size_t>(t0 + r) * d + k0 + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    __syncthreads();
    if (e < N) {
#pragma unroll
      for (int kk = 0; kk < KS; kk += 4) {
        const float4 w = *reinterpret_cast<const float4*>(&Ws[e * LD + kk]);
#pragma unroll
        for (int t = 0; t < TPT; ++t) {
          const float4 v = *reinterpret_cast<const float4*>(&Xs[(tb + t) * LD + kk]);
          acc[t] = fmaf(w.x, v.x, acc[t]);
          acc[t] = fmaf(w.y, v.y, acc[t]);
          acc[t] = fmaf(w.z, v.z, acc[t]);
          acc[t] = fmaf(w.w, v.w, acc[t]);
        }
      }
    }
    __syncthreads();
  }
  if (e < N) {
#pragma unroll
    for (int t = 0; t < TPT; ++t)
      if (t0 + tb + t < T) logits[static_cast<size_t>(t0 + tb + t) * N + e] = acc[t];
  }
}

// Token-batch logits on the fp32 matrix cores (v_mfma_f32_16x16x4_f32).  A workgroup computes a
// 16-token x 16-row block; its four waves take one quarter of the columns each and their partial
// sums are added in wave order through LDS.  W_r stays fp32 and x is widened exactly, so the
// products are those of the FMA kernels and only the summation order differs.  Lane l owns token
// l%16 and router row l%16; for each 16-column step it reads columns 4(l/16) .. +3 of both (one 8-
// or 16-byte load each, issued a step ahead) for four MFMA steps, which keeps the column index of a
// lane's A and B operands equal, as the product requires.  Output lane l: tokens 4(l/16) .. +3, row l%16.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
template <int XT>
__global__ void __launch_bounds__(256) router_logits_mfma_kernel(const float* __restrict__ wr,
                                                                 const void* __restrict__ x, int T, int N, int d,
                                                                 float* __restrict__ logits) {
  __shared__ f32x4_t part[3][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t0 = blockIdx.x * 16, e0 = blockIdx.y * 16;
  const int r = lane & 15, g = lane >> 4;
  const bool tok_ok = t0 + r < T;
  const int kq = d / 4;                         // columns per wave (d % 64 == 0)
  const int kbeg = wave * kq;
  const float* wrow = wr + static_cast<size_t>(e0 + r) * d + kbeg + 4 * g;
  const size_t xoff = static_cast<size_t>(tok_ok ? t0 + r : 0) * d + kbeg + 4 * g;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  float4 w = *reinterpret_cast<const float4*>(wrow);
  float4 v = tok_ok ? load_x4<XT>(x, xoff) : make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k0 = 0; k0 < kq; k0 += 16) {
    float4 wn = w, vn = v;
    if (k0 + 16 < kq) {
      wn = *reinterpret_cast<const float4*>(wrow + k0 + 16);
      if (tok_ok) vn = load_x4<XT>(x, xoff + k0 + 16);
    }
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(v.x, w.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(v.y, w.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(v.z, w.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(v.w, w.w, acc, 0, 0, 0);
    w = wn;
    v = vn;
  }
  if (wave > 0) part[wave - 1][lane] = acc;
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const f32x4_t p = part[q][lane];
      acc[0] += p[0];
      acc[1] += p[1];
      acc[2] += p[2];
      acc[3] += p[3];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int t = t0 + 4 * g + q;
      if (t < T) logits[static_cast<size_t>(t) * N + e0 + r] = acc[q];
    }
  }
}

// Selection (select.hpp) of the workgroup's four tokens; wave w, lane j < k writes rank j of
// token blockIdx.x * 4 + w.  The indices can also be published to host-coherent memory as 64-bit
// (seq << 32 | id) words: the host knows an entry is current from its tag alone, so it needs no
// copy, event or fence to read them.
__global__ void __launch_bounds__(256) router_select_kernel(const float* __restrict__ logits, int T, int N, int k,
                                                            int route, int n_groups, int topk_groups,
                                                            int32_t* __restrict__ idx, float* __restrict__ w,
                                                            uint64_t* __restrict__ idx_host, uint32_t seq) {
  __shared__ SelectShared sh;
  select_tokens(logits, 0, blockIdx.x * 4, T, N, k, route, n_groups, topk_groups, sh);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  if (t < T && lane < k) {
    const int e = sh.sel[wave][lane];
    idx[t * k + lane] = e;
    w[t * k + lane] = sh.gate[wave][lane];
    if (idx_host)
      __hip_atomic_store(idx_host + t * k + lane, (static_cast<uint64_t>(seq) << 32) | static_cast<uint32_t>(e),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// Router logits and the selection of up to four tokens in one launch (decode).  Workgroup e computes
// logit row e (router_row: the arithmetic of router_logits_wide_kernel), publishes it as tagged words
// (tag_logit, one atomic store each) and counts itself in *arrive; the workgroup whose arrival
// completes the count resets the counter and selects on the complete logits, reading each word until
// it carries this launch's tag, and writes idx, w and, if asked, the tagged ids for the host.  No
// workgroup waits for another's progress: the count only elects the selecting workgroup, and the
// tags (not an ordering of the counter after the stores) make it read this launch's logits.
template <int XT>
__global__ void __launch_bounds__(256) route_select_kernel(const float* __restrict__ wr, const void* __restrict__ x,
                                                           int d, uint64_t* __restrict__ logits, uint32_t tag,
                                                           uint32_t* __restrict__ arrive, int T, int N, int k,
                                                           int route, int n_groups, int topk_groups,
                                                           int32_t* __restrict__ idx, float* __restrict__ w,
                                                           uint64_t* __restrict__ idx_host, uint32_t seq) {
  __shared__ SelectShared sh;
  __shared__ float part[4][4];
  __shared__ int last;
  const int e = blockIdx.x;
  const float z = router_row<XT>(wr, x, 0, T, d, e, part);
  if (static_cast<int>(threadIdx.x) < T)
    __hip_atomic_store(logits + static_cast<size_t>(threadIdx.x) * N + e, tag_logit(tag, z), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t before = __hip_atomic_fetch_add(arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last = before + 1 == static_cast<uint32_t>(N);
    if (last) __hip_atomic_store(arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!last) return;
  select_tokens<true>(logits, tag, 0, T, N, k, route, n_groups, topk_groups, sh);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (wave < T && lane < k) {
    const int s = sh.sel[wave][lane];
    idx[wave * k + lane] = s;
    w[wave * k + lane] = sh.gate[wave][lane];
    if (idx_host)
      __hip_atomic_store(idx_host + wave * k + lane, (static_cast<uint64_t>(seq) << 32) | static_cast<uint32_t>(s),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

}  // namespace

hipError_t launch_route_select(const float* wr, const void* x, int x_dtype, int d, uint64_t* logits, uint32_t tag,
                               uint32_t* arrive, int T, int N, int k, int route, int n_groups, int topk_groups,
                               int32_t* idx, float* w, uint64_t* idx_host, uint32_t seq, hipStream_t st,
                               const LaunchTiming& tm) {
  if (T < 1 || T > 4 || N < 1 || N > 256 || k < 1 || k > 8 || d % 4 != 0 ||
      (route == R_SIGMOID_GROUP && (n_groups > 32 || N % n_groups != 0)))
    return hipErrorInvalidValue;
  if (x_dtype == DT_F32)
    hipExtLaunchKernelGGL(route_select_kernel<DT_F32>, dim3(N), dim3(256), 0, st, tm.start, tm.stop, 0, wr, x, d, logits,
                          tag, arrive, T, N, k, route, n_groups, topk_groups, idx, w, idx_host, seq);
  else
    hipExtLaunchKernelGGL(route_select_kernel<DT_BF16>, dim3(N), dim3(256), 0, st, tm.start, tm.stop, 0, wr, x, d,
                          logits, tag, arrive, T, N, k, route, n_groups, topk_groups, idx, w, idx_host, seq);
  return hipGetLastError();
}

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
  if (N % 16 == 0 && d % 64 == 0) {
    dim3 grid((T + 15) / 16, N / 16), block(256);
    if (x_dtype == DT_F32)
      hipExtLaunchKernelGGL(router_logits_mfma_kernel<DT_F32>, grid, block, 0, st, tm.start, tm.stop, 0, wr, x, T, N,
                            d, logits);
    else
      hipExtLaunchKernelGGL(router_logits_mfma_kernel<DT_BF16>, grid, block, 0, st, tm.start, tm.stop, 0, wr, x, T,
                            N, d, logits);
    return hipGetLastError();
  }
  if (d % 32 == 0 && N <= 256) {
    dim3 grid((T + 15) / 16), block(256);
    const bool half = N <= 128;
    if (x_dtype == DT_F32) {
      if (half)
        hipExtLaunchKernelGGL(router_logits_tiled_kernel<DT_F32, 8>, grid, block, 0, st, tm.start, tm.stop, 0, wr, x,
                              T, N, d, logits);
      else
        hipExtLaunchKernelGGL(router_logits_tiled_kernel<DT_F32, 16>, grid, block, 0, st, tm.start, tm.stop, 0, wr,
                              x, T, N, d, logits);
    } else {
      if (half)
        hipExtLaunchKernelGGL(router_logits_tiled_kernel<DT_BF16, 8>, grid, block, 0, st, tm.start, tm.stop, 0, wr,
                              x, T, N, d, logits);
      else
        hipExtLaunchKernelGGL(router_logits_tiled_kernel<DT_BF16, 16>, grid, block, 0, st, tm.start, tm.stop, 0, wr,
                              x, T, N, d, logits);
    }
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
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
