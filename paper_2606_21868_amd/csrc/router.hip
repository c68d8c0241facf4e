// Router scoring and top-k for gfx950 (the routing that decides R at each layer, WiSP Sec. 3.1).
//
// router_logits: z[t, e] = W_r[e] . x[t] in fp32.  Decode sizes (T <= 8): one workgroup per
//   expert row, so the fp32 router matrix is read by N workgroups at once (one HBM round trip);
//   token batches: fp32 matrix cores (64 tokens against all router rows over a slice of the columns
//   per workgroup, slices summed by the selection) when N is a multiple of 16, else a workgroup per
//   16 tokens with LDS-staged slices of W_r.
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

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Token-batch logits with the router matrix read once per 64 tokens: a workgroup computes 64 tokens
// against all N router rows over one of n_split slices of the columns (grid: token blocks x slices),
// on the fp32 matrix cores (v_mfma_f32_16x16x4_f32).  Wave w takes the 16-row blocks b = w, w + 4,
// ... of W_r and all four 16-token blocks; per 16-column step lane l (r = l % 16, g = l / 16) holds
// columns 4g .. 4g + 3 of token r of each token block and of row r of each row block, one step ahead
// of the matrix-core work.  The slice's sums go to partial[slice][token][row]; the selection adds the
// slices in order.  (W_r is re-read T / 64 times instead of T / 16 times by 16 x 16 blocks.)
template <int XT, int RB>
__global__ void __launch_bounds__(256) router_logits_split_kernel(const float* __restrict__ wr,
                                                                  const void* __restrict__ x, int T, int N, int d,
                                                                  int ks, float* __restrict__ partial) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int t0 = blockIdx.x * 64, q = blockIdx.y, kbeg = q * ks;
  const int nb = N / 16;
  const float* wrow[RB];
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const int blk = min(wave + 4 * b, nb - 1);   // a block past N repeats the last (never stored)
    wrow[b] = wr + static_cast<size_t>(16 * blk + r) * d + kbeg + 4 * g;
  }
  size_t xoff[4];
#pragma unroll
  for (int tb = 0; tb < 4; ++tb) {
    const int t = t0 + 16 * tb + r;
    xoff[tb] = static_cast<size_t>(t < T ? t : 0) * d + kbeg + 4 * g;
  }
  f32x4_t acc[4][RB];
#pragma unroll
  for (int tb = 0; tb < 4; ++tb)
#pragma unroll
    for (int b = 0; b < RB; ++b) acc[tb][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // operands of PF 16-column steps in flight (one wave per SIMD: the loads of a step are issued PF
  // steps before its matrix-core work); step j lives in ring slot j % PF.  The loads are unconditional
  // (a token past T reads token 0's row, never stored) and the inputs stay raw until used, so no load
  // waits for another.
  constexpr int PF = 4;
  constexpr int XW = XT == DT_F32 ? 4 : 2;   // 32-bit words of four inputs
  float4 w[PF][RB];
  uint32_t v[PF][4][XW];
  auto load = [&](int slot, int k0) {
#pragma unroll
    for (int b = 0; b < RB; ++b) w[slot][b] = *reinterpret_cast<const float4*>(wrow[b] + k0);
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      if constexpr (XT == DT_F32) {
        const uint4 q4 = *reinterpret_cast<const uint4*>(static_cast<const float*>(x) + xoff[tb] + k0);
        v[slot][tb][0] = q4.x; v[slot][tb][1] = q4.y; v[slot][tb][2] = q4.z; v[slot][tb][3] = q4.w;
      } else {
        const uint2 q2 = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(x) + xoff[tb] + k0);
        v[slot][tb][0] = q2.x; v[slot][tb][1] = q2.y;
      }
    }
  };
  // input c (0..3) of token block tb in slot `slot`, widened exactly to fp32
  auto xin = [&](int slot, int tb, int c) -> float {
    if constexpr (XT == DT_F32) return __uint_as_float(v[slot][tb][c]);
    const uint32_t q = v[slot][tb][c >> 1];
    return __uint_as_float((c & 1) ? (q & 0xFFFF0000u) : (q << 16));
  };
  // one column of the quad at a time over all 4 x RB accumulators, so that consecutive matrix-core
  // instructions never wait on each other's result (each accumulator still takes its columns in order)
  auto mma = [&](int slot) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int b = 0; b < RB; ++b) {
          const float wc = c == 0 ? w[slot][b].x : c == 1 ? w[slot][b].y : c == 2 ? w[slot][b].z : w[slot][b].w;
          acc[tb][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(xin(slot, tb, c), wc, acc[tb][b], 0, 0, 0);
        }
  };
  const int steps = ks / 16;   // a multiple of PF or below it (ks = d / n_split, d % 16 == 0)
  // the first PF steps' loads, unconditional like every other load (a step past the slice loads the
  // slice's last columns again, never used)
#pragma unroll
  for (int j = 0; j < PF; ++j) load(j, 16 * min(j, steps - 1));
  // every step but the last PF loads the step PF ahead, with no branch around the loads (a load
  // behind a branch makes the compiler wait for every load in flight before the next step's work)
  int j0 = 0;
  for (; j0 + PF < steps; j0 += PF) {
#pragma unroll
    for (int j = 0; j < PF; ++j) {
      mma(j);
      load(j, 16 * (j0 + j + PF));
      __builtin_amdgcn_sched_barrier(0);   // keeps the scheduler from moving later steps above the loads
    }
  }
#pragma unroll
  for (int j = 0; j < PF; ++j)
    if (j0 + j < steps) mma(j);
  float* out = partial + static_cast<size_t>(q) * T * N;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const int blk = wave + 4 * b;
    if (blk >= nb) break;
#pragma unroll
    for (int tb = 0; tb < 4; ++tb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + 16 * tb + 4 * g + i;
        if (t < T) out[static_cast<size_t>(t) * N + 16 * blk + r] = acc[tb][b][i];
      }
  }
}

// Selection (select.hpp) of the workgroup's four tokens; wave w, lane j < k writes rank j of
// token blockIdx.x * 4 + w.  The indices can also be published to host-coherent memory as 64-bit
// (seq << 32 | id) words: the host knows an entry is current from its tag alone, so it needs no
// copy, event or fence to read them.
__global__ void __launch_bounds__(256) router_select_kernel(const float* __restrict__ logits, int n_split, int T,
                                                            int N, int k, int route, int n_groups, int topk_groups,
                                                            int32_t* __restrict__ idx, float* __restrict__ w,
                                                            uint64_t* __restrict__ idx_host, uint32_t seq) {
  __shared__ SelectShared sh;
  select_tokens(logits, 0, blockIdx.x * 4, T, N, k, route, n_groups, topk_groups, sh, n_split,
                static_cast<size_t>(T) * N);
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
// logit row e (router_row: the arithmetic of router_logits_wide_kernel) and publishes it as tagged words
// (tag_logit, one atomic store each); workgroup 0, after its own row, selects on the complete logits,
// reading each word until it carries this launch's tag, and writes idx, w and, if asked, the tagged ids
// for the host.  The other workgroups wait for nothing, and the tags (atomic accesses to one location
// are coherent) make workgroup 0 read this launch's logits with no ordering between locations.
template <int XT>
__global__ void __launch_bounds__(256) route_select_kernel(const float* __restrict__ wr, const void* __restrict__ x,
                                                           int d, uint64_t* __restrict__ logits, uint32_t tag, int T,
                                                           int N, int k, int route, int n_groups, int topk_groups,
                                                           int32_t* __restrict__ idx, float* __restrict__ w,
                                                           uint64_t* __restrict__ idx_host, uint32_t seq) {
  __shared__ SelectShared sh;
  __shared__ float part[4][4];
  const int e = blockIdx.x;
  const float z = router_row<XT>(wr, x, 0, T, d, e, part);
  if (static_cast<int>(threadIdx.x) < T)
    __hip_atomic_store(logits + static_cast<size_t>(threadIdx.x) * N + e, tag_logit(tag, z), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  if (e != 0) return;
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
                               int T, int N, int k, int route, int n_groups, int topk_groups,
                               int32_t* idx, float* w, uint64_t* idx_host, uint32_t seq, hipStream_t st,
                               const LaunchTiming& tm) {
  if (T < 1 || T > 4 || N < 1 || N > 256 || k < 1 || k > 8 || d % 4 != 0 ||
      (route == R_SIGMOID_GROUP && (n_groups > 32 || N % n_groups != 0)))
    return hipErrorInvalidValue;
  if (x_dtype == DT_F32)
    hipExtLaunchKernelGGL(route_select_kernel<DT_F32>, dim3(N), dim3(256), 0, st, tm.start, tm.stop, 0, wr, x, d, logits,
                          tag, T, N, k, route, n_groups, topk_groups, idx, w, idx_host, seq);
  else
    hipExtLaunchKernelGGL(route_select_kernel<DT_BF16>, dim3(N), dim3(256), 0, st, tm.start, tm.stop, 0, wr, x, d,
                          logits, tag, T, N, k, route, n_groups, topk_groups, idx, w, idx_host, seq);
  return hipGetLastError();
}

hipError_t launch_router_logits(const float* wr, const void* x, int x_dtype, int T, int N, int d, float* logits,
                                int* n_split, hipStream_t st, const LaunchTiming& tm) {
  *n_split = 1;
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
  if (N % 16 == 0 && N <= 256 && d % 16 == 0) {
    // enough (token block, column slice) workgroups to give every CU one, at most kRouterMaxSplit slices
    const int tiles = (T + 63) / 64;
    int S = 1;
    while (2 * S <= kRouterMaxSplit && 2 * tiles * S <= 256 && d % (32 * S) == 0 &&
           ((d / (2 * S)) / 16 % 4 == 0 || (d / (2 * S)) / 16 < 4))
      S *= 2;
    *n_split = S;
    dim3 grid(tiles, S), block(256);
    const int ks = d / S;
    using K = void (*)(const float*, const void*, int, int, int, int, float*);
    K kern = nullptr;
    const int rb = (N / 16 + 3) / 4;
    if (x_dtype == DT_F32)
      kern = rb == 1 ? &router_logits_split_kernel<DT_F32, 1> : rb == 2 ? &router_logits_split_kernel<DT_F32, 2>
           : rb == 3 ? &router_logits_split_kernel<DT_F32, 3> : &router_logits_split_kernel<DT_F32, 4>;
    else
      kern = rb == 1 ? &router_logits_split_kernel<DT_BF16, 1> : rb == 2 ? &router_logits_split_kernel<DT_BF16, 2>
           : rb == 3 ? &router_logits_split_kernel<DT_BF16, 3> : &router_logits_split_kernel<DT_BF16, 4>;
    hipExtLaunchKernelGGL(kern, grid, block, 0, st, tm.start, tm.stop, 0, wr, x, T, N, d, ks, logits);
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

hipError_t launch_router_select(const float* logits, int n_split, int T, int N, int k, int route, int n_groups,
                                int topk_groups, int32_t* idx, float* w, uint64_t* idx_host, uint32_t seq,
                                hipStream_t st, const LaunchTiming& tm) {
  if (T <= 0) return hipSuccess;
  if (N > 256 || k > 8 || k < 1 || (route == R_SIGMOID_GROUP && (n_groups > 32 || N % n_groups != 0)))
    return hipErrorInvalidValue;
  dim3 grid((T + 3) / 4), block(256);
  if (n_split < 1 || n_split > kRouterMaxSplit) return hipErrorInvalidValue;
  hipExtLaunchKernelGGL(router_select_kernel, grid, block, 0, st, tm.start, tm.stop, 0, logits, n_split, T, N, k,
                        route, n_groups, topk_groups, idx, w, idx_host, seq);
  return hipGetLastError();
}

}  // namespace wisp
