// Device-resident pager: the router's selection and Algorithm 1 of WiSP (Sec. 3.2) for one
// layer-step in one 256-thread workgroup, with the slot table (pi, pi^-1, tau, c) kept in HBM.
//
// The host pager needs the routed ids on the host before it can page (one device->host round
// trip per layer, then copies issued by the host).  Here the decision runs where the ids are
// produced, and its result is the launch plan of the layer's FFN: the expert map of this step
// (slot address per expert), which experts fault, and the host master each fault streams from.
// The FFN kernels read that plan from HBM, so a decode step is a fixed sequence of kernels with
// no host synchronisation.  The rule is the same as the host table's: the reference set R is the
// union of the tokens' selections (|R| <= C here); faults are R's absent ids in ascending order;
// victims are the slots whose occupant is not in R, by (tau asc, slot asc), empty slots first
// (tau = 0); fault i takes victim i; then c += 1 and every expert of R gets tick c.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "router_row.hpp"
#include "select.hpp"

namespace wisp {
namespace {

struct PagerShared {
  SelectShared s;
  int32_t pi[256];       // the layer's slot table, read once at kernel start
  int32_t pinv[256];
  uint64_t tau[256];
  uint64_t slot[256];
  uint64_t clock;
  uint64_t vkey[256];    // victim order key (tau << 8 | slot) of a candidate slot, ~0 otherwise
  uint8_t in_r[256];
  int32_t hits[32], hslot[32], faults[32], fslot[32], victim[32];
  int32_t nh, nf;
};

// The layer's slot table into LDS (it does not depend on the routing, so these reads can be issued
// before the logits are known).
__device__ __forceinline__ void load_table(PagerShared& sh, int N, int C, const int32_t* __restrict__ pi,
                                           const int32_t* __restrict__ pinv, const uint64_t* __restrict__ tau,
                                           const uint64_t* __restrict__ clock, const uint64_t* __restrict__ slot_ptr) {
  const int tid = threadIdx.x;
  if (tid < N) sh.pi[tid] = pi[tid];
  if (tid < C) {
    sh.pinv[tid] = pinv[tid];
    sh.tau[tid] = tau[tid];
    sh.slot[tid] = slot_ptr[tid];
  }
  if (tid == 0) sh.clock = *clock;
  sh.in_r[tid] = 0;
}

// The table entries of thread tid held in registers, so that loading them does not make the
// thread wait before its next loads are issued (an LDS store of a loaded value waits for the load).
struct TableRegs {
  int32_t pi, pinv;
  uint64_t tau, slot, clock;
};

__device__ __forceinline__ TableRegs load_table_regs(int N, int C, const int32_t* __restrict__ pi,
                                                     const int32_t* __restrict__ pinv,
                                                     const uint64_t* __restrict__ tau,
                                                     const uint64_t* __restrict__ clock,
                                                     const uint64_t* __restrict__ slot_ptr) {
  // every thread loads (indices clamped into the tables) and keeps only its own entries: with no
  // load behind a branch, the loads go out together and nothing waits for them here
  const int tid = threadIdx.x;
  const int ie = min(tid, N - 1), is = min(tid, C - 1);
  const int32_t v_pi = pi[ie], v_pinv = pinv[is];
  const uint64_t v_tau = tau[is], v_slot = slot_ptr[is], v_clock = *clock;
  TableRegs r;
  r.pi = tid < N ? v_pi : -1;
  r.pinv = tid < C ? v_pinv : -1;
  r.tau = tid < C ? v_tau : 0;
  r.slot = tid < C ? v_slot : 0;
  r.clock = tid == 0 ? v_clock : 0;
  return r;
}

__device__ __forceinline__ void store_table(PagerShared& sh, int N, int C, const TableRegs& r) {
  const int tid = threadIdx.x;
  if (tid < N) sh.pi[tid] = r.pi;
  if (tid < C) {
    sh.pinv[tid] = r.pinv;
    sh.tau[tid] = r.tau;
    sh.slot[tid] = r.slot;
  }
  if (tid == 0) sh.clock = r.clock;
  sh.in_r[tid] = 0;
}

// Selection, Algorithm 1 and the launch plan for one layer-step, by one workgroup whose table is in
// sh (load_table) and whose threads have not yet synchronised since.
template <bool TAGGED>
__device__ __forceinline__ void select_and_page(
    PagerShared& sh, const void* __restrict__ logits, uint32_t tag, int T, int N, int k, int route, int n_groups,
    int topk_groups,
    int32_t* __restrict__ idx, float* __restrict__ w, int32_t* __restrict__ pi, int32_t* __restrict__ pinv,
    uint64_t* __restrict__ tau, uint64_t* __restrict__ clock, int C, const uint8_t* master_base,
    uint64_t master_stride, const uint8_t* shared_dev, int has_shared, FfnBatch* __restrict__ plan,
    uint32_t* __restrict__ stats) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  select_tokens<TAGGED>(logits, tag, 0, T, N, k, route, n_groups, topk_groups, sh.s);   // ends with a barrier
  if (wave < T && lane < k) {
    idx[wave * k + lane] = sh.s.sel[wave][lane];
    w[wave * k + lane] = sh.s.gate[wave][lane];
  }
  // reference set R
  if (tid < T * k) sh.in_r[sh.s.sel[tid / k][tid % k]] = 1;
  __syncthreads();
  // resident (hit) and absent (fault) ids of R, ascending; victim candidates: slots whose
  // occupant is not in R (empty ones included)
  if (wave == 0) {
    int nh = 0, nf = 0;
    for (int base = 0; base < N; base += 64) {
      const int e = base + lane;
      const bool in = e < N && sh.in_r[e];
      const int s = in ? sh.pi[e] : -1;
      const bool hit = in && s >= 0, flt = in && s < 0;
      const uint64_t mh = __ballot(hit), mf = __ballot(flt);
      const uint64_t below = (1ull << lane) - 1ull;
      if (hit) {
        const int p = nh + __popcll(mh & below);
        sh.hits[p] = e;
        sh.hslot[p] = s;
      }
      if (flt) sh.faults[nf + __popcll(mf & below)] = e;
      nh += __popcll(mh);
      nf += __popcll(mf);
    }
    if (lane == 0) { sh.nh = nh; sh.nf = nf; }
  }
  // (tau, slot) packed into one key per slot (a tick never reaches 2^56 and slots are < 256), so the
  // victim order is plain unsigned order; non-candidates, and the padding up to a multiple of 16,
  // get the largest key
  const int c_pad = (C + 15) & ~15;
  if (tid < c_pad) {
    const int occ = tid < C ? sh.pinv[tid] : 0;
    const bool cand = tid < C && (occ < 0 || !sh.in_r[occ]);
    sh.vkey[tid] = cand ? (sh.tau[tid] << 8) | static_cast<uint64_t>(tid) : ~0ull;
  }
  __syncthreads();
  const int nh = sh.nh, nf = sh.nf;
  // victims: the nf smallest keys among the candidates, by ranks (branch-free broadcast reads)
  if (nf > 0 && tid < C) {
    const uint64_t kt = sh.vkey[tid];
    if (kt != ~0ull) {
      int rank = 0;
      for (int s2 = 0; s2 < c_pad; s2 += 16) {
#pragma unroll
        for (int q = 0; q < 16; ++q) rank += sh.vkey[s2 + q] < kt ? 1 : 0;
      }
      if (rank < nf) sh.victim[rank] = tid;
    }
  }
  __syncthreads();
  // fault i takes victim i (the victim's occupant leaves the map); every expert of R gets c + 1
  const uint64_t c1 = sh.clock + 1;
  if (tid < nf) {
    const int s = sh.victim[tid];
    const int old = sh.pinv[s];
    if (old >= 0) pi[old] = -1;
    pi[sh.faults[tid]] = s;
    pinv[s] = sh.faults[tid];
    tau[s] = c1;
    sh.fslot[tid] = s;
  }
  if (tid < nh) tau[sh.hslot[tid]] = c1;
  if (tid == 0) {
    *clock = c1;
    stats[0] = static_cast<uint32_t>(nh);
    stats[1] = static_cast<uint32_t>(nf);
    plan->n_items = nh + nf + (has_shared ? 1 : 0);
    plan->max_ntok = T;   // an upper bound: each token picks an expert at most once
  }
  __syncthreads();
  // launch plan: residents ascending, faults ascending, then the shared expert
  const int n_items = nh + nf + (has_shared ? 1 : 0);
  if (tid < n_items) {
    FfnItem& it = plan->items[tid];
    int e = -1, slot = -1, fault = 0;
    if (tid < nh) { e = sh.hits[tid]; slot = sh.hslot[tid]; }
    else if (tid < nh + nf) { e = sh.faults[tid - nh]; slot = sh.fslot[tid - nh]; fault = 1; }
    int n = 0;
    for (int t = 0; t < T; ++t) {
      int out = -1;
      if (e < 0) out = t * (k + 1) + k;   // shared expert, every token
      else
        for (int j = 0; j < k; ++j)
          if (sh.s.sel[t][j] == e) out = t * (k + 1) + j;
      if (out >= 0) {
        it.tok[n] = t;
        it.out[n] = out;
        ++n;
      }
    }
    for (int q = n; q < kMaxTokPerItem; ++q) { it.tok[q] = 0; it.out[q] = 0; }
    it.ntok = n;
    it.fault = fault;
    it.w = e < 0 ? shared_dev : reinterpret_cast<const uint8_t*>(sh.slot[slot]);
    it.src = fault ? master_base + static_cast<uint64_t>(e) * master_stride : nullptr;
  }
}

__global__ void __launch_bounds__(256) select_page_kernel(
    const float* __restrict__ logits, int T, int N, int k, int route, int n_groups, int topk_groups,
    int32_t* __restrict__ idx, float* __restrict__ w, int32_t* __restrict__ pi, int32_t* __restrict__ pinv,
    uint64_t* __restrict__ tau, uint64_t* __restrict__ clock, int C, const uint64_t* __restrict__ slot_ptr,
    const uint8_t* master_base, uint64_t master_stride, const uint8_t* shared_dev, int has_shared,
    FfnBatch* __restrict__ plan, uint32_t* __restrict__ stats) {
  __shared__ PagerShared sh;
  load_table(sh, N, C, pi, pinv, tau, clock, slot_ptr);
  select_and_page<false>(sh, logits, 0, T, N, k, route, n_groups, topk_groups, idx, w, pi, pinv, tau, clock, C,
                         master_base, master_stride, shared_dev, has_shared, plan, stats);
}

// Router logits, selection and Algorithm 1 of one layer-step in one launch.  Workgroup e computes logit
// row e (router_row, as the router kernel does) and publishes it as tagged words (tag_logit, one atomic
// store each); workgroup 0, which has loaded the slot table into registers before its row, then runs the
// selection and the pager on the complete logits, reading each word until it carries this launch's tag.
// The other workgroups wait for nothing.
template <int XT>
__global__ void __launch_bounds__(256) route_page_kernel(
    const float* __restrict__ wr, const void* __restrict__ x, int d, uint64_t* __restrict__ logits, uint32_t tag,
    int T, int N, int k, int route, int n_groups, int topk_groups,
    int32_t* __restrict__ idx, float* __restrict__ w, int32_t* __restrict__ pi, int32_t* __restrict__ pinv,
    uint64_t* __restrict__ tau, uint64_t* __restrict__ clock, int C, const uint64_t* __restrict__ slot_ptr,
    const uint8_t* master_base, uint64_t master_stride, const uint8_t* shared_dev, int has_shared,
    FfnBatch* __restrict__ plan, uint32_t* __restrict__ stats) {
  __shared__ PagerShared sh;
  __shared__ float part[4][4];
  const int e = blockIdx.x;
  if (e != 0) {
    const float z = router_row<XT>(wr, x, 0, T, d, e, part);
    if (static_cast<int>(threadIdx.x) < T)
      __hip_atomic_store(logits + static_cast<size_t>(threadIdx.x) * N + e, tag_logit(tag, z), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  // the table goes into registers first (its loads do not depend on the routing), the row loads follow
  // without waiting for it
  const TableRegs tab = load_table_regs(N, C, pi, pinv, tau, clock, slot_ptr);
  const float z = router_row<XT>(wr, x, 0, T, d, e, part);
  if (static_cast<int>(threadIdx.x) < T)
    __hip_atomic_store(logits + static_cast<size_t>(threadIdx.x) * N + e, tag_logit(tag, z), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  store_table(sh, N, C, tab);   // read after select_tokens' first barrier
  select_and_page<true>(sh, logits, tag, T, N, k, route, n_groups, topk_groups, idx, w, pi, pinv, tau, clock, C,
                        master_base, master_stride, shared_dev, has_shared, plan, stats);
}

}  // namespace

hipError_t launch_route_page(const float* wr, const void* x, int x_dtype, int d, uint64_t* logits, uint32_t tag,
                             int T,
                             int N, int k, int route, int n_groups, int topk_groups, int32_t* idx, float* w,
                             int32_t* pi, int32_t* pinv, uint64_t* tau, uint64_t* clock, int C,
                             const uint64_t* slot_ptr, const uint8_t* master_base, uint64_t master_stride,
                             const uint8_t* shared_dev, int has_shared, FfnBatch* plan, uint32_t* stats,
                             hipStream_t st, const LaunchTiming& tm) {
  if (T < 1 || T > 4 || N > 256 || C > 256 || k > 8 || T * k > 32 || T * k > C || d % 4 != 0 ||
      T * k + (has_shared ? 1 : 0) > kMaxItems)
    return hipErrorInvalidValue;
  if (x_dtype == DT_F32)
    hipExtLaunchKernelGGL(route_page_kernel<DT_F32>, dim3(N), dim3(256), 0, st, tm.start, tm.stop, 0, wr, x, d, logits,
                          tag, T, N, k, route, n_groups, topk_groups, idx, w, pi, pinv, tau, clock, C, slot_ptr,
                          master_base, master_stride, shared_dev, has_shared, plan, stats);
  else
    hipExtLaunchKernelGGL(route_page_kernel<DT_BF16>, dim3(N), dim3(256), 0, st, tm.start, tm.stop, 0, wr, x, d,
                          logits, tag, T, N, k, route, n_groups, topk_groups, idx, w, pi, pinv, tau, clock, C,
                          slot_ptr, master_base, master_stride, shared_dev, has_shared, plan, stats);
  return hipGetLastError();
}

hipError_t launch_select_page(const float* logits, int T, int N, int k, int route, int n_groups, int topk_groups,
                              int32_t* idx, float* w, int32_t* pi, int32_t* pinv, uint64_t* tau, uint64_t* clock,
                              int C, const uint64_t* slot_ptr, const uint8_t* master_base, uint64_t master_stride,
                              const uint8_t* shared_dev, int has_shared, FfnBatch* plan, uint32_t* stats,
                              hipStream_t st, const LaunchTiming& tm) {
  if (T < 1 || T > 4 || N > 256 || C > 256 || k > 8 || T * k > 32 || T * k > C ||
      T * k + (has_shared ? 1 : 0) > kMaxItems)
    return hipErrorInvalidValue;
  hipExtLaunchKernelGGL(select_page_kernel, dim3(1), dim3(256), 0, st, tm.start, tm.stop, 0, logits, T, N, k, route,
                        n_groups, topk_groups, idx, w, pi, pinv, tau, clock, C, slot_ptr, master_base, master_stride,
                        shared_dev, has_shared, plan, stats);
  return hipGetLastError();
}

}  // namespace wisp
