// Token-batch (prefill) expert FFN: grouped GEMMs on the bf16 matrix cores of gfx950 over
// slot-indirected experts (the FusedMoE call of WiSP Algorithm 1 for large token batches).
//
// With thousands of tokens per layer each expert sees ~T*k/N of them, so its weights are reused
// across many rows and the FFN is a set of small dense GEMMs, one per expert:
//   H_e = silu(X_e W1_e^T) * (X_e W3_e^T)     X_e: the rows of the tokens routed to e  [n_e, d]
//   O_e = H_e W2_e^T                                                                    [n_e, d]
// The (token, rank) pairs are first ordered by expert (permute_count_kernel + permute_scatter_kernel:
// a stable counting sort, so expert e owns rows [off_e, off_e + n_e) of the sorted order and, inside,
// its pairs ascend).  The GEMM kernels read the weights through the expert's slot address and gather or
// scatter rows through the permutation; H is kept in the sorted order (bf16, as in decode) and O
// lands in the per-(token, rank) rows that the combine reads.
//
// Tiles: 64 rows x 64 h-columns for gate/up (the B tile holds the matching 64 rows of W1 and of
// W3, so SwiGLU is applied in registers), 64 rows x 128 columns for down; K in stages of 64 through
// one LDS buffer with padded rows, the next two stages loaded into registers meanwhile (k_loop
// below), four workgroups per CU.  Four waves per
// workgroup, each a 32-row slab of the tile on v_mfma_f32_32x32x16_bf16 (A lane l holds row l%32,
// k 8*(l/32)..+7; B lane l holds column l%32, same k; D lane l holds column l%32, rows
// 8*(r/4) + 4*(l/32) + r%4).  Every output element is one
// fixed-order reduction over K, independent of where its row sits in a tile or which launch holds
// its expert, so paged and fully resident runs give identical bits.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace wisp {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));   // a plain vector: stays in registers

constexpr int GM = 64;          // rows (pairs) per tile
constexpr int GN_UP = 64;       // h columns per gate/up tile
constexpr int GN_DOWN = 128;    // output columns per down tile
constexpr int KS_UP = 64;       // K per LDS stage, gate/up (K = d): 27 KB of LDS per workgroup
constexpr int KS_DOWN = 64;     // K per LDS stage, down (K = I)
constexpr int kWgsPerCu = 4;    // occupancy the kernels are compiled for (≤ 128 registers per lane)

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Tile -> (group, row tile, column tile).  Workgroups are dealt to the 8 XCDs round-robin by
// blockIdx.x, and each XCD has its own L2; the logical tile order is remapped so that every XCD gets
// one contiguous run of logical tiles.  Logical tiles run expert by expert, and inside an expert
// column-tile-major: the 2-3 row tiles of a column tile are adjacent (they read the same weight rows
// at the same time), and an expert's gathered rows (≈0.5 MB) stay in the L2 across its column
// tiles.  Against row-tile-major order this cut the gate/up launch's fetched bytes from 1.56x to
// 1.17x the algorithmic bytes.
constexpr int kXcds = 8;
__device__ __forceinline__ void tile_of(const GroupedBatch& gb, int n_ctiles, int& g, int& mt, int& ct) {
  const int n = static_cast<int>(gridDim.x);
  const int xcd = static_cast<int>(blockIdx.x) % kXcds, j = static_cast<int>(blockIdx.x) / kXcds;
  const int q = n / kXcds, r = n % kXcds;
  const int logical = xcd * q + min(xcd, r) + j;   // a bijection of [0, n)
  const int mt_all = logical / n_ctiles;          // expert g owns logical tiles [t0, t_end) x n_ctiles
  int lo = 0, hi = gb.n_groups - 1;   // the first group whose tiles end past mt_all
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (mt_all >= gb.tile_end[mid]) lo = mid + 1;
    else hi = mid;
  }
  g = lo;
  const int t0 = g > 0 ? gb.tile_end[g - 1] : 0, n_mt = gb.tile_end[g] - t0;
  const int local = logical - t0 * n_ctiles;
  ct = local / n_mt;
  mt = local - ct * n_mt;
}

// Stable counting sort of the pairs p = t*k + j by expert id idx[p], in two launches over segments of
// kPermSeg pairs: permute_count_kernel counts each expert in each segment; permute_scatter_kernel (a
// workgroup of 16 waves per segment, 64 pairs per wave) places every pair at
//   (pairs of smaller experts) + (pairs of its expert in earlier segments)
//   + (pairs of its expert in earlier waves of its segment) + (earlier lanes of its wave with that expert),
// the last found by matching lanes with equal ids through eight ballots over the id bits.  The result
// is the unique stable order: the pairs of each expert in ascending pair order.
constexpr int kPermSeg = 1024;

__global__ void __launch_bounds__(256) permute_count_kernel(const int32_t* __restrict__ idx, int P, int N,
                                                            int32_t* __restrict__ counts) {
  __shared__ int32_t h[256];
  const int tid = threadIdx.x, seg = blockIdx.x;
  h[tid] = 0;
  __syncthreads();
  const int p0 = seg * kPermSeg;
  int ev[kPermSeg / 256];
#pragma unroll
  for (int i = 0; i < kPermSeg / 256; ++i) {   // the loads go out together
    const int p = p0 + i * 256 + tid;
    ev[i] = p < P ? idx[p] : -1;
  }
#pragma unroll
  for (int i = 0; i < kPermSeg / 256; ++i)
    if (ev[i] >= 0) atomicAdd(&h[ev[i]], 1);
  __syncthreads();
  if (tid < N) counts[seg * N + tid] = h[tid];
}

__global__ void __launch_bounds__(1024) permute_scatter_kernel(const int32_t* __restrict__ idx, int P, int N,
                                                               const int32_t* __restrict__ counts, int n_seg,
                                                               int32_t* __restrict__ perm) {
  __shared__ int32_t cnt[16][256];
  __shared__ int32_t base[256];
  __shared__ int32_t wsum[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, seg = blockIdx.x;
  const int p = seg * kPermSeg + wave * 64 + lane;
  const bool valid = p < P;
  const int e = valid ? idx[p] : 0;
  for (int i = tid; i < 16 * 256; i += 1024) (&cnt[0][0])[i] = 0;
  // per expert: all its pairs (for the offsets) and those in earlier segments
  int tot = 0, before = 0;
  if (tid < N) {
    for (int q = 0; q < n_seg; ++q) {
      const int c = counts[q * N + tid];
      tot += c;
      before += q < seg ? c : 0;
    }
  }
  // exclusive scan of the totals over experts: an inclusive scan per wave (threads 0..255), then the
  // totals of the waves before
  int x = tot;
  if (tid < 256) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(x, off, 64);
      if (lane >= off) x += y;
    }
    if (lane == 63) wsum[wave] = x;
  }
  __syncthreads();
  if (tid < 256) {
    for (int w = 0; w < wave; ++w) x += wsum[w];
    base[tid] = x - tot + before;
  }
  // lanes of this wave with the same expert, and the rank among them
  uint64_t same = __ballot(valid);
#pragma unroll
  for (int bi = 0; bi < 8; ++bi) {
    const bool bit = (e >> bi) & 1;
    const uint64_t m = __ballot(bit);
    same &= bit ? m : ~m;
  }
  const uint64_t below = (1ull << lane) - 1ull;
  if (valid && (same & below) == 0) cnt[wave][e] = __popcll(same);
  __syncthreads();
  // per expert: the counts of the waves to exclusive offsets inside the segment
  if (tid < N) {
    int run = 0;
    for (int w = 0; w < 16; ++w) {
      const int c = cnt[w][tid];
      cnt[w][tid] = run;
      run += c;
    }
  }
  __syncthreads();
  if (valid) perm[base[e] + cnt[wave][e] + __popcll(same & below)] = p;
}

// One K stage of a 64-row A tile and a 128-row B tile through LDS.  A thread loads 16-byte pieces
// of TPR-thread row segments (KS bf16 = 2*KS contiguous bytes of a row per stage: whole 128-byte
// lines for KS = 64).  Loads are buffer loads: one uniform resource per operand (base and size in
// scalar registers), a 32-bit byte offset per piece and the stage's K offset as the scalar offset,
// which keeps the per-thread address state to one register per piece.  An A row past the expert's
// rows gets an offset beyond the resource's size, and the hardware's range check returns zeros for
// it without touching memory.  LDS holds one stage, rows padded by 16 bytes (the 16-byte reads of 16
// consecutive rows hit distinct banks).
template <int KS>
struct Stage {
  static constexpr int TPR = KS * 2 / 16;     // threads per row segment
  static constexpr int RPI = 256 / TPR;       // rows per load instruction
  static constexpr int AL = GM / RPI;         // A loads per thread
  static constexpr int BL = 128 / RPI;        // B loads per thread
  static constexpr int LDK = KS + 8;          // LDS row stride, bf16 elements
};

constexpr uint32_t kOutOfRange = 0x80000000u;   // a byte offset past every resource below 2 GiB

__device__ __forceinline__ __amdgpu_buffer_rsrc_t operand(const void* base, uint32_t bytes) {
  // raw (stride 0) resource over [base, base + bytes); the third word is the gfx9 data format 32
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}

template <int KS>
__device__ __forceinline__ void stage_load(__amdgpu_buffer_rsrc_t ar, const uint32_t* a_off, __amdgpu_buffer_rsrc_t br,
                                           const uint32_t* b_off, int kb, u32x4_t* ra, u32x4_t* rb) {
  const int sk = __builtin_amdgcn_readfirstlane(kb * 2);   // uniform: the scalar offset, not a per-lane one
#pragma unroll
  for (int i = 0; i < Stage<KS>::AL; ++i) ra[i] = __builtin_amdgcn_raw_buffer_load_b128(ar, a_off[i], sk, 0);
#pragma unroll
  for (int i = 0; i < Stage<KS>::BL; ++i) rb[i] = __builtin_amdgcn_raw_buffer_load_b128(br, b_off[i], sk, 0);
}

template <int KS>
__device__ __forceinline__ void stage_store(uint16_t* As, uint16_t* Bs, int tr, int tq, const u32x4_t* ra,
                                            const u32x4_t* rb) {
  using S = Stage<KS>;
#pragma unroll
  for (int i = 0; i < S::AL; ++i) *reinterpret_cast<u32x4_t*>(&As[(tr + S::RPI * i) * S::LDK + tq]) = ra[i];
#pragma unroll
  for (int i = 0; i < S::BL; ++i) *reinterpret_cast<u32x4_t*>(&Bs[(tr + S::RPI * i) * S::LDK + tq]) = rb[i];
}

// The K loop of a tile (nk stages, nk even and >= 2).  LDS holds stage s while stages s + 1 and
// s + 2 are in flight in two register sets, so a global load has two stages of MFMA work to arrive
// in; with one stage in flight the loop waited on load latency (a stage took ≈2 µs against ≈0.3 µs
// of matrix-core work).  A register set is stored to LDS only after its own loads, and the next
// loads into it are issued right after the store.  Every load in the loop is unconditional and the
// last four stages are peeled (nk = 2, SHORT, is an instantiation of its own): then each store waits only for its own set's loads (the other set's
// six stay in flight), and the loop has one exit, so the accumulators keep one set of registers.
// compute() runs the MFMAs of the stage in LDS.
template <int KS, bool SHORT, typename F>
__device__ __forceinline__ void k_loop(int nk, __amdgpu_buffer_rsrc_t ar, const uint32_t* a_off,
                                       __amdgpu_buffer_rsrc_t br, const uint32_t* b_off, uint16_t* As, uint16_t* Bs,
                                       int tr, int tq, F&& compute) {
  using S = Stage<KS>;
  u32x4_t ra0[S::AL], rb0[S::BL], ra1[S::AL], rb1[S::BL];
  auto load0 = [&](int st) { stage_load<KS>(ar, a_off, br, b_off, st * KS, ra0, rb0); };
  auto load1 = [&](int st) { stage_load<KS>(ar, a_off, br, b_off, st * KS, ra1, rb1); };
  auto store0 = [&]() { __syncthreads(); stage_store<KS>(As, Bs, tr, tq, ra0, rb0); __syncthreads(); };
  auto store1 = [&]() { __syncthreads(); stage_store<KS>(As, Bs, tr, tq, ra1, rb1); __syncthreads(); };
  load0(0);
  load1(1);
  stage_store<KS>(As, Bs, tr, tq, ra0, rb0);
  __syncthreads();
  if constexpr (SHORT) {   // nk = 2 (a short K, such as I = 128 in the down GEMM)
    compute();
    store1();
    compute();
  } else {
    load0(2);
    int s = 0;
    for (; s + 4 < nk; s += 2) {
      compute();     // stage s
      store1();      // stage s + 1
      load1(s + 3);
      compute();
      store0();      // stage s + 2
      load0(s + 4);
    }
    compute();       // stage nk - 4
    store1();
    load1(nk - 1);
    compute();       // nk - 3
    store0();
    compute();       // nk - 2
    store1();
    compute();       // nk - 1
  }
}

// H rows [off_g + m0, +64) x h columns [c0, +64) of one expert: silu(X W1^T) * (X W3^T) -> bf16.
// The B tile's rows 0..63 are W1 rows c0.., rows 64..127 the W3 rows of the same columns.  x has
// x_bytes bytes (the token rows).
template <int KS, bool SHORT>
__global__ void __launch_bounds__(256, kWgsPerCu) grouped_gateup_kernel(GroupedBatch gb, const uint16_t* __restrict__ x,
                                                                         uint32_t x_bytes,
                                                                         const int32_t* __restrict__ perm, int k, int d,
                                                                         int I, uint16_t* __restrict__ hs) {
  using S = Stage<KS>;
  __shared__ __attribute__((aligned(16))) uint16_t As[GM * S::LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2 * GN_UP * S::LDK];
  int g, mt, ct;
  tile_of(gb, I / GN_UP, g, mt, ct);
  const int rows = gb.rows[g], base = gb.row_off[g];
  const int m0 = mt * GM, c0 = ct * GN_UP;
  const int tid = threadIdx.x;
  const int tr = tid / S::TPR, tq = (tid % S::TPR) * 8;
  uint32_t a_off[S::AL];
#pragma unroll
  for (int i = 0; i < S::AL; ++i) {
    const int r = m0 + tr + S::RPI * i;
    a_off[i] = r < rows ? static_cast<uint32_t>(perm[base + r] / k) * d * 2 + tq * 2 : kOutOfRange;
  }
  uint32_t b_off[S::BL];
#pragma unroll
  for (int i = 0; i < S::BL; ++i) {
    const int j = tr + S::RPI * i;     // B tile row: W1 row c0 + j, or W3 row c0 + j - 64 (W3 follows W1)
    b_off[i] = static_cast<uint32_t>(j < GN_UP ? c0 + j : I + c0 + j - GN_UP) * d * 2 + tq * 2;
  }
  const __amdgpu_buffer_rsrc_t ar = operand(x, x_bytes);
  const __amdgpu_buffer_rsrc_t br = operand(gb.w[g], static_cast<uint32_t>(2 * I) * d * 2);
  const int wave = tid >> 6, lane = tid & 63, wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 31, fk = (lane >> 5) * 8;
  f32x16_t accg = {}, accu = {};
  k_loop<KS, SHORT>(d / KS, ar, a_off, br, b_off, As, Bs, tr, tq, [&]() {
#pragma unroll
    for (int kk = 0; kk < KS; kk += 16) {
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(&As[(wm * 32 + fr) * S::LDK + kk + fk]);
      const bf16x8_t bg = *reinterpret_cast<const bf16x8_t*>(&Bs[(wn * 32 + fr) * S::LDK + kk + fk]);
      const bf16x8_t bu = *reinterpret_cast<const bf16x8_t*>(&Bs[(GN_UP + wn * 32 + fr) * S::LDK + kk + fk]);
      accg = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bg, accg, 0, 0, 0);
      accu = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bu, accu, 0, 0, 0);
    }
  });
  const int hc = c0 + wn * 32 + fr;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
    if (m0 + i < rows) {
      const float a = accg[r];
      const float h = a / (1.0f + __expf(-a)) * accu[r];
      hs[static_cast<size_t>(base + m0 + i) * I + hc] = bf16_rne(h);
    }
  }
}

// O rows of one expert x output columns [c0, +128): H W2^T in fp32, scattered to the rows
// t*(k+1) + j of the pairs.  hs has hs_bytes bytes (the sorted pair rows).
template <int KS, bool SHORT>
__global__ void __launch_bounds__(256, kWgsPerCu) grouped_down_kernel(GroupedBatch gb, const uint16_t* __restrict__ hs,
                                                                       uint32_t hs_bytes,
                                                                       const int32_t* __restrict__ perm, int k, int d,
                                                                       int I, float* __restrict__ buf) {
  using S = Stage<KS>;
  __shared__ __attribute__((aligned(16))) uint16_t As[GM * S::LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[GN_DOWN * S::LDK];
  int g, mt, ct;
  tile_of(gb, d / GN_DOWN, g, mt, ct);
  const int rows = gb.rows[g], base = gb.row_off[g];
  const int m0 = mt * GM, c0 = ct * GN_DOWN;
  const int tid = threadIdx.x;
  const int tr = tid / S::TPR, tq = (tid % S::TPR) * 8;
  uint32_t a_off[S::AL];
#pragma unroll
  for (int i = 0; i < S::AL; ++i) {
    const int r = m0 + tr + S::RPI * i;
    a_off[i] = r < rows ? static_cast<uint32_t>(base + r) * I * 2 + tq * 2 : kOutOfRange;
  }
  uint32_t b_off[S::BL];
#pragma unroll
  for (int i = 0; i < S::BL; ++i) b_off[i] = static_cast<uint32_t>(c0 + tr + S::RPI * i) * I * 2 + tq * 2;
  const __amdgpu_buffer_rsrc_t ar = operand(hs, hs_bytes);
  const __amdgpu_buffer_rsrc_t br =
      operand(reinterpret_cast<const uint16_t*>(gb.w[g]) + 2 * static_cast<size_t>(I) * d, static_cast<uint32_t>(I) * d * 2);
  const int wave = tid >> 6, lane = tid & 63, wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 31, fk = (lane >> 5) * 8;
  f32x16_t acc0 = {}, acc1 = {};
  k_loop<KS, SHORT>(I / KS, ar, a_off, br, b_off, As, Bs, tr, tq, [&]() {
#pragma unroll
    for (int kk = 0; kk < KS; kk += 16) {
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(&As[(wm * 32 + fr) * S::LDK + kk + fk]);
      const bf16x8_t b0 = *reinterpret_cast<const bf16x8_t*>(&Bs[(wn * 64 + fr) * S::LDK + kk + fk]);
      const bf16x8_t b1 = *reinterpret_cast<const bf16x8_t*>(&Bs[(wn * 64 + 32 + fr) * S::LDK + kk + fk]);
      acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b1, acc1, 0, 0, 0);
    }
  });
  const int oc = c0 + wn * 64 + fr;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
    if (m0 + i < rows) {
      const int p = perm[base + m0 + i];
      const size_t orow = static_cast<size_t>(p / k) * (k + 1) + (p % k);
      buf[orow * d + oc] = acc0[r];
      buf[orow * d + oc + 32] = acc1[r];
    }
  }
}

}  // namespace

bool grouped_supported(const FfnShape& s, int has_shared) {
  return !has_shared && s.blob.w_dtype == DT_BF16 && s.x_dtype == DT_BF16 && s.h_dtype == DT_BF16 &&
         s.blob.d % GN_DOWN == 0 && s.blob.I % GN_UP == 0 &&
         s.blob.d % (2 * KS_UP) == 0 && s.blob.I % (2 * KS_DOWN) == 0;   // K loops take stages in pairs
}

int grouped_row_tiles(int rows) { return (rows + GM - 1) / GM; }

namespace {
// the buffer loads address x, h and an expert's weights by 32-bit byte offsets below kOutOfRange
bool offsets_fit(const FfnShape& s, int n_tok, int k) {
  const uint64_t lim = kOutOfRange;
  const uint64_t d = s.blob.d, I = s.blob.I;
  return n_tok >= 1 && k >= 1 && static_cast<uint64_t>(n_tok) * d * 2 < lim &&
         static_cast<uint64_t>(n_tok) * k * I * 2 < lim && 2 * I * d * 2 < lim;
}
}  // namespace

int permute_segments(int n_pairs) { return (n_pairs + kPermSeg - 1) / kPermSeg; }

hipError_t launch_permute_pairs(const int32_t* idx, int n_pairs, int N, int32_t* perm, int32_t* counts, hipStream_t st,
                                const LaunchTiming& tm) {
  if (n_pairs <= 0) return hipSuccess;
  if (N < 1 || N > 256) return hipErrorInvalidValue;
  const int n_seg = permute_segments(n_pairs);
  hipExtLaunchKernelGGL(permute_count_kernel, dim3(n_seg), dim3(256), 0, st, tm.start, nullptr, 0, idx, n_pairs, N,
                        counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(permute_scatter_kernel, dim3(n_seg), dim3(1024), 0, st, nullptr, tm.stop, 0, idx, n_pairs, N,
                        counts, n_seg, perm);
  return hipGetLastError();
}

hipError_t launch_grouped_gateup(const GroupedBatch& b, const FfnShape& s, const void* x, int n_tok,
                                 const int32_t* perm, int k, void* hs, hipStream_t st, const LaunchTiming& tm) {
  if (b.n_groups <= 0) return hipSuccess;
  if (b.n_groups > kMaxGroups || !grouped_supported(s, 0) || !offsets_fit(s, n_tok, k)) return hipErrorInvalidValue;
  const int tiles = b.tile_end[b.n_groups - 1] * (s.blob.I / GN_UP);
  const uint32_t x_bytes = static_cast<uint32_t>(n_tok) * s.blob.d * 2;
  auto* kern = s.blob.d == 2 * KS_UP ? grouped_gateup_kernel<KS_UP, true> : grouped_gateup_kernel<KS_UP, false>;
  hipExtLaunchKernelGGL(kern, dim3(tiles), dim3(256), 0, st, tm.start, tm.stop, 0, b,
                        static_cast<const uint16_t*>(x), x_bytes, perm, k, s.blob.d, s.blob.I,
                        static_cast<uint16_t*>(hs));
  return hipGetLastError();
}

hipError_t launch_grouped_down(const GroupedBatch& b, const FfnShape& s, const void* hs, int n_tok, const int32_t* perm,
                               int k, float* buf, hipStream_t st, const LaunchTiming& tm) {
  if (b.n_groups <= 0) return hipSuccess;
  if (b.n_groups > kMaxGroups || !grouped_supported(s, 0) || !offsets_fit(s, n_tok, k)) return hipErrorInvalidValue;
  const int tiles = b.tile_end[b.n_groups - 1] * (s.blob.d / GN_DOWN);
  const uint32_t hs_bytes = static_cast<uint32_t>(n_tok) * k * s.blob.I * 2;
  auto* kern = s.blob.I == 2 * KS_DOWN ? grouped_down_kernel<KS_DOWN, true> : grouped_down_kernel<KS_DOWN, false>;
  hipExtLaunchKernelGGL(kern, dim3(tiles), dim3(256), 0, st, tm.start, tm.stop, 0, b,
                        static_cast<const uint16_t*>(hs), hs_bytes, perm, k, s.blob.d, s.blob.I, buf);
  return hipGetLastError();
}

}  // namespace wisp
