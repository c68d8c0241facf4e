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
// The matrix cores run v_mfma_f32_32x32x16_bf16 with the token rows as the A operand (lane l holds
// row l%32, k 8*(l/32)..+7 of a 16-step), the weight rows as B (lane l holds weight row l%32, same k)
// and D lane l holding column l%32, rows 8*(r/4) + 4*(l/32) + r%4.  Every output element is one
// fixed-order reduction over K in ascending 16-steps, independent of where its row sits in a tile or
// which launch holds its expert, so paged and fully resident runs give identical bits.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>
#include <utility>

#include "kernels.hpp"

namespace wisp {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));   // a plain vector: stays in registers

constexpr uint32_t kOutOfRange = 0x80000000u;   // a byte offset past every resource below 2 GiB

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Stable counting sort of the pairs p = t*k + j by expert id idx[p] over segments of kPermSeg pairs:
// the count of each expert in each segment (permute_count_kernel, or, while those counts fit in LDS,
// every workgroup of the scatter kernel for itself from all the ids, so the sort is one launch); then
// permute_scatter_kernel (a workgroup of 16 waves per segment, 64 pairs per wave) places every pair at
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

constexpr int kPermFusedCounts = 8192;   // segments x experts counted in LDS by the one-launch sort

template <bool FUSED>
__global__ void __launch_bounds__(1024) permute_scatter_kernel(const int32_t* __restrict__ idx, int P, int N,
                                                               const int32_t* __restrict__ counts, int n_seg,
                                                               int32_t* __restrict__ perm,
                                                               uint64_t* __restrict__ totals, uint32_t seq) {
  __shared__ int32_t cnt[16][256];
  __shared__ int32_t base[256];
  __shared__ int32_t wsum[4];
  extern __shared__ int32_t hist[];   // FUSED: [n_seg][N] counts
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, seg = blockIdx.x;
  const int p = seg * kPermSeg + wave * 64 + lane;
  const bool valid = p < P;
  const int e = valid ? idx[p] : 0;
  for (int i = tid; i < 16 * 256; i += 1024) (&cnt[0][0])[i] = 0;
  if constexpr (FUSED) {
    // every pair once into its segment's count of its expert (integer adds: the same counts in any order)
    for (int i = tid; i < n_seg * N; i += 1024) hist[i] = 0;
    __syncthreads();
    for (int q0 = 0; q0 < P; q0 += 4 * 1024) {
      int ev[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {   // the loads go out together
        const int q = q0 + u * 1024 + tid;
        ev[u] = q < P ? idx[q] : -1;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (ev[u] >= 0) atomicAdd(&hist[((q0 + u * 1024 + tid) / kPermSeg) * N + ev[u]], 1);
    }
    __syncthreads();
  }
  // per expert: all its pairs (for the offsets) and those in earlier segments
  int tot = 0, before = 0;
  if (tid < N) {
    for (int q = 0; q < n_seg; ++q) {
      const int c = FUSED ? hist[q * N + tid] : counts[q * N + tid];
      tot += c;
      before += q < seg ? c : 0;
    }
    // the first segment's workgroup hands every expert's pair count to the host: one word per
    // expert with the call's sequence number above the count, by one atomic store
    if (totals && seg == 0)
      __hip_atomic_store(totals + tid, (static_cast<uint64_t>(seq) << 32) | static_cast<uint32_t>(tot),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
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

// ------------------------------------------------------------------------------------------
// The GEMM kernels are persistent: one 512-thread workgroup per CU walks its share of the tiles, and
// the K stages of all its tiles form one sequence, so the loads of the next tile's first stages are
// in flight while the current tile finishes (no pipeline start per tile).
//
// Weights (B operand: 256 weight rows x 64 K per stage, 32 KB) go from HBM straight into a ring of
// kNB LDS slots by buffer-to-LDS loads (buffer_load_dwordx4 ... lds), kNB - 1 stages ahead, so the
// bytes in flight do not occupy registers.  Inside a slot, 16-byte chunk c of weight row r sits at
// position c ^ swz(r), which keeps the fragment reads free of bank conflicts.  The token rows (A
// operand) are private to a wave (wave w owns rows 32 w .. 32 w + 31 of the row block): they are loaded
// into registers in the matrix cores' operand layout, the same kNB - 1 stages ahead (the vector-memory
// counter retires loads in issue order, so a shallower A prefetch would also retire the deeper weight
// loads early).  A weight fragment is read from LDS by an inline ds_read (the compiler then does not
// make the LDS reads wait for every buffer-to-LDS load in flight); the workgroup barrier is a plain
// s_barrier after an explicit wait for this stage's loads.
//
// Tiles: 128 h columns (W1 and W3 rows c0 .. c0 + 127, so SwiGLU is applied in registers) for gate/up,
// 256 output columns (W2 rows) for down, each over up to kRB = 256 rows of one expert: all of them at
// the routing's usual ~T k / N rows per expert, so each weight byte is read once and rows are padded
// only to the 32-row slab of a wave.  The wide tiles halve how often an expert's token rows are
// re-read (once per column tile) and how many tile ends there are.
// ------------------------------------------------------------------------------------------
constexpr int kRB = 256;                 // rows per row block: 8 slabs of 32, one per wave
constexpr int kGW = 8;                   // waves per workgroup
constexpr int kKS = 64;                  // K per stage
constexpr int kNB = 3;                   // LDS ring slots; loads run kNB - 1 stages ahead
constexpr int kD = kNB - 1;
constexpr int kBR = 256;                 // weight rows per tile (gate/up: 128 W1 + 128 W3 rows)
constexpr int kCB = kBR / 32;            // 32-column blocks per tile
constexpr int kSlot = kBR * kKS * 2;     // bytes per slot: 256 weight rows x 64 K, bf16
constexpr int kBI = kSlot / 1024 / kGW;  // buffer-to-LDS loads per wave per stage (1 KB each)
constexpr int kAI = kKS / 16;            // A fragment loads per wave per stage (16 B per lane each)
constexpr int MODE_UP = 0, MODE_DN = 1;
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// s_waitcnt immediate (gfx9 encoding) that waits for vector-memory count n only: vmcnt in bits 3:0
// and 15:14, expcnt (6:4) and lgkmcnt (11:8) left at their maximum.
constexpr int vmcnt_only(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// chunk swizzle of weight row r inside a slot: rows r .. r + 7 take distinct positions for one chunk,
// and so do the pairs (r & 1, position) of rows r .. r + 15
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Tile T of a launch -> its expert, row block and column tile.  Tiles run expert by expert, row block
// by row block, column tile fastest; gb.tile_end holds the cumulative row blocks per expert.
struct Tile {
  const uint8_t* w;
  int rows, base, m0, c0;
};
template <int MODE>
__device__ __forceinline__ Tile decode_tile(const GroupedBatch& gb, int T, int n_ct) {
  const int rb_all = T / n_ct, ct = T - rb_all * n_ct;
  int lo = 0, hi = gb.n_groups - 1;   // the first expert whose row blocks end past rb_all
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (rb_all >= gb.tile_end[mid]) lo = mid + 1;
    else hi = mid;
  }
  const int rb = rb_all - (lo > 0 ? gb.tile_end[lo - 1] : 0);
  return Tile{gb.w[lo], gb.rows[lo], gb.row_off[lo], rb * kRB, ct * (MODE == MODE_UP ? kBR / 2 : kBR)};
}

// The eight weight fragments (32-column blocks, 4 KB apart) of one 16-step of a slot, read by inline
// ds_reads from the lane's address in the slot.
__device__ __forceinline__ void read_frags(u32x4_t (&f)[kCB], uint32_t addr) {
  asm volatile(
      "ds_read_b128 %0, %8\n\t"
      "ds_read_b128 %1, %8 offset:4096\n\t"
      "ds_read_b128 %2, %8 offset:8192\n\t"
      "ds_read_b128 %3, %8 offset:12288\n\t"
      "ds_read_b128 %4, %8 offset:16384\n\t"
      "ds_read_b128 %5, %8 offset:20480\n\t"
      "ds_read_b128 %6, %8 offset:24576\n\t"
      "ds_read_b128 %7, %8 offset:28672\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(f[0]), "=&v"(f[1]), "=&v"(f[2]), "=&v"(f[3]), "=&v"(f[4]), "=&v"(f[5]), "=&v"(f[6]), "=&v"(f[7])
      : "v"(addr)
      : "memory");
}

// The A fragments of one stage: four 16-byte loads (the stage's four 16-steps) into registers, by
// inline asm so that the compiler neither counts them nor waits for them: the caller waits by count
// (every load of a stage is older than those of the stages after it) and then passes the registers
// through pin_frags, after which the compiler reads them.
__device__ __forceinline__ void load_a(u32x4_t (&a)[kAI], u32x4_t rs, uint32_t voff, uint32_t soff) {
  asm volatile(
      "buffer_load_dwordx4 %0, %4, %5, %6 offen\n\t"
      "buffer_load_dwordx4 %1, %4, %5, %6 offen offset:32\n\t"
      "buffer_load_dwordx4 %2, %4, %5, %6 offen offset:64\n\t"
      "buffer_load_dwordx4 %3, %4, %5, %6 offen offset:96"
      : "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3])
      : "v"(voff), "s"(rs), "s"(soff)
      : "memory");
}
__device__ __forceinline__ void pin_frags(u32x4_t (&a)[kAI]) {
  asm volatile("" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]));
}
// One int32 per lane, loaded the same way (waited for by count, then pinned).
__device__ __forceinline__ int32_t load_i32(const int32_t* p) {
  int32_t v;
  asm volatile("global_load_dword %0, %1, off" : "=&v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ void pin_i32(int32_t& v) { asm volatile("" : "+v"(v)); }
// raw buffer resource words (stride 0) over [p, p + bytes), as uniform values
__device__ __forceinline__ u32x4_t rsrc_words(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  u32x4_t r;
  r.x = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
  r.y = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32) & 0xFFFFu);
  r.z = __builtin_amdgcn_readfirstlane(bytes);
  r.w = 0x00020000u;
  return r;
}

template <int... Us, typename F>
__device__ __forceinline__ void ring_unroll(std::integer_sequence<int, Us...>, F&& f) {
  (f(std::integral_constant<int, Us>{}), ...);
}

template <int MODE>
__global__ void __launch_bounds__(512) grouped_kernel(GroupedBatch gb, const uint16_t* __restrict__ a_src,
                                                      uint32_t a_bytes, const int32_t* __restrict__ perm, int k,
                                                      int d, int I, void* __restrict__ out) {
  __shared__ __attribute__((aligned(1024))) uint8_t ring[kNB * kSlot];
  const int K = MODE == MODE_UP ? d : I;             // reduction length
  const int spt = K / kKS;                           // stages per tile
  const int n_ct = MODE == MODE_UP ? I / (kBR / 2) : d / kBR;
  const int n_tiles = gb.tile_end[gb.n_groups - 1] * n_ct;
  // XCD-aware: workgroups are dealt to the 8 XCDs round-robin, and the workgroups of one XCD take
  // consecutive logical indices, so at any time they work on consecutive tiles (the column tiles of
  // the same one to three experts, whose token rows then stay in that XCD's L2)
  const int G = static_cast<int>(gridDim.x);
  const int xcd = static_cast<int>(blockIdx.x) % 8, jx = static_cast<int>(blockIdx.x) / 8;
  const int L = xcd * (G / 8) + min(xcd, G % 8) + jx;
  const int my_tiles = (n_tiles - L + G - 1) / G;
  const int nq = my_tiles * spt;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, lr = lane & 31, hb = lane >> 5;
  const uint32_t wrow = static_cast<uint32_t>(K) * 2;   // bytes per weight row
  const uint32_t arow = static_cast<uint32_t>(K) * 2;   // bytes per A row (x: d, h: I)

  // buffer-to-LDS pattern: slot position p = (wave kBI + i) 64 + lane holds chunk (p & 7) ^ swz(row)
  // of weight row p >> 3 (gate/up: rows 0..127 are W1 rows c0.., 128..255 the W3 rows of the same
  // columns)
  uint32_t bpat[kBI];
#pragma unroll
  for (int i = 0; i < kBI; ++i) {
    const int pp = (wave * kBI + i) * 64 + lane, r = pp >> 3, c = (pp & 7) ^ swz(r);
    const int wr = MODE == MODE_UP ? (r < kBR / 2 ? r : I - kBR / 2 + r) : r;
    bpat[i] = static_cast<uint32_t>(wr) * wrow + c * 16;
  }
  // fragment reads: lane l reads weight row 32 cb + l % 32, chunk 2 kk + l / 32 of the 16-step pair
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)ring));
  uint32_t fo[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) fo[kk] = lds0 + lr * 128 + (((2 * kk + hb) ^ swz(lr)) << 4);
  const u32x4_t ar = rsrc_words(a_src, a_bytes);
  const uint32_t wbytes = static_cast<uint32_t>(I) * d * 2 * (MODE == MODE_UP ? 2 : 1);
  const size_t woff = MODE == MODE_UP ? 0 : static_cast<size_t>(2) * I * d * 2;   // W2 follows W1, W3

  // the issue cursor: the stage whose loads go out next
  int is_tile = 0, is_s = 0;
  __amdgpu_buffer_rsrc_t wr_rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a_src), 0, 0, 0x00020000);
  uint32_t bvo[kBI], avo = 0;
  // a lane's rows are read through the pair order: lane l holds the pair of row 32 wave + l % 32 of a
  // tile (its last row where the tile has fewer), loaded a whole tile ahead of its use and waited for
  // by count (all at once where a tile has fewer stages than the count covers)
  const bool short_k = spt < kD + 2;
  auto pair_of = [&](const Tile& t) __attribute__((always_inline)) -> int32_t {
    return load_i32(perm + t.base + min(t.m0 + wave * 32 + lr, t.rows - 1));
  };
  int32_t pn = 0;   // gate/up: the pair of this lane's row in the issue cursor's next tile
  auto enter_tile = [&](int i) __attribute__((always_inline)) {   // issue cursor enters its i-th tile
    const Tile t = decode_tile<MODE>(gb, L + i * G, n_ct);
    wr_rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(t.w + woff), 0, static_cast<int>(wbytes), 0x00020000);
#pragma unroll
    for (int j = 0; j < kBI; ++j) bvo[j] = bpat[j] + static_cast<uint32_t>(t.c0) * wrow;
    const int row = t.m0 + wave * 32 + lr;
    if constexpr (MODE == MODE_UP) {
      if (short_k) __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
      pin_i32(pn);
      avo = row < t.rows ? static_cast<uint32_t>(pn / k) * arow + hb * 16 : kOutOfRange;
      if (i + 1 < my_tiles) pn = pair_of(decode_tile<MODE>(gb, L + (i + 1) * G, n_ct));
    } else {
      avo = row < t.rows ? static_cast<uint32_t>(t.base + row) * arow + hb * 16 : kOutOfRange;
    }
  };
  u32x4_t A[kNB][kAI];
  auto issue = [&](int slot, u32x4_t (&a)[kAI]) __attribute__((always_inline)) {   // the loads of the issue cursor's stage
    if (is_s == 0) enter_tile(is_tile);
    const int sk = __builtin_amdgcn_readfirstlane(is_s * kKS * 2);
    load_a(a, ar, avo, sk);
#pragma unroll
    for (int j = 0; j < kBI; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr_rs, (lds_ptr_t)(ring + slot * kSlot + (wave * kBI + j) * 1024), 16,
                                               bvo[j], sk, 0, 0);
    if (++is_s == spt) {
      is_s = 0;
      ++is_tile;
    }
  };

  // the compute cursor
  int cs_tile = 0, cs_s = 0;
  Tile ct = decode_tile<MODE>(gb, L, n_ct);
  f32x16_t acc[kCB] = {};
  int32_t pq = 0;   // down: the pair of this lane's row in the compute cursor's tile
  if constexpr (MODE == MODE_UP) {
    pn = pair_of(ct);
    __builtin_amdgcn_s_waitcnt(vmcnt_only(0));   // nothing else is in flight yet
  } else {
    pq = pair_of(ct);
  }
  // Epilogue of a tile: each wave's 32 x 128 outputs (h columns for gate/up: silu(g) * u over the two
  // gate and up blocks), one column per lane as the matrix cores leave them.
  auto epilogue = [&]() __attribute__((always_inline)) {
    const int n_rows = ct.rows - ct.m0 - wave * 32;   // rows of this wave's slab in the tile (may be <= 0)
    if constexpr (MODE == MODE_UP) {
      uint16_t* hs = static_cast<uint16_t*>(out);
#pragma unroll
      for (int cb = 0; cb < kCB / 2; ++cb) {
        const int col = ct.c0 + cb * 32 + lr;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = (r >> 2) * 8 + hb * 4 + (r & 3);
          if (i < n_rows) {
            const float a = acc[cb][r];
            const float h = a / (1.0f + __expf(-a)) * acc[cb + kCB / 2][r];
            hs[static_cast<size_t>(ct.base + ct.m0 + wave * 32 + i) * I + col] = bf16_rne(h);
          }
        }
      }
    } else {
      uint16_t* buf = static_cast<uint16_t*>(out);
      if (short_k) __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
      pin_i32(pq);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = (r >> 2) * 8 + hb * 4 + (r & 3);
        const int p = __shfl(pq, i, 64);
        if (i < n_rows) {
          const size_t orow = static_cast<size_t>(p / k) * (k + 1) + (p % k);
#pragma unroll
          for (int cb = 0; cb < kCB; ++cb) buf[orow * d + ct.c0 + cb * 32 + lr] = bf16_rne(acc[cb][r]);
        }
      }
    }
  };

  // prologue: the first kD stages
#pragma unroll
  for (int u = 0; u < kD; ++u)
    if (u < nq) issue(u, A[u]);

  auto step = [&](auto U_, int q) __attribute__((always_inline)) {
    constexpr int U = decltype(U_)::value;   // q % kNB: the slot and the A register set
    // stage q's own loads (its A fragments, then this wave's share of the slot) have landed: the
    // operations issued after them are the loads of the kD - 1 later stages (fewer at the end of the
    // sequence: then everything), plus, after a tile's end, its stores and pair loads (the count then
    // waits a little longer than it must)
    if (is_tile * spt + is_s == q + kD)
      __builtin_amdgcn_s_waitcnt(vmcnt_only((kD - 1) * (kBI + kAI)));
    else
      __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
    pin_frags(A[U]);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();   // every wave's share landed; every wave is done with stage q - 1
    asm volatile("" ::: "memory");
    if (is_tile * spt + is_s < nq) issue((U + kD) % kNB, A[(U + kD) % kNB]);
    if (wave * 32 < ct.rows - ct.m0) {   // the wave's slab has rows in this tile
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        u32x4_t f[kCB];
        read_frags(f, fo[kk] + U * kSlot);
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, A[U][kk]);
#pragma unroll
        for (int cb = 0; cb < kCB; ++cb)
          acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8_t, f[cb]), acc[cb], 0, 0, 0);
      }
    }
    if (++cs_s == spt) {
      epilogue();
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) acc[cb] = f32x16_t{};
      cs_s = 0;
      if (++cs_tile < my_tiles) {
        ct = decode_tile<MODE>(gb, L + cs_tile * G, n_ct);
        if constexpr (MODE == MODE_DN) pq = pair_of(ct);
      }
    }
  };
  // the loop is unrolled over the ring, so that slots and register sets have fixed indices
  for (int q = 0; q < nq; q += kNB)
    ring_unroll(std::make_integer_sequence<int, kNB>{}, [&](auto U_) __attribute__((always_inline)) {
      if (q + decltype(U_)::value < nq) step(U_, q + decltype(U_)::value);
    });
}

}  // namespace

bool grouped_supported(const FfnShape& s, int has_shared) {
  return !has_shared && s.blob.w_dtype == DT_BF16 && s.x_dtype == DT_BF16 && s.h_dtype == DT_BF16 &&
         s.blob.d % kBR == 0 && s.blob.I % (kBR / 2) == 0;   // whole column tiles and K stages
}

int grouped_row_tiles(int rows) { return (rows + kRB - 1) / kRB; }

namespace {
// the buffer loads address x, h and an expert's weights by 32-bit byte offsets below kOutOfRange
bool offsets_fit(const FfnShape& s, int n_tok, int k) {
  const uint64_t lim = kOutOfRange;
  const uint64_t d = s.blob.d, I = s.blob.I;
  return n_tok >= 1 && k >= 1 && static_cast<uint64_t>(n_tok) * d * 2 < lim &&
         static_cast<uint64_t>(n_tok) * k * I * 2 < lim && 2 * I * d * 2 < lim &&
         static_cast<uint64_t>(n_tok) * (k + 1) * d * 4 < lim;
}
}  // namespace

int permute_segments(int n_pairs) { return (n_pairs + kPermSeg - 1) / kPermSeg; }

hipError_t launch_permute_pairs(const int32_t* idx, int n_pairs, int N, int32_t* perm, int32_t* counts, hipStream_t st,
                                const LaunchTiming& tm, uint64_t* totals, uint32_t seq) {
  if (n_pairs <= 0) return hipSuccess;
  if (N < 1 || N > 256) return hipErrorInvalidValue;
  const int n_seg = permute_segments(n_pairs);
  if (n_seg * N <= kPermFusedCounts) {   // one launch: each workgroup counts all the ids in LDS
    hipExtLaunchKernelGGL(permute_scatter_kernel<true>, dim3(n_seg), dim3(1024),
                          static_cast<uint32_t>(sizeof(int32_t) * n_seg * N), st, tm.start, tm.stop, 0, idx, n_pairs,
                          N, counts, n_seg, perm, totals, seq);
    return hipGetLastError();
  }
  hipExtLaunchKernelGGL(permute_count_kernel, dim3(n_seg), dim3(256), 0, st, tm.start, nullptr, 0, idx, n_pairs, N,
                        counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(permute_scatter_kernel<false>, dim3(n_seg), dim3(1024), 0, st, nullptr, tm.stop, 0, idx,
                        n_pairs, N, counts, n_seg, perm, totals, seq);
  return hipGetLastError();
}

namespace {
int compute_units() {
  static int cus = 0;
  if (!cus) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}
}  // namespace

hipError_t launch_grouped_gateup(const GroupedBatch& b, const FfnShape& s, const void* x, int n_tok,
                                 const int32_t* perm, int k, void* hs, hipStream_t st, const LaunchTiming& tm) {
  if (b.n_groups <= 0) return hipSuccess;
  if (b.n_groups > kMaxGroups || !grouped_supported(s, 0) || !offsets_fit(s, n_tok, k)) return hipErrorInvalidValue;
  const int tiles = b.tile_end[b.n_groups - 1] * (s.blob.I / (kBR / 2));
  const uint32_t x_bytes = static_cast<uint32_t>(n_tok) * s.blob.d * 2;
  hipExtLaunchKernelGGL(grouped_kernel<MODE_UP>, dim3(std::min(tiles, compute_units())), dim3(512), 0, st, tm.start,
                        tm.stop, 0, b, static_cast<const uint16_t*>(x), x_bytes, perm, k, s.blob.d, s.blob.I, hs);
  return hipGetLastError();
}

hipError_t launch_grouped_down(const GroupedBatch& b, const FfnShape& s, const void* hs, int n_tok, const int32_t* perm,
                               int k, uint16_t* buf, hipStream_t st, const LaunchTiming& tm) {
  if (b.n_groups <= 0) return hipSuccess;
  if (b.n_groups > kMaxGroups || !grouped_supported(s, 0) || !offsets_fit(s, n_tok, k)) return hipErrorInvalidValue;
  const int tiles = b.tile_end[b.n_groups - 1] * (s.blob.d / kBR);
  const uint32_t hs_bytes = static_cast<uint32_t>(n_tok) * k * s.blob.I * 2;
  hipExtLaunchKernelGGL(grouped_kernel<MODE_DN>, dim3(std::min(tiles, compute_units())), dim3(512), 0, st, tm.start,
                        tm.stop, 0, b, static_cast<const uint16_t*>(hs), hs_bytes, perm, k, s.blob.d, s.blob.I,
                        static_cast<void*>(buf));
  return hipGetLastError();
}

}  // namespace wisp
