// Internal interface between the pager (host C++) and the HIP kernels for gfx950.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace wisp {

// Element formats (same codes as wisp_dtype).
enum : int { DT_F32 = 0, DT_BF16 = 1, DT_FP8 = 2 };

// Bytes of the expert blob and offsets of its parts (W1 | W3 | W2 [| S1 | S3 | S2]).
struct BlobLayout {
  int d = 0, I = 0, w_dtype = 0;
  size_t elem = 0;          // bytes per stored weight element (4, 2, 1)
  size_t off_w1 = 0, off_w3 = 0, off_w2 = 0;
  size_t off_s1 = 0, off_s3 = 0, off_s2 = 0;  // fp8 scales (bf16)
  size_t bytes = 0;
};
BlobLayout make_blob_layout(int d, int I, int w_dtype);

// One unit of expert-FFN work: an expert blob (already in HBM) and up to kMaxTokPerItem tokens
// that chose it.  out[t] is the row of the h / buf scratch that receives token tok[t]'s result
// (row = token * (k + 1) + rank; rank k is the shared expert).
constexpr int kMaxTokPerItem = 4;
constexpr int kMaxItems = 40;

struct FfnItem {
  const uint8_t* w;      // the expert's blob in its HBM slot (or the shared expert's slab)
  const uint8_t* src;    // device-planned launches, faulted expert: its pinned host master
  int32_t ntok;
  int32_t fault;         // device-planned launches: 1 = stream from src into w while computing
  int32_t tok[kMaxTokPerItem];
  int32_t out[kMaxTokPerItem];
};

// The device-side expert map of one launch: passed by value as a kernel argument by the host
// pager, or written to HBM by the device pager.
struct FfnBatch {
  FfnItem items[kMaxItems];
  int32_t n_items;
  int32_t max_ntok;
};

struct FfnShape {
  BlobLayout blob;
  int x_dtype;     // DT_F32 or DT_BF16 input rows
  int h_dtype;     // DT_F32 (fp32 models) or DT_BF16 (h rounded to bf16 between the GEMVs)
};

// Timing hook: if ev0/ev1 are non-null they bracket the launch (hipExtLaunchKernel events).
struct LaunchTiming {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// Phase 1: h[out] = silu(W1 x[tok]) * (W3 x[tok]) for every item/token; h row stride = I.
hipError_t launch_ffn_gateup(const FfnBatch& b, const FfnShape& s, const void* x, void* h, hipStream_t st,
                             const LaunchTiming& tm);
// Phase 2: buf[out] = W2 h[out]; buf row stride = d (fp32).
hipError_t launch_ffn_down(const FfnBatch& b, const FfnShape& s, const void* h, float* buf, hipStream_t st,
                           const LaunchTiming& tm);
// Down projection fused with the combine, one token (bf16 weights and h): for the items (an expert
// blob and the output row `rank`: its rank j < k, or k for the shared expert), o_rank = W2 h[rank]
// and y = sum_j gates[j] o_j (j ascending) + o_k if has_shared, with the bits of launch_ffn_down +
// launch_combine.  The items must cover every rank 0..k-1 (and k with the shared expert).
struct FusedT1Items {
  const uint8_t* w[kMaxItems];
  int32_t rank[kMaxItems];
  int32_t n_items;
};
bool down_combine_supported(const FfnShape& s);
hipError_t launch_down_combine_t1(const FusedT1Items& items, const FfnShape& s, const void* h, const float* gates,
                                  float* y, int k, int has_shared, hipStream_t st, const LaunchTiming& tm);
// The same over the device pager's plan (single-token items; out[0] is the rank).
hipError_t launch_down_combine_dev(const FfnBatch* plan, int max_items, const FfnShape& s, const void* h,
                                   const float* gates, float* y, int k, int has_shared, hipStream_t st,
                                   const LaunchTiming& tm);

// Device-planned FFN of one layer-step (plan written to HBM by the device pager): gate/up, with
// faulted experts streamed from their pinned masters into their slots by the same kernel, then (if
// with_down) down into buf for the caller's combine.  max_items bounds the plan (T*k + shared).
hipError_t launch_ffn_dev(const FfnBatch* plan, int max_items, const FfnShape& s, const void* x, void* h,
                          float* buf, bool with_down, hipStream_t st, const LaunchTiming& tm_gateup,
                          const LaunchTiming& tm_down);
bool ffn_dev_supported(const FfnShape& s, int T, int k, int has_shared);

// y[t] = sum_j w[t, j] buf[t*(k+1)+j] (j ascending) + (shared ? buf[t*(k+1)+k] : 0).
hipError_t launch_combine(int T, int k, int d, int has_shared, const float* w, const float* buf, float* y,
                          hipStream_t st, const LaunchTiming& tm);
// The same sum over bf16 expert outputs (the grouped GEMMs' rows; no shared expert).
hipError_t launch_combine_bf16(int T, int k, int d, const float* w, const uint16_t* buf, float* y, hipStream_t st,
                               const LaunchTiming& tm);

// Token batches (prefill): grouped GEMMs on the matrix cores over slot-indirected experts.
// The (token, rank) pairs p = t*k + j are ordered by expert (stable); expert g of a launch owns
// rows [row_off, row_off + rows) of that order.  Up to kMaxGroups experts per launch (the batch is a
// 2.5 KB kernel argument).
constexpr int kMaxGroups = 128;
constexpr int kGroupedMinTokens = 16;   // token batches from this size take the grouped GEMMs
struct GroupedBatch {
  const uint8_t* w[kMaxGroups];   // the expert's blob in its HBM slot
  int32_t row_off[kMaxGroups];    // first row of the expert in the expert-sorted pair order
  int32_t rows[kMaxGroups];       // pairs routed to the expert (>= 1)
  int32_t tile_end[kMaxGroups];   // cumulative row-tile counts (grouped_row_tiles)
  int32_t n_groups;
};
bool grouped_supported(const FfnShape& s, int has_shared);
int grouped_row_tiles(int rows);
// perm[off_e + i] = the i-th pair (ascending) routed to expert e; off_e = pairs of experts < e.
// counts: device scratch of permute_segments(n_pairs) * N int32.  If totals is not NULL (N words of
// host-coherent memory), totals[e] = seq << 32 | pairs routed to e, each written by one atomic store.
int permute_segments(int n_pairs);
hipError_t launch_permute_pairs(const int32_t* idx, int n_pairs, int N, int32_t* perm, int32_t* counts, hipStream_t st,
                                const LaunchTiming& tm, uint64_t* totals = nullptr, uint32_t seq = 0);
// hs[row] = bf16(silu(W1 x[t]) * (W3 x[t])) for every row of the batch's experts (row in sorted order);
// x holds n_tok token rows, hs n_tok * k pair rows.
hipError_t launch_grouped_gateup(const GroupedBatch& b, const FfnShape& s, const void* x, int n_tok,
                                 const int32_t* perm, int k, void* hs, hipStream_t st, const LaunchTiming& tm);
// buf[t*(k+1)+j] = bf16(W2 hs[row]) for the pair p = t*k+j of every row (bf16, as h is: the combine
// reads half the bytes).
hipError_t launch_grouped_down(const GroupedBatch& b, const FfnShape& s, const void* hs, int n_tok, const int32_t* perm,
                               int k, uint16_t* buf, hipStream_t st, const LaunchTiming& tm);

// Router: logits[t, e] = W_r[e] . x[t] (fp32 accumulate), written as *n_split partial sums over column
// slices (slice s at logits + s * T * N; 1 for decode sizes, at most kRouterMaxSplit), which the
// selection adds in slice order.  logits must hold kRouterMaxSplit * T * N floats.
constexpr int kRouterMaxSplit = 8;
hipError_t launch_router_logits(const float* wr, const void* x, int x_dtype, int T, int N, int d, float* logits,
                                int* n_split, hipStream_t st, const LaunchTiming& tm);
// Router selection: idx/w [T, k] by routing variant.  If idx_host is given, entry t*k+j of it (in
// host-coherent memory) also receives (seq << 32 | id) as one 64-bit store.
// Decode (T <= 4): router logits and selection in one launch (workgroup 0 selects once every row is
// published); the same ids, gates and tagged ids as launch_router_logits + launch_router_select.
// logits: [T, N] 64-bit words (at least 4 x N) where the rows are published tagged with `tag`, which
// must differ from the tag of the launch that last wrote them (a per-launch sequence number, never 0;
// the words start at 0).
hipError_t launch_route_select(const float* wr, const void* x, int x_dtype, int d, uint64_t* logits, uint32_t tag,
                               int T, int N, int k, int route, int n_groups, int topk_groups,
                               int32_t* idx, float* w, uint64_t* idx_host, uint32_t seq, hipStream_t st,
                               const LaunchTiming& tm);
hipError_t launch_router_select(const float* logits, int n_split, int T, int N, int k, int route, int n_groups,
                                int topk_groups, int32_t* idx, float* w, uint64_t* idx_host, uint32_t seq,
                                hipStream_t st, const LaunchTiming& tm);

// Device pager: selection of T <= 4 tokens + Algorithm 1 on the layer's slot table in HBM + the
// launch plan of the layer's FFN (one workgroup).  Requires T * k <= C.
hipError_t launch_select_page(const float* logits, int T, int N, int k, int route, int n_groups, int topk_groups,
                              int32_t* idx, float* w, int32_t* pi, int32_t* pinv, uint64_t* tau, uint64_t* clock,
                              int C, const uint64_t* slot_ptr, const uint8_t* master_base, uint64_t master_stride,
                              const uint8_t* shared_dev, int has_shared, FfnBatch* plan, uint32_t* stats,
                              hipStream_t st, const LaunchTiming& tm);

// Device pager, fused: the router logits of T <= 4 tokens (one workgroup per expert row, as
// launch_router_logits) and, in workgroup 0 once every row is published, launch_select_page's work.
// logits and tag as for launch_route_select.
hipError_t launch_route_page(const float* wr, const void* x, int x_dtype, int d, uint64_t* logits, uint32_t tag,
                             int T, int N, int k, int route, int n_groups, int topk_groups, int32_t* idx, float* w,
                             int32_t* pi, int32_t* pinv, uint64_t* tau, uint64_t* clock, int C,
                             const uint64_t* slot_ptr, const uint8_t* master_base, uint64_t master_stride,
                             const uint8_t* shared_dev, int has_shared, FfnBatch* plan, uint32_t* stats,
                             hipStream_t st, const LaunchTiming& tm);

// Diagnostics.
// Fills by the compute units: dst[i][0, bytes) <- src[i][0, bytes) for i < n, reading pinned host
// memory over the host link.  Up to kMaxFills blobs per launch.
constexpr int kMaxFills = 64;
struct FillList {
  const uint8_t* src[kMaxFills];
  uint8_t* dst[kMaxFills];
  int32_t n;
};
hipError_t launch_fill(const FillList& fl, uint64_t bytes, hipStream_t st, const LaunchTiming& tm);
hipError_t launch_hbm_copy(const void* src, void* dst, size_t bytes, hipStream_t st);
// A streaming read of `bytes` (a multiple of 16) from src; sink receives at most one word.
hipError_t launch_hbm_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t st);
// wgs workgroups of 256 threads, each wave 4 * iters bf16 32x32x16 matrix-core instructions on registers.
hipError_t launch_mfma_peak(int wgs, int iters, float* sink, hipStream_t st);
hipError_t launch_decode_fp8(const uint8_t* codes, float* out, int n, hipStream_t st);

}  // namespace wisp
