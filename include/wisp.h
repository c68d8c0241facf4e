/*
 * wisp.h — C ABI of the paged MoE layer for AMD MI355X (gfx950).
 *
 * Implements the per-layer decode step of WiSP (arXiv 2606.21868): a routing-aware expert pager
 * over a slot-indirected expert FFN.  One layer-step is
 *   1. router scoring and top-k                    wisp_route_topk   (Sec. 3.1, selection of R)
 *   2. slot lookup, fault list, LRU victims        wisp_page_in      (Algorithm 1, faults/victims/assign)
 *   3. async host->device fills of the faults      wisp_page_in      (Algorithm 1, copy_async + map update)
 *   4. slot-indirected SwiGLU FFN + combine        wisp_moe_forward  (Algorithm 1, final FusedMoE call)
 * and the expert budget is set or resized with wisp_set_budget (cap C = B_exp / (L * M_e),
 * Sec. 3.1; resize at a drained barrier, keeping the prior state on failure, Sec. 3.5 and App. B).
 *
 * Conventions
 *  - Every call returns a wisp_status and never throws.  On error nothing has changed: arguments
 *    are validated before any state is touched, and resizes are transactional.  The message of
 *    the last error on the calling thread is returned by wisp_last_error().
 *  - A context is one model; it is not thread-safe.  All device pointers must belong to the
 *    device that was current at wisp_create.  `stream` arguments are hipStream_t handles passed
 *    as void* (NULL = the legacy default stream; a non-blocking stream is recommended).
 *  - The caller owns x, idx, w, y, the router weights and the streams.  The library owns the
 *    pinned host masters of every expert, the device expert slots, its internal side stream and
 *    events, and its scratch buffers.
 *  - Expert blob format (the unit that is paged; one contiguous blob per expert):
 *      W1 [I, d] row-major | W3 [I, d] row-major | W2 [d, I] row-major
 *    fp32 / bf16 store the elements; WISP_FP8E4M3_B128 stores OCP E4M3FN codes and appends
 *    bf16 scales S1 [I/128, d/128] | S3 [I/128, d/128] | S2 [d/128, I/128] (one per 128x128
 *    block); a weight is code * scale.  The expert computes o = W2 (silu(W1 x) * (W3 x)).
 */
#ifndef WISP_H
#define WISP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct wisp_ctx wisp_ctx;

typedef enum {
  WISP_OK = 0,
  WISP_E_INVAL = -1,        /* bad argument (range, shape, null pointer) */
  WISP_E_NOMEM = -2,        /* host or device allocation failed; state unchanged */
  WISP_E_HIP = -3,          /* a HIP runtime call failed */
  WISP_E_NOT_RESIDENT = -4, /* a routed expert is not resident when the FFN would run */
  WISP_E_STATE = -5         /* call out of order (no budget set, no pending page-in, ...) */
} wisp_status;

typedef enum {
  WISP_ROUTE_SOFTMAX_RENORM = 0, /* p = softmax(z) over all N, top-k of p, g = p_R / sum p_R */
  WISP_ROUTE_TOPK_SOFTMAX = 1,   /* top-k of z, g = softmax(z_R) */
  WISP_ROUTE_SIGMOID_GROUP = 2   /* s = sigmoid(z); groups of N/n_groups ids scored by their two
                                    largest s; keep topk_groups groups; top-k s; g = s_R / sum s_R */
} wisp_route;

typedef enum { WISP_F32 = 0, WISP_BF16 = 1, WISP_FP8E4M3_B128 = 2 } wisp_dtype;

typedef struct {
  int32_t n_layers;    /* L */
  int32_t d_model;     /* d */
  int32_t d_ff;        /* I, expert intermediate width */
  int32_t n_experts;   /* N routed experts per layer (<= 256) */
  int32_t top_k;       /* k (<= 8) */
  int32_t n_groups;    /* WISP_ROUTE_SIGMOID_GROUP only, else 1 */
  int32_t topk_groups; /* WISP_ROUTE_SIGMOID_GROUP only, else 1 */
  int32_t has_shared;  /* 1: every layer has one always-resident shared expert (weight 1) */
  int32_t route;       /* wisp_route */
  int32_t w_dtype;     /* wisp_dtype of expert weights */
  int32_t x_dtype;     /* WISP_F32 or WISP_BF16 hidden states */
  int32_t max_tokens;  /* largest T passed to route / forward */
  int32_t pageable_masters; /* 0: masters in pinned host memory (one DMA copy per fault).  1: masters
                             * in ordinary pageable memory, for master sets larger than the pinned
                             * memory a process may hold: faults are copied piece by piece through a
                             * small pinned bounce ring by host threads (wisp_page_in then blocks
                             * while it stages), and the device pager is not available. */
} wisp_model_desc;

typedef struct {
  uint32_t hits;      /* distinct routed experts already resident */
  uint32_t misses;    /* faults: experts copied host -> device */
  uint32_t chunks;    /* Algorithm 1 steps taken (more than one when the union exceeds C) */
  uint32_t steps;     /* layer-steps counted (cumulative statistics) */
  uint64_t h2d_bytes; /* misses * M_e */
} wisp_page_stats;

/* Bytes M_e of one expert blob for a description (weights + fp8 scales). */
wisp_status wisp_expert_bytes(const wisp_model_desc* desc, uint64_t* bytes);

/* Create a context on the current device: pinned host masters for every expert (and the shared
 * experts), the side stream and events, and scratch sized by max_tokens.  No expert slots exist
 * until wisp_set_budget.  The masters are uninitialised: fill them through wisp_expert_host_ptr
 * and then call wisp_masters_ready.  (Masters in pinned host memory: App. C.) */
wisp_status wisp_create(const wisp_model_desc* desc, wisp_ctx** out);

/* Wait for all outstanding work of the context and free everything it owns. */
wisp_status wisp_destroy(wisp_ctx* ctx);

/* Host address and size of expert `expert` of `layer` in the pinned masters (expert = -1: the
 * shared expert).  The caller writes the blob there before wisp_masters_ready. */
wisp_status wisp_expert_host_ptr(wisp_ctx* ctx, int32_t layer, int32_t expert, void** ptr, uint64_t* bytes);

/* Declare the masters final: copies the shared experts to their fixed device slab and drops every
 * resident expert so later faults re-read the masters: every layer's slot table restarts cold (all
 * slots empty, LRU clock at 0).  Synchronous. */
wisp_status wisp_masters_ready(wisp_ctx* ctx);

/* Router weights of `layer`: device pointer to W_r [N, d] fp32 row-major, caller-owned, valid
 * for the life of the context. */
wisp_status wisp_router_weights(wisp_ctx* ctx, int32_t layer, const float* w_r_dev);

/* Set the VRAM expert budget B_exp (bytes).  The per-layer cap becomes C = floor(B_exp / (L * M_e))
 * (Sec. 3.1); it must satisfy 1 <= C <= N.  Runs at a drained barrier: waits for every
 * outstanding fill and FFN of the context; fails with WISP_E_STATE if a page-in is pending.
 * Shrink keeps each layer's C most recently used experts (largest LRU tick, ties to the lower
 * slot), renumbers them in slot order and frees the rest first; grow allocates new empty slots.
 * Device footprint never exceeds max(old, new).  On failure (WISP_E_NOMEM) every layer keeps its
 * previous slots, tables and contents.  cap_out (optional) receives C. */
wisp_status wisp_set_budget(wisp_ctx* ctx, uint64_t expert_bytes, int32_t* cap_out);

/* Make experts 0 .. C-1 of every layer resident (one Algorithm 1 step per layer over those ids)
 * and wait for the copies.  With C = N this is the fully resident mode in which a run takes no
 * faults.  Not counted in the statistics. */
wisp_status wisp_preload(wisp_ctx* ctx);

/* Where Algorithm 1 runs.
 * WISP_PAGER_HOST (default): the slot table lives on the host; wisp_route_topk hands the routed
 *   ids to the host, wisp_page_in decides and issues hipMemcpyAsync fills on the side stream,
 *   wisp_moe_forward runs the FFN ordered after the fills by events.
 * WISP_PAGER_DEVICE: the slot table lives in HBM and a one-workgroup kernel runs the same rule
 *   right after the router, writing the launch plan of the layer's FFN to HBM; the gate/up
 *   kernel streams each faulted expert from its pinned host master over PCIe (computing with it
 *   and filling its slot in the same pass), so a decode step (wisp_decode_step) is a fixed kernel
 *   sequence with no host round trip.  Needs every layer-step to be one Algorithm 1 step
 *   (C >= max_tokens * k), max_tokens <= 4 and a supported layer shape; wisp_page_in and
 *   wisp_moe_forward are not available in this mode (WISP_E_STATE).
 * Switching drains the context and moves the tables; paging decisions and outputs are the same
 * in both modes. */
typedef enum { WISP_PAGER_HOST = 0, WISP_PAGER_DEVICE = 1 } wisp_pager;
wisp_status wisp_set_pager(wisp_ctx* ctx, int32_t pager);

/* Route T tokens of `layer`: x_dev [T, d] (x_dtype) -> idx_dev [T, k] int32 and w_dev [T, k] fp32
 * on `stream`, ranks ordered (score desc, expert id asc).  If idx_host is not NULL the call
 * waits for the indices and copies them there (T*k int32): this is the one device->host
 * synchronisation of a layer-step, needed because the pager runs on the host (the selection kernel
 * writes the ids, tagged with a per-call sequence number, straight to host-coherent memory).  For a token batch
 * that takes the grouped FFN, the call also enqueues, after the copy, the ordering of the (token,
 * rank) pairs by expert from idx_dev; the next wisp_moe_forward of this layer uses that order when
 * it is handed the same ids through wisp_page_in, and otherwise orders the pairs itself. */
wisp_status wisp_route_topk(wisp_ctx* ctx, int32_t layer, const void* x_dev, int32_t T, int32_t* idx_dev,
                            float* w_dev, int32_t* idx_host, void* stream);

/* Algorithm 1 lines for faults, victims, assignment, fills, map update and ticks, for the routing
 * ids_host [T, k] of `layer`.  The reference set is the union of the T selections.  If it fits
 * in C it is one step; otherwise it is split into chunks of C (resident ids ascending, then the
 * rest ascending), whose fills are issued by wisp_moe_forward between chunk computations.  Fills
 * are hipMemcpyAsync copies of whole blobs from the pinned masters on the library's side stream,
 * ordered after the layer's previous FFN (write-after-read on victim slots).  Asynchronous.
 * st (optional) receives this step's counts.  Must be followed by wisp_moe_forward for the
 * same layer and T before the next page-in of that layer. */
wisp_status wisp_page_in(wisp_ctx* ctx, int32_t layer, const int32_t* ids_host, int32_t T, wisp_page_stats* st);

/* The FFN over the routing given to the preceding wisp_page_in of `layer`: for every token t and
 * rank j, o_tj = W2 (silu(W1 x_t) * (W3 x_t)) with the weights of expert idx[t,j] read from its
 * slot, then y_t = sum_j w_dev[t,j] o_tj in rank order (+ the shared expert's output).  Experts
 * that were resident start at once; faulted ones wait for their fill.  x_dev [T, d], w_dev [T, k]
 * fp32, y_dev [T, d] fp32, on `stream`.  Returns WISP_E_NOT_RESIDENT if a routed expert is not
 * resident (exactness invariant, Sec. 3.2).  st (optional) receives the step's counts.  Precision:
 * fp32 accumulation; with bf16 or fp8 weights h is rounded to bf16, and token batches of 16 or more
 * tokens on the grouped matrix-core GEMMs (bf16 weights) also round each o_tj to bf16 before the
 * combine (single-token and small batches keep o_tj in fp32). */
wisp_status wisp_moe_forward(wisp_ctx* ctx, int32_t layer, const void* x_dev, int32_t T, const float* w_dev,
                             float* y_dev, void* stream, wisp_page_stats* st);

/* One decode step over all layers in order (route, page-in, forward per layer): x_dev [L, T, d],
 * idx_dev [L, T, k], w_dev [L, T, k], y_dev [L, T, d].  Layer l+1 is routed only after layer l's
 * FFN has been issued.  st (optional) receives [L] per-layer counts.  With the host pager, a token
 * batch that takes the grouped FFN (and no prefetch mode) keeps its ids on the device: the kernel
 * that orders its pairs by expert hands each expert's pair count to the host, which pages in the
 * set of experts with pairs (Algorithm 1 depends only on that set) and sizes the grouped launches
 * from the counts; decisions and outputs are those of the route / page-in / forward calls. */
wisp_status wisp_decode_step(wisp_ctx* ctx, const void* x_dev, int32_t T, int32_t* idx_dev, float* w_dev,
                             float* y_dev, void* stream, wisp_page_stats* st);

/* Static offload at a VRAM expert budget: the comparison arm of the paper's iso-VRAM evaluation
 * (Sec. 1 and Sec. 5.2: static layer-level offload keeps most weights on the host and moves them over
 * the link when the layer runs, routing-blind).  Layers 0 .. R-1 keep all N experts resident; the
 * others are served from the masters every step, by mode:
 *  WISP_OFFLOAD_BULK: the N experts of each other layer are copied in one bulk copy into one of two
 *    layer-sized staging buffers on the side stream, the next layer's copy overlapping the current
 *    layer's compute; R = floor((expert_bytes - 2 N M_e) / (N M_e)); needs two layers' worth of bytes.
 *  WISP_OFFLOAD_ZERO_COPY: no staging; the expert kernels read the routed experts of the other
 *    layers straight from the pinned masters (zero-copy over the host link, nothing cached);
 *    R = floor(expert_bytes / (N M_e)); needs pinned masters.
 * R = L when every layer fits.  wisp_offload_step takes the arguments of wisp_decode_step and runs the
 * same router, expert and combine kernels as the pager, so outputs equal those of the paged and fully
 * resident runs bit for bit.  wisp_offload_end waits for outstanding copies and frees the buffers.
 * The pager's own slots are left as they are (unused meanwhile).  Host pager only. */
typedef enum { WISP_OFFLOAD_BULK = 0, WISP_OFFLOAD_ZERO_COPY = 1 } wisp_offload_mode;
wisp_status wisp_offload_begin(wisp_ctx* ctx, uint64_t expert_bytes, int32_t mode, int32_t* resident_layers_out);
wisp_status wisp_offload_step(wisp_ctx* ctx, const void* x_dev, int32_t T, int32_t* idx_dev, float* w_dev,
                              float* y_dev, void* stream);
wisp_status wisp_offload_end(wisp_ctx* ctx);

/* The description the context was created with. */
wisp_status wisp_get_desc(wisp_ctx* ctx, wisp_model_desc* desc);

/* Cumulative counts of `layer` since creation or the last wisp_reset_stats. */
wisp_status wisp_get_stats(wisp_ctx* ctx, int32_t layer, wisp_page_stats* cumulative);
wisp_status wisp_reset_stats(wisp_ctx* ctx);

/* Current cap C (0 before the first wisp_set_budget). */
wisp_status wisp_get_cap(wisp_ctx* ctx, int32_t* cap);

/* Slot of `expert` in `layer` (-1 if not resident), and the expert held by `slot` (-1 if empty). */
wisp_status wisp_slot_of(wisp_ctx* ctx, int32_t layer, int32_t expert, int32_t* slot);
wisp_status wisp_expert_in_slot(wisp_ctx* ctx, int32_t layer, int32_t slot, int32_t* expert);

/* Copy the device bytes of `slot` of `layer` to host memory dst (M_e bytes); synchronous. */
wisp_status wisp_read_slot(wisp_ctx* ctx, int32_t layer, int32_t slot, void* dst);

/* Fused decode kernels (on by default).  (1) A layer-step of one token with bf16 weights whose
 * union fits the cap runs the down projection of all its experts and the gate-weighted combine in
 * one launch (the per-expert outputs stay on chip) instead of a down launch per expert group and a
 * combine launch.  (2) The device pager computes the router logits and, in its first workgroup once
 * every logit row is published, the selection and Algorithm 1 in one launch instead of two.  (3)
 * wisp_route_topk (and the host pager's decode step) computes the logits of up to four tokens and, in
 * its first workgroup once every row is published, their selection in one launch instead of two.  Every logit, row,
 * decision and sum is computed by the same operations in the same order either way, so routing,
 * paging and outputs are bit-identical.  on = 0 selects the separate kernels (for comparison).
 * WISP_E_STATE while a page-in is pending. */
wisp_status wisp_set_fusion(wisp_ctx* ctx, int32_t on);

/* Kernel timing.  Launches of the classes whose bit is set in class_mask (1 << wisp_kernel_class;
 * 0 = off) are bracketed by HIP events on their own stream (kernels through the launch's own
 * start/stop events, fill batches by events on the side stream); durations accumulate per class.
 * Classes: */
typedef enum {
  WISP_K_ROUTER_LOGITS = 0, WISP_K_ROUTER_SELECT = 1, WISP_K_FFN_GATEUP = 2, WISP_K_FFN_DOWN = 3,
  WISP_K_COMBINE = 4, WISP_K_H2D_FILL = 5, WISP_K_GROUPED_GATEUP = 6, WISP_K_GROUPED_DOWN = 7,
  WISP_K_PERMUTE = 8, WISP_K_DOWN_COMBINE = 9, WISP_K_NUM = 10
} wisp_kernel_class;
wisp_status wisp_set_profiling(wisp_ctx* ctx, int32_t class_mask);
/* Waits for outstanding timed work, then returns the accumulated total milliseconds, number of
 * launches, algorithmic HBM bytes (weights and activations each read or written once) and
 * algorithmic floating-point operations (2 per multiply-add; counted for the grouped GEMM classes)
 * of a class.  Any output pointer may be NULL. */
wisp_status wisp_kernel_times(wisp_ctx* ctx, int32_t kclass, double* total_ms, uint64_t* launches,
                              uint64_t* bytes, uint64_t* flops);
wisp_status wisp_reset_kernel_times(wisp_ctx* ctx);

/* Measure host->device bandwidth of the expert path: `reps` rounds, each copying `count` expert
 * blobs (M_e each) from the pinned masters to a scratch device buffer on the side stream; returns
 * the median GB/s (1e9 bytes/s).  Allocates and frees the scratch buffer itself. */
wisp_status wisp_probe_h2d(wisp_ctx* ctx, int32_t count, int32_t reps, double* gbps);

/* The same measurement with the engine of the fills chosen: WISP_LINK_COPY_ENGINE (one
 * hipMemcpyAsync per blob, as wisp_probe_h2d) or WISP_LINK_CUS (the compute units stream the blobs,
 * 32 per launch, as the fills of token batches and the device pager do).  WISP_LINK_CUS needs pinned
 * masters (WISP_E_INVAL otherwise); WISP_E_INVAL for an unknown engine. */
typedef enum { WISP_LINK_COPY_ENGINE = 0, WISP_LINK_CUS = 1 } wisp_link_engine;
wisp_status wisp_probe_h2d_engine(wisp_ctx* ctx, int32_t count, int32_t reps, int32_t engine, double* gbps);

/* A plain device copy kernel (16-byte loads and stores) of `bytes` from src to dst on `stream`:
 * the reference for HBM counters and for measured copy bandwidth.  bytes must be a multiple of
 * 16 and both pointers 16-byte aligned. */
wisp_status wisp_hbm_copy(const void* src, void* dst, uint64_t bytes, void* stream);

/* The read floor of a launch size: `launches` back-to-back launches of a plain streaming-read kernel
 * (16-byte non-temporal loads, 16 KB per workgroup, nothing stored), each reading `bytes` from its
 * own window of a device buffer of at least 2 GiB, so that no launch finds its bytes in the 256 MB
 * last-level cache; returns the mean time per launch in microseconds.  bytes in [16, 4 GiB] and a
 * multiple of 16, launches >= 1 (WISP_E_INVAL otherwise).  Allocates, uses and frees its own buffer
 * and stream (WISP_E_NOMEM when the buffer does not fit). */
wisp_status wisp_probe_hbm_read(uint64_t bytes, int32_t launches, double* us_per_launch);

/* The dense bf16 matrix-core rate the current device sustains: `launches` back-to-back launches of a
 * kernel whose waves (eight per SIMD) issue only v_mfma_f32_32x32x16_bf16 on register operands, four
 * independent chains per wave; returns TFLOP/s (1e12 flops/s, 2*32*32*16 flops per instruction).
 * launches >= 1 (WISP_E_INVAL otherwise).  Allocates and frees a 256-byte sink and its own stream. */
wisp_status wisp_probe_mfma(int32_t launches, double* tflops);

/* Decode n fp8 E4M3 codes to fp32 on the device with the same conversion the FFN kernels use
 * (for checking the hardware conversion against the format definition). */
wisp_status wisp_decode_fp8(const uint8_t* codes_dev, float* out_dev, int32_t n, void* stream);

/* Router scoring and top-k for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the selection of wisp_route_topk
 * without a context.  Routes T tokens x_dev [T, d] (x_dtype WISP_F32 or WISP_BF16) with router weights
 * w_r_dev [N, d] fp32 row-major into idx_dev [T, k] int32 and w_dev [T, k] fp32 on `stream`, ranks
 * ordered (score desc, expert id asc), route / n_groups / topk_groups as in wisp_model_desc.  It runs
 * the same kernels as wisp_route_topk with fusion on (one launch for T <= 4, logits then selection
 * above), so ids and gates are bit-identical to it; nothing is published to the host.
 * Allocates nothing: its scratch (the tagged logit words of the one-launch path, and the logits, kept
 * for token batches as up to eight partial sums over column slices) is a fixed device array of
 * 8192 + 32 * WISP_NOALLOC_MAX_LOGITS bytes that each device the library runs on holds until the process
 * ends; its address is looked up on the first call on a device (which also clears the tag words with a
 * kernel on `stream`).  Every call on a device shares that array: calls that overlap on one device
 * (other streams, other threads) race and must be serialised by the caller.  WISP_E_INVAL when
 * T * N > WISP_NOALLOC_MAX_LOGITS, for a null pointer or an unsupported shape (more than 8 tokens need
 * N and d multiples of 16, or d a multiple of 32); validation happens before any GPU call. */
#define WISP_NOALLOC_MAX_LOGITS 524288
wisp_status wisp_route_topk_noalloc(const float* w_r_dev, const void* x_dev, int32_t x_dtype, int32_t T, int32_t N,
                                    int32_t d, int32_t k, int32_t route, int32_t n_groups, int32_t topk_groups,
                                    int32_t* idx_dev, float* w_dev, void* stream);

/* Hazard check for tests (host pager): with on != 0, every slot chosen as a victim is overwritten
 * with 0xFF bytes (NaN in every weight format, and in the fp8 block scales) on the side stream right
 * after the stream's write-after-read wait on the layer's last FFN, before the fill copies the
 * master in (faults, chunked unions and speculative prefetch alike).  Outputs stay exact exactly when
 * every FFN read of a slot is ordered after its fill and every fill after the slot's last read
 * (Sec. 3.2, the exactness invariant).  Costs one memset per fault. */
wisp_status wisp_debug_poison_victims(wisp_ctx* ctx, int32_t on);

/* Fault injection for tests of the transactional resize: the next `n`-th device slot allocation
 * (counting from 1, across later wisp_set_budget calls) fails as if out of memory.  0 = off. */
wisp_status wisp_debug_fail_slot_alloc(wisp_ctx* ctx, int32_t n);

/* Message of the last error on this thread ("" if none). */
const char* wisp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WISP_H */
