/*
 * wisp_predictor.h — the co-activation predictor of WiSP (arXiv 2606.21868, App. E) and speculative
 * expert prefetch through it (the experiment of Sec. 4, whose finding is that prefetch does not buy
 * single-stream decode speed when the host link is the bottleneck).
 *
 * Predictor.  For a source layer l and a later target layer l' (l' - l <= horizon) the predictor
 * counts how often expert e at l and expert e' at l' fire in the same forward pass, A_{l,l'}(e, e'),
 * and normalises by the source marginal: P_{l,l'}(e' | e) = A(e, e') / sum_j A(e, j).  A candidate e'
 * of a target layer scores
 *   s_{l'}(e') = sum_{l < l', l' - l <= horizon} gamma^{l' - l} sum_{e in R_l} P_{l,l'}(e' | e)
 * over the sets R_l already routed in the current pass; the highest scores are the prediction.  The
 * tables start empty and learn online: a pass's sets are counted when the pass ends.  The paper sums
 * over every earlier layer (horizon >= L - 1 does the same); a smaller horizon bounds the tables
 * (L * horizon * N^2 counts) and the cost of a prediction.  Host memory and host code only, no GPU.
 * A predictor is not thread-safe.  Scores are summed in double precision.
 *
 * Prefetch.  A speculative page-in of a layer uses that layer's slot table and LRU rule and the
 * same host link as demand faults (host pager only).  It is ordered after the layer's last FFN
 * (write-after-read on the victim slots), and the layer's next FFN that reads a prefetched expert
 * waits for the copies.  Outputs are unchanged by prefetch (the FFN reads the same bytes); only
 * residency and link traffic change.
 *
 * Errors: every call returns a wisp_status, checks its arguments before it changes anything, and
 * sets the message returned by wisp_last_error.
 */
#ifndef WISP_PREDICTOR_H
#define WISP_PREDICTOR_H

#include <stdint.h>

#include "wisp.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct wisp_predictor wisp_predictor;

/* New empty predictor for n_layers x n_experts (n_experts <= 4096), source layers within `horizon`
 * (>= 1; clamped to L - 1) of the target, distance decay 0 < gamma <= 1.  WISP_E_INVAL if the tables
 * (L * horizon * N^2 32-bit counts) would exceed 1.5e9 cells; WISP_E_NOMEM if host memory runs out. */
wisp_status wisp_predictor_create(int32_t n_layers, int32_t n_experts, int32_t horizon, double gamma,
                                  wisp_predictor** out);
wisp_status wisp_predictor_destroy(wisp_predictor* p);
/* The layer and expert counts the predictor was created with. */
wisp_status wisp_predictor_shape(const wisp_predictor* p, int32_t* n_layers, int32_t* n_experts);
/* R_layer of the current pass: ids[0..n) (duplicates count once; ids in [0, N)).  A second call for
 * the same layer in one pass replaces the first. */
wisp_status wisp_predictor_observe(wisp_predictor* p, int32_t layer, const int32_t* ids, int32_t n);
/* Count the current pass's co-activations into the tables and start a new, empty pass. */
wisp_status wisp_predictor_end_pass(wisp_predictor* p);
/* The `depth` highest-scoring experts of `layer` from the layers already observed in the current
 * pass, ordered (score desc, id asc); only positive scores are returned.  ids_out (and scores_out,
 * which may be NULL) have room for `depth` entries; *n_out receives the count (<= depth). */
wisp_status wisp_predictor_predict(wisp_predictor* p, int32_t layer, int32_t depth, int32_t* ids_out, int32_t* n_out,
                                   double* scores_out);

/* Speculative prefetch of ids[0..n) into `layer`'s slots (host pager).  The distinct ids, in the
 * order given and at most C of them, are made resident: each absent one takes a victim among the
 * slots whose occupant is not one of them, ordered (tick asc, slot asc), and gets the layer's
 * current tick (no step is counted).  Its blob is copied from the pinned master on the side stream
 * after the layer's last FFN.  The copies use the link the demand faults need, and a victim may be an
 * expert the next step routes to (Sec. 4).  WISP_E_STATE between a page-in of the layer and its
 * forward, with the device pager, during static offload, or with no budget set. */
wisp_status wisp_prefetch(wisp_ctx* ctx, int32_t layer, const int32_t* ids, int32_t n);

/* Prefetch inside wisp_decode_step (host pager): before layer l is routed, its predicted experts
 * are prefetched.
 *   WISP_PREFETCH_OFF: none (the default).
 *   WISP_PREFETCH_PREDICTOR: the top `depth` (1..N) of `predictor` (same L and N as the model, owned
 *     by the caller and kept alive while this mode is set) from the layers 0..l-1 routed in the same
 *     step; wisp_decode_step observes every layer's routed ids and ends the predictor's pass at the
 *     end of the step, so the predictor learns online.  Layer 0 has no earlier layer: no prefetch.
 *   WISP_PREFETCH_HINTS: the ids given by wisp_set_prefetch_hints, used by the next decode step only.
 * WISP_E_STATE with the device pager (and wisp_set_pager refuses the device pager while prefetch is
 * on). */
typedef enum { WISP_PREFETCH_OFF = 0, WISP_PREFETCH_PREDICTOR = 1, WISP_PREFETCH_HINTS = 2 } wisp_prefetch_mode;
wisp_status wisp_set_prefetch(wisp_ctx* ctx, int32_t mode, wisp_predictor* predictor, int32_t depth);
/* ids [L][n] row-major (n <= N; -1 = no id): the experts to prefetch for each layer during the next
 * wisp_decode_step.  The library copies them.  WISP_E_STATE unless the mode is WISP_PREFETCH_HINTS. */
wisp_status wisp_set_prefetch_hints(wisp_ctx* ctx, const int32_t* ids, int32_t n);
/* The ids wisp_decode_step asked to prefetch for `layer` in its last call (predictor output or hints,
 * before deduplication; empty when prefetch is off or had nothing to offer).  ids_out has room for
 * `cap` ids; WISP_E_INVAL if that is too small (N always suffices).  For logging and tests. */
wisp_status wisp_prefetch_requests(wisp_ctx* ctx, int32_t layer, int32_t* ids_out, int32_t cap, int32_t* n_out);
/* Prefetch counters since creation or the last wisp_reset_stats: experts copied speculatively, and of
 * those, how many the next page-in of their layer routed to while they were still resident. */
wisp_status wisp_prefetch_stats(wisp_ctx* ctx, uint64_t* issued, uint64_t* useful);

#ifdef __cplusplus
}
#endif

#endif /* WISP_PREDICTOR_H */
