/*
 * wisp_mvwsa.h — the expert <-> KV allocator of WiSP (arXiv 2606.21868) around the paged MoE layer:
 * miss curves, the MV-WSA startup configurator, the dual-resize control law and the drained-barrier
 * move between the expert scratch and a KV block pool.
 *
 * Units: C is the per-layer expert cap, a = L * M_e the bytes of one more resident expert per layer
 * over all layers, kappa the KV pool in blocks, b the bytes of one KV block over all layers, B the
 * pageable budget B = C a + kappa b (Sec. 3.1, Eq. 1).  Conventions as in wisp.h: every call returns a
 * wisp_status, validates before it changes anything, and never throws.
 */
#ifndef WISP_MVWSA_H
#define WISP_MVWSA_H

#include <stdint.h>

#include "wisp.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Expert miss curve m(C) of one layer from a routing trace (Sec. 3.2, "Reuse-distance miss curves"):
 * ids [steps][refs] holds the routed ids of each step (duplicates within a step count once).
 * Algorithm 1 gives the experts of one step the same LRU tick, so the reuse distance of a reference is
 * counted at step level: the distinct experts referenced in the steps strictly between its previous
 * reference and this one.  A reference misses at cap C iff it is the first reference to its expert or
 * that distance is >= C.  This is a lower bound on Algorithm 1's misses (exact when every step has one
 * reference).  misses receives n_experts + 1 counts, C = 0 .. n_experts.  misses_upper (optional, NULL
 * to skip) receives the upper bound: a reference also counts when its distance plus the number of other
 * experts of its previous step is >= C (those share its tick, so any of them may be evicted after it).
 * One pass, O(R log S) for R references and S steps (a Fenwick tree over steps).  Host memory only. */
wisp_status wisp_miss_curve(const int32_t* ids, int32_t steps, int32_t refs, int32_t n_experts, uint64_t* misses,
                            uint64_t* misses_upper);

/* MV-WSA startup configurator (Sec. 3.3 and 3.4, Eqs. 3-5). */
typedef struct {
  uint64_t budget_bytes;    /* B */
  uint64_t expert_set_bytes; /* a = L * M_e */
  uint64_t kv_block_bytes;  /* b */
  int64_t kv_min_blocks;    /* kappa_min = W * ceil(l_ctx / b_tok) (Eq. 4) */
  double c_exp;             /* cost of one expert miss, M_e * t_byte (seconds) */
  double c_kv;              /* cost of one KV miss, beta * b_tok (seconds) */
  int32_t n_experts;        /* N: m_exp has N + 1 entries */
  int64_t kv_curve_len;     /* entries of m_kv, kappa = 0 .. len - 1; larger pools take the last entry */
} wisp_mvwsa_problem;

typedef struct {
  int32_t cap;              /* C of Eq. 5 */
  int64_t kv_blocks;        /* kappa = floor((B - C a) / b) */
  uint64_t kv_bytes;        /* B_kv of Eq. 5 as whole blocks: kappa * b */
  double f;                 /* the split f^ = C* a / B that minimises the latency model of Eq. 3 */
  double latency;           /* T at the returned cap */
  int32_t floor_binding;    /* 1 when the admission floor lowered the cap below the minimiser */
} wisp_mvwsa_split;

/* The split f^ minimises T(C) = c_exp m_exp(C) + c_kv m_kv(floor((B - C a) / b)) (Eq. 3) over the caps
 * 0 .. min(N, floor(B / a)) (ties to the smaller cap: a discrete equimarginal point, Eq. 2); Eq. 5 then
 * gives C = min(floor(f^ B / a), floor((B - kappa_min b) / a)) and B_kv = B - C a.  WISP_E_INVAL when
 * B < kappa_min b (no split admits the floor) or an argument is out of range. */
wisp_status wisp_mvwsa_configure(const wisp_mvwsa_problem* problem, const uint64_t* m_exp, const double* m_kv,
                                 wisp_mvwsa_split* out);

/* Dual-resize control law (App. B, Eqs. 6-8): from the peak KV occupancy p (blocks in use) of the last
 * burst, kappa~ = max(kappa_min, ceil((1 + h) p)), C~ = clip(floor((B - kappa~ b) / a), C_min, C_max),
 * kappa~ <- floor((B - C~ a) / b).  *move_out = 1 unless |C~ - cap_now| < dead_zone (or C~ = cap_now). */
typedef struct {
  uint64_t budget_bytes, expert_set_bytes, kv_block_bytes;
  int64_t kv_min_blocks;
  double headroom;          /* h */
  int32_t cap_min, cap_max; /* 1 <= C_min <= C_max <= N */
  int32_t dead_zone;        /* Delta, in experts per layer */
} wisp_resize_law;

wisp_status wisp_resize_target(const wisp_resize_law* law, int64_t peak_kv_blocks, int32_t cap_now, int32_t* cap_out,
                               int64_t* kv_blocks_out, int32_t* move_out);

/* A KV block pool on the current device: kappa blocks of b bytes in device memory, held in chunks
 * of at most 64 blocks.  A shrink frees every chunk left without a block (it never fails; the pool
 * keeps fewer than 64 blocks beyond its size); a grow first uses that slack and, if an allocation
 * fails, frees what it added and keeps the previous size (WISP_E_NOMEM).  It holds the bytes of the
 * KV side of the budget; its contents are not used here (the KV cache is simulated). */
typedef struct wisp_kv_pool wisp_kv_pool;
wisp_status wisp_kv_pool_create(uint64_t block_bytes, int64_t blocks, wisp_kv_pool** out);
wisp_status wisp_kv_pool_blocks(const wisp_kv_pool* pool, int64_t* blocks);
wisp_status wisp_kv_pool_resize(wisp_kv_pool* pool, int64_t blocks);  /* WISP_E_NOMEM: previous size kept */
wisp_status wisp_kv_pool_destroy(wisp_kv_pool* pool);

/* The drained-barrier move of App. B: resize the expert scratch to cap_new (wisp_set_budget with
 * cap_new * L * M_e bytes) and the pool to kv_blocks_new, freeing the shrinking side first (an expert
 * grow shrinks KV first; an expert shrink frees slots first), so the transient footprint stays
 * max(old, new).  If the growing side fails, the shrunk side is grown back and WISP_E_NOMEM is
 * returned with the previous split in place.  Drains the context like wisp_set_budget. */
wisp_status wisp_dual_resize(wisp_ctx* ctx, wisp_kv_pool* pool, int32_t cap_new, int64_t kv_blocks_new);

/* The online controller of MV-WSA (Sec. 3.5 "Dynamic Dual-Resize", App. B): the caller reports the KV
 * blocks in use after each decode step; at each drained barrier the controller takes the peak since
 * the previous barrier as p, computes the target of the control law (wisp_resize_target, Eqs. 6-8,
 * with its dead-zone) against the split it last applied, and, if a move is due, applies it with
 * wisp_dual_resize.  A move that fails for lack of memory is skipped and the previous split stays
 * (*moved_out = -1); *moved_out = 1 after a move, 0 when none was due or nothing was observed since the
 * last barrier.  ctx and pool NULL: the decision only, nothing resized.  *peak_out receives p (-1 if
 * nothing was observed).  Host memory only; one controller per (context, pool). */
typedef struct wisp_controller wisp_controller;
wisp_status wisp_controller_create(const wisp_resize_law* law, int32_t cap_now, int64_t kv_blocks_now,
                                   wisp_controller** out);
wisp_status wisp_controller_observe(wisp_controller* ctl, int64_t kv_blocks_in_use);
wisp_status wisp_controller_barrier(wisp_controller* ctl, wisp_ctx* ctx, wisp_kv_pool* pool, int32_t* cap_out,
                                    int64_t* kv_blocks_out, int32_t* moved_out, int64_t* peak_out);
wisp_status wisp_controller_destroy(wisp_controller* ctl);

#ifdef __cplusplus
}
#endif

#endif /* WISP_MVWSA_H */
