/*
 * wisp_slot_table.h — the pager's host-side slot table, exported for CPU tests.
 *
 * This is the exact bookkeeping wisp_page_in and wisp_set_budget run for one layer (Algorithm 1
 * of WiSP, arXiv 2606.21868, Sec. 3.2): expert -> slot map pi, slot -> expert map pi^-1, LRU
 * ticks tau and clock c over C slots.  It performs no HIP call and needs no GPU.
 *
 * Rules: the reference set R of a layer-step is the distinct ids given.  If |R| <= C it is one
 * step; otherwise it is processed as chunks of C ids (resident ids ascending, then the others
 * ascending), each one step.  A step assigns faults (ascending id) to victims ordered by
 * (tau asc, slot asc) among slots whose occupant is not in the step's set (empty slots have
 * tau = 0), then sets c += 1 and tau[pi(e)] = c for every e in the set.  Resize keeps the
 * most recently used experts (tau desc, ties to the lower slot) renumbered in slot order.
 */
#ifndef WISP_SLOT_TABLE_H
#define WISP_SLOT_TABLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct wisp_slot_table wisp_slot_table;

/* New empty table with N experts and C slots (1 <= C <= N); NULL on bad arguments. */
wisp_slot_table* wisp_slot_table_create(int32_t n_experts, int32_t cap);
void wisp_slot_table_destroy(wisp_slot_table* t);

/* One layer-step over ids[0..n) (duplicates allowed; ids in [0, N)).  Outputs: hits, misses,
 * chunks; miss_ids / miss_slots (capacity n) in assignment order; miss_chunk (capacity n, may be
 * NULL) the chunk index of each fault.  Returns 0, or -1 on a bad id (table unchanged). */
int32_t wisp_slot_table_step(wisp_slot_table* t, const int32_t* ids, int32_t n, int32_t* hits, int32_t* misses,
                             int32_t* chunks, int32_t* miss_ids, int32_t* miss_slots, int32_t* miss_chunk);

/* Speculative page-in (no step is counted): the distinct ids of ids[0..n), in order and at most C of
 * them, are made resident.  Each absent one takes a victim among the slots whose occupant is not one
 * of those ids, ordered (tau asc, slot asc), and gets tau = c (the current clock).  fill_ids /
 * fill_slots (capacity min(n, C), may be NULL) receive the copies to issue in order.  Returns their
 * count, or -1 on a bad id (table unchanged). */
int32_t wisp_slot_table_prefetch(wisp_slot_table* t, const int32_t* ids, int32_t n, int32_t* fill_ids,
                                 int32_t* fill_slots);

/* Change the cap (1 <= cap <= N); returns 0 or -1 (table unchanged). */
int32_t wisp_slot_table_resize(wisp_slot_table* t, int32_t cap);

int32_t wisp_slot_table_slot_of(const wisp_slot_table* t, int32_t expert);
int32_t wisp_slot_table_expert_in(const wisp_slot_table* t, int32_t slot);
uint64_t wisp_slot_table_tick(const wisp_slot_table* t, int32_t slot);
int32_t wisp_slot_table_cap(const wisp_slot_table* t);

#ifdef __cplusplus
}
#endif

#endif /* WISP_SLOT_TABLE_H */
