// Host-side slot table of one MoE layer: the bookkeeping of Algorithm 1 (WiSP, Sec. 3.2).
// Pure C++; no HIP calls.  The pager turns a StepPlan into copies and kernel launches.
#pragma once

#include <cstdint>
#include <utility>
#include <vector>

namespace wisp {

// One Algorithm 1 step over a set of distinct experts (a chunk of the layer-step's union).
struct ChunkPlan {
  std::vector<int32_t> experts;  // residents ascending, then faults ascending
  std::vector<int32_t> slots;    // slot holding each expert while this chunk computes
  std::vector<uint8_t> fault;    // 1 if the expert is copied in by this chunk
  int32_t n_faults = 0;
};

struct StepPlan {
  int32_t hits = 0;
  int32_t misses = 0;
  std::vector<ChunkPlan> chunks;
};

class SlotTable {
 public:
  SlotTable(int32_t n_experts, int32_t cap);

  int32_t n_experts() const { return N_; }
  int32_t cap() const { return C_; }
  int32_t slot_of(int32_t e) const { return pi_[e]; }
  int32_t expert_in(int32_t s) const { return pinv_[s]; }
  uint64_t tick(int32_t s) const { return tau_[s]; }
  uint64_t clock() const { return clock_; }

  // One layer-step over ids[0..n).  Returns false (table unchanged) if an id is out of range.
  bool step(const int32_t* ids, int32_t n, StepPlan* plan);

  // Resize to new_cap.  old_slot_of_new[i] = the old slot whose contents become slot i, or -1 for
  // a new empty slot.  Returns false (table unchanged) on a bad cap.
  bool resize(int32_t new_cap, std::vector<int32_t>* old_slot_of_new);

  // Speculative page-in of ids[0..n) (distinct ids taken in order, at most C): each absent one takes
  // a victim, the slots whose occupant is not among the ids ordered (tick asc, slot asc), and gets
  // the current clock as its tick (recent, but no step is counted).  fills receives (expert, slot)
  // per copy to issue.  Returns false (table unchanged) if an id is out of range.
  bool prefetch(const int32_t* ids, int32_t n, std::vector<std::pair<int32_t, int32_t>>* fills);

  // Drop every resident expert (all slots empty, ticks 0); the clock keeps counting.
  void clear();

  // Raw state, for moving the table to and from the device pager.
  void export_state(int32_t* pi, int32_t* pinv, uint64_t* tau, uint64_t* clock) const;
  void import_state(const int32_t* pi, const int32_t* pinv, const uint64_t* tau, uint64_t clock);

 private:
  void alg1(const int32_t* G, int32_t g, ChunkPlan* cp);

  int32_t N_, C_;
  std::vector<int32_t> pi_;     // expert -> slot, -1 if absent
  std::vector<int32_t> pinv_;   // slot -> expert, -1 if empty
  std::vector<uint64_t> tau_;   // slot -> tick of last use
  uint64_t clock_ = 0;
  // scratch
  std::vector<uint8_t> mark_;
  std::vector<int32_t> cand_;
};

}  // namespace wisp
