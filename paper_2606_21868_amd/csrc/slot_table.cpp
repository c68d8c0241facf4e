// Slot table of one MoE layer (Algorithm 1 of WiSP, Sec. 3.2), and its C export for CPU tests.
#include "slot_table.hpp"

#include <algorithm>
#include <new>

#include "wisp_slot_table.h"

namespace wisp {

SlotTable::SlotTable(int32_t n_experts, int32_t cap)
    : N_(n_experts), C_(cap), pi_(n_experts, -1), pinv_(cap, -1), tau_(cap, 0), mark_(n_experts, 0) {
  cand_.reserve(cap);
}

// A cold table: every slot empty and the clock back at 0, as before the first step.  (A clock left
// running would give a prefetch before the first step a tick above the empty slots' 0, where a
// cold table gives it 0: the victim order of the next step would then differ.)
void SlotTable::clear() {
  std::fill(pi_.begin(), pi_.end(), -1);
  std::fill(pinv_.begin(), pinv_.end(), -1);
  std::fill(tau_.begin(), tau_.end(), 0);
  clock_ = 0;
}

void SlotTable::export_state(int32_t* pi, int32_t* pinv, uint64_t* tau, uint64_t* clock) const {
  std::copy(pi_.begin(), pi_.end(), pi);
  std::copy(pinv_.begin(), pinv_.end(), pinv);
  std::copy(tau_.begin(), tau_.end(), tau);
  *clock = clock_;
}

void SlotTable::import_state(const int32_t* pi, const int32_t* pinv, const uint64_t* tau, uint64_t clock) {
  std::copy(pi, pi + N_, pi_.begin());
  std::copy(pinv, pinv + C_, pinv_.begin());
  std::copy(tau, tau + C_, tau_.begin());
  clock_ = clock;
}

// One step on the distinct ids G (|G| <= C): faults in ascending id take the victims with the
// smallest (tick, slot) among slots whose occupant is not in G; then every id of G gets the new
// tick (all experts of a step share it).
void SlotTable::alg1(const int32_t* G, int32_t g, ChunkPlan* cp) {
  for (int32_t i = 0; i < g; ++i) mark_[G[i]] = 1;
  std::vector<int32_t> res, flt;
  res.reserve(g);
  flt.reserve(g);
  for (int32_t i = 0; i < g; ++i) (pi_[G[i]] >= 0 ? res : flt).push_back(G[i]);
  std::sort(res.begin(), res.end());
  std::sort(flt.begin(), flt.end());
  if (!flt.empty()) {
    cand_.clear();
    for (int32_t s = 0; s < C_; ++s)
      if (pinv_[s] < 0 || !mark_[pinv_[s]]) cand_.push_back(s);
    const size_t nv = flt.size();
    auto by_age = [&](int32_t a, int32_t b) { return tau_[a] < tau_[b] || (tau_[a] == tau_[b] && a < b); };
    std::partial_sort(cand_.begin(), cand_.begin() + nv, cand_.end(), by_age);
    for (size_t i = 0; i < nv; ++i) {
      const int32_t s = cand_[i];
      if (pinv_[s] >= 0) pi_[pinv_[s]] = -1;
      pi_[flt[i]] = s;
      pinv_[s] = flt[i];
    }
  }
  ++clock_;
  for (int32_t i = 0; i < g; ++i) {
    tau_[pi_[G[i]]] = clock_;
    mark_[G[i]] = 0;
  }
  cp->experts.clear();
  cp->slots.clear();
  cp->fault.clear();
  for (int32_t e : res) { cp->experts.push_back(e); cp->slots.push_back(pi_[e]); cp->fault.push_back(0); }
  for (int32_t e : flt) { cp->experts.push_back(e); cp->slots.push_back(pi_[e]); cp->fault.push_back(1); }
  cp->n_faults = static_cast<int32_t>(flt.size());
}

bool SlotTable::step(const int32_t* ids, int32_t n, StepPlan* plan) {
  for (int32_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= N_) return false;
  // distinct ids
  std::vector<int32_t> R;
  R.reserve(n);
  for (int32_t i = 0; i < n; ++i)
    if (!mark_[ids[i]]) { mark_[ids[i]] = 1; R.push_back(ids[i]); }
  for (int32_t e : R) mark_[e] = 0;
  plan->chunks.clear();
  plan->hits = plan->misses = 0;
  const int32_t nr = static_cast<int32_t>(R.size());
  if (nr == 0) return true;
  if (nr <= C_) {
    plan->chunks.emplace_back();
    alg1(R.data(), nr, &plan->chunks.back());
  } else {
    // residency is judged once, at the start of the layer-step
    std::vector<int32_t> res, non;
    for (int32_t e : R) (pi_[e] >= 0 ? res : non).push_back(e);
    std::sort(res.begin(), res.end());
    std::sort(non.begin(), non.end());
    std::vector<int32_t> ord(res);
    ord.insert(ord.end(), non.begin(), non.end());
    for (int32_t off = 0; off < nr; off += C_) {
      plan->chunks.emplace_back();
      alg1(ord.data() + off, std::min(C_, nr - off), &plan->chunks.back());
    }
  }
  for (const auto& c : plan->chunks) plan->misses += c.n_faults;
  plan->hits = nr - plan->misses;
  return true;
}

bool SlotTable::prefetch(const int32_t* ids, int32_t n, std::vector<std::pair<int32_t, int32_t>>* fills) {
  fills->clear();
  for (int32_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= N_) return false;
  std::vector<int32_t> P;
  for (int32_t i = 0; i < n && static_cast<int32_t>(P.size()) < C_; ++i)
    if (!mark_[ids[i]]) { mark_[ids[i]] = 1; P.push_back(ids[i]); }
  std::vector<int32_t> victims;
  for (int32_t s = 0; s < C_; ++s)
    if (pinv_[s] < 0 || !mark_[pinv_[s]]) victims.push_back(s);
  std::sort(victims.begin(), victims.end(),
            [&](int32_t a, int32_t b) { return tau_[a] < tau_[b] || (tau_[a] == tau_[b] && a < b); });
  size_t v = 0;
  for (int32_t e : P) {
    mark_[e] = 0;
    if (pi_[e] >= 0 || v >= victims.size()) continue;
    const int32_t s = victims[v++];
    if (pinv_[s] >= 0) pi_[pinv_[s]] = -1;
    pi_[e] = s;
    pinv_[s] = e;
    tau_[s] = clock_;
    fills->push_back({e, s});
  }
  return true;
}

bool SlotTable::resize(int32_t new_cap, std::vector<int32_t>* old_slot_of_new) {
  if (new_cap < 1 || new_cap > N_) return false;
  std::vector<int32_t> map(new_cap, -1);
  if (new_cap >= C_) {
    for (int32_t s = 0; s < C_; ++s) map[s] = s;
  } else {
    std::vector<int32_t> occ;
    for (int32_t s = 0; s < C_; ++s)
      if (pinv_[s] >= 0) occ.push_back(s);
    auto recent = [&](int32_t a, int32_t b) { return tau_[a] > tau_[b] || (tau_[a] == tau_[b] && a < b); };
    const size_t keep = std::min(occ.size(), static_cast<size_t>(new_cap));
    std::partial_sort(occ.begin(), occ.begin() + keep, occ.end(), recent);
    std::vector<int32_t> kept(occ.begin(), occ.begin() + keep);
    std::sort(kept.begin(), kept.end());  // renumber in old slot order
    for (size_t i = 0; i < kept.size(); ++i) map[i] = kept[i];
  }
  std::vector<int32_t> pinv(new_cap, -1);
  std::vector<uint64_t> tau(new_cap, 0);
  for (int32_t i = 0; i < new_cap; ++i) {
    if (map[i] >= 0 && map[i] < C_) { pinv[i] = pinv_[map[i]]; tau[i] = tau_[map[i]]; }
  }
  std::fill(pi_.begin(), pi_.end(), -1);
  for (int32_t i = 0; i < new_cap; ++i)
    if (pinv[i] >= 0) pi_[pinv[i]] = i;
  pinv_.swap(pinv);
  tau_.swap(tau);
  C_ = new_cap;
  if (old_slot_of_new) *old_slot_of_new = map;
  return true;
}

}  // namespace wisp

// ------------------------------------------------------------------------------------------
// C export for CPU tests
// ------------------------------------------------------------------------------------------
struct wisp_slot_table {
  wisp::SlotTable t;
  wisp::StepPlan plan;
  wisp_slot_table(int32_t n, int32_t c) : t(n, c) {}
};

extern "C" {

wisp_slot_table* wisp_slot_table_create(int32_t n_experts, int32_t cap) {
  if (n_experts < 1 || cap < 1 || cap > n_experts) return nullptr;
  return new (std::nothrow) wisp_slot_table(n_experts, cap);
}

void wisp_slot_table_destroy(wisp_slot_table* t) { delete t; }

int32_t wisp_slot_table_step(wisp_slot_table* t, const int32_t* ids, int32_t n, int32_t* hits, int32_t* misses,
                             int32_t* chunks, int32_t* miss_ids, int32_t* miss_slots, int32_t* miss_chunk) {
  if (!t || (n > 0 && !ids) || n < 0) return -1;
  if (!t->t.step(ids, n, &t->plan)) return -1;
  int32_t m = 0;
  for (size_t c = 0; c < t->plan.chunks.size(); ++c) {
    const auto& cp = t->plan.chunks[c];
    for (size_t i = 0; i < cp.experts.size(); ++i) {
      if (!cp.fault[i]) continue;
      if (miss_ids) miss_ids[m] = cp.experts[i];
      if (miss_slots) miss_slots[m] = cp.slots[i];
      if (miss_chunk) miss_chunk[m] = static_cast<int32_t>(c);
      ++m;
    }
  }
  if (hits) *hits = t->plan.hits;
  if (misses) *misses = t->plan.misses;
  if (chunks) *chunks = static_cast<int32_t>(t->plan.chunks.size());
  return 0;
}

int32_t wisp_slot_table_prefetch(wisp_slot_table* t, const int32_t* ids, int32_t n, int32_t* fill_ids,
                                 int32_t* fill_slots) {
  if (!t || (n > 0 && !ids) || n < 0) return -1;
  std::vector<std::pair<int32_t, int32_t>> fills;
  if (!t->t.prefetch(ids, n, &fills)) return -1;
  for (size_t i = 0; i < fills.size(); ++i) {
    if (fill_ids) fill_ids[i] = fills[i].first;
    if (fill_slots) fill_slots[i] = fills[i].second;
  }
  return static_cast<int32_t>(fills.size());
}

int32_t wisp_slot_table_resize(wisp_slot_table* t, int32_t cap) {
  if (!t) return -1;
  return t->t.resize(cap, nullptr) ? 0 : -1;
}

int32_t wisp_slot_table_slot_of(const wisp_slot_table* t, int32_t e) {
  return (t && e >= 0 && e < t->t.n_experts()) ? t->t.slot_of(e) : -1;
}
int32_t wisp_slot_table_expert_in(const wisp_slot_table* t, int32_t s) {
  return (t && s >= 0 && s < t->t.cap()) ? t->t.expert_in(s) : -1;
}
uint64_t wisp_slot_table_tick(const wisp_slot_table* t, int32_t s) {
  return (t && s >= 0 && s < t->t.cap()) ? t->t.tick(s) : 0;
}
int32_t wisp_slot_table_cap(const wisp_slot_table* t) { return t ? t->t.cap() : 0; }

}  // extern "C"
