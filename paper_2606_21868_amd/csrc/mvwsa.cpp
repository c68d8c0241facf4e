// Expert <-> KV allocator of WiSP (Sec. 3.3-3.5, App. B): miss curves from routing traces, the
// MV-WSA startup configurator, the dual-resize control law, a KV block pool and the drained-barrier
// move between the two pools.  Host code; the pool and the expert slots are device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <new>
#include <vector>

#include "errors.hpp"
#include "wisp_mvwsa.h"

using wisp::set_error;

namespace {

// Fenwick tree over reference positions (prefix sums of +/-1 marks).
class Fenwick {
 public:
  explicit Fenwick(size_t n) : t_(n + 1, 0) {}
  void add(size_t i, int v) {
    for (++i; i < t_.size(); i += i & (~i + 1)) t_[i] += v;
  }
  int64_t prefix(size_t i) const {  // sum over [0, i)
    int64_t s = 0;
    for (; i > 0; i -= i & (~i + 1)) s += t_[i];
    return s;
  }

 private:
  std::vector<int64_t> t_;
};

}  // namespace

struct wisp_kv_pool {
  uint64_t block_bytes = 0;
  int device = 0;
  std::vector<void*> chunks;
  std::vector<int64_t> chunk_cap;   // blocks each chunk holds
  int64_t capacity = 0;             // sum of chunk_cap
  int64_t blocks = 0;               // the pool's size (<= capacity < size + kChunkBlocks)
};

// The online dual-resize controller (Sec. 3.5, App. B): the law, the split it last applied, and the
// peak KV occupancy observed since the last drained barrier.
struct wisp_controller {
  wisp_resize_law law{};
  int32_t cap = 0;
  int64_t kv = 0;
  int64_t peak = -1;          // -1: nothing observed since the last barrier
  int64_t observed = 0;       // decode steps observed since the last barrier
};

namespace {

constexpr int64_t kChunkBlocks = 64;

// Grow to `blocks`: use the slack of the last chunk, then add chunks; on failure free what was added.
wisp_status pool_grow(wisp_kv_pool* p, int64_t blocks) {
  const size_t n0 = p->chunks.size();
  const int64_t c0 = p->capacity;
  while (p->capacity < blocks) {
    const int64_t add = std::min(kChunkBlocks, blocks - p->capacity);
    void* m = nullptr;
    if (hipMalloc(&m, static_cast<size_t>(add) * p->block_bytes) != hipSuccess) {
      (void)hipGetLastError();
      while (p->chunks.size() > n0) {
        (void)hipFree(p->chunks.back());
        p->chunks.pop_back();
        p->chunk_cap.pop_back();
      }
      p->capacity = c0;
      return WISP_E_NOMEM;
    }
    p->chunks.push_back(m);
    p->chunk_cap.push_back(add);
    p->capacity += add;
  }
  p->blocks = blocks;
  return WISP_OK;
}

// Shrink to `blocks`: free every trailing chunk that no longer holds a block (never fails).
void pool_shrink(wisp_kv_pool* p, int64_t blocks) {
  p->blocks = blocks;
  while (!p->chunks.empty() && p->capacity - p->chunk_cap.back() >= blocks) {
    (void)hipFree(p->chunks.back());
    p->capacity -= p->chunk_cap.back();
    p->chunks.pop_back();
    p->chunk_cap.pop_back();
  }
}

}  // namespace

extern "C" {

wisp_status wisp_miss_curve(const int32_t* ids, int32_t steps, int32_t refs, int32_t n_experts, uint64_t* misses,
                            uint64_t* misses_upper) {
  if (!ids || !misses || steps < 0 || refs < 0 || n_experts < 1)
    return set_error(WISP_E_INVAL, "miss curve: NULL pointer or non-positive shape");
  for (int64_t i = 0; i < static_cast<int64_t>(steps) * refs; ++i)
    if (ids[i] < 0 || ids[i] >= n_experts) return set_error(WISP_E_INVAL, "miss curve: expert id out of range");
  // Step-level reuse distance: for a reference to e at step t whose previous reference was at step
  // p, the number of experts whose latest reference lies in steps p+1 .. t-1.  A Fenwick tree over
  // steps holds one mark per expert, at the step of its latest reference; a step's distances are
  // read before its own marks move.
  std::vector<uint64_t> hist(static_cast<size_t>(n_experts) + 1, 0);
  std::vector<uint64_t> hist_up(static_cast<size_t>(n_experts) + 1, 0);   // distance + peers
  uint64_t cold = 0;
  std::vector<int32_t> last(n_experts, -1);
  std::vector<int32_t> step_size(static_cast<size_t>(std::max(steps, 1)), 0);   // distinct ids per step
  std::vector<int32_t> step_ids;
  Fenwick fw(static_cast<size_t>(std::max(steps, 1)));
  for (int32_t t = 0; t < steps; ++t) {
    step_ids.clear();
    for (int32_t r = 0; r < refs; ++r) {
      const int32_t e = ids[static_cast<size_t>(t) * refs + r];
      if (last[e] != t && std::find(step_ids.begin(), step_ids.end(), e) == step_ids.end()) step_ids.push_back(e);
    }
    for (int32_t e : step_ids) {
      const int32_t p = last[e];
      if (p < 0) {
        ++cold;
      } else {
        const int64_t dist = fw.prefix(static_cast<size_t>(t)) - fw.prefix(static_cast<size_t>(p) + 1);
        ++hist[static_cast<size_t>(std::min<int64_t>(dist, n_experts))];
        // the other experts of step p share e's tick and may be evicted after it: the upper bound
        const int64_t up = dist + step_size[static_cast<size_t>(p)] - 1;
        ++hist_up[static_cast<size_t>(std::min<int64_t>(up, n_experts))];
      }
    }
    step_size[static_cast<size_t>(t)] = static_cast<int32_t>(step_ids.size());
    for (int32_t e : step_ids) {
      if (last[e] >= 0) fw.add(static_cast<size_t>(last[e]), -1);
      fw.add(static_cast<size_t>(t), +1);
      last[e] = t;
    }
  }
  // m(C) = cold + #{distance >= C}; the upper curve counts distance + peers >= C
  uint64_t tail = 0, tail_up = 0;
  for (int32_t C = n_experts; C >= 0; --C) {
    tail += hist[C];
    tail_up += hist_up[C];
    misses[C] = cold + tail;
    if (misses_upper) misses_upper[C] = cold + tail_up;
  }
  return WISP_OK;
}

wisp_status wisp_mvwsa_configure(const wisp_mvwsa_problem* pr, const uint64_t* m_exp, const double* m_kv,
                                 wisp_mvwsa_split* out) {
  if (!pr || !m_exp || !m_kv || !out) return set_error(WISP_E_INVAL, "configure: NULL argument");
  if (pr->budget_bytes == 0 || pr->expert_set_bytes == 0 || pr->kv_block_bytes == 0 || pr->n_experts < 1 ||
      pr->kv_curve_len < 1 || pr->kv_min_blocks < 0 || !(pr->c_exp >= 0.0) || !(pr->c_kv >= 0.0))
    return set_error(WISP_E_INVAL, "configure: argument out of range");
  const uint64_t B = pr->budget_bytes, a = pr->expert_set_bytes, b = pr->kv_block_bytes;
  if (B < static_cast<uint64_t>(pr->kv_min_blocks) * b)
    return set_error(WISP_E_INVAL, "configure: the budget is below the KV admission floor");
  auto latency = [&](int64_t C) {
    const int64_t kappa = static_cast<int64_t>((B - static_cast<uint64_t>(C) * a) / b);
    return pr->c_exp * static_cast<double>(m_exp[C]) + pr->c_kv * m_kv[std::min(kappa, pr->kv_curve_len - 1)];
  };
  const int64_t cmax = std::min<int64_t>(pr->n_experts, static_cast<int64_t>(B / a));
  int64_t best = 0;
  double best_t = latency(0);
  for (int64_t C = 1; C <= cmax; ++C) {
    const double t = latency(C);
    if (t < best_t) {
      best_t = t;
      best = C;
    }
  }
  const int64_t floor_cap = static_cast<int64_t>((B - static_cast<uint64_t>(pr->kv_min_blocks) * b) / a);
  const int64_t C = std::min(best, floor_cap);
  out->cap = static_cast<int32_t>(C);
  out->kv_blocks = static_cast<int64_t>((B - static_cast<uint64_t>(C) * a) / b);
  out->kv_bytes = static_cast<uint64_t>(out->kv_blocks) * b;
  out->f = static_cast<double>(best) * static_cast<double>(a) / static_cast<double>(B);
  out->latency = latency(C);
  out->floor_binding = C < best ? 1 : 0;
  return WISP_OK;
}

wisp_status wisp_resize_target(const wisp_resize_law* law, int64_t peak_kv_blocks, int32_t cap_now, int32_t* cap_out,
                               int64_t* kv_blocks_out, int32_t* move_out) {
  if (!law || !cap_out || !kv_blocks_out || !move_out) return set_error(WISP_E_INVAL, "resize target: NULL argument");
  if (law->expert_set_bytes == 0 || law->kv_block_bytes == 0 || law->kv_min_blocks < 0 || !(law->headroom >= 0.0) ||
      law->cap_min < 0 || law->cap_max < law->cap_min || law->dead_zone < 0 || peak_kv_blocks < 0)
    return set_error(WISP_E_INVAL, "resize target: argument out of range");
  const uint64_t B = law->budget_bytes, a = law->expert_set_bytes, b = law->kv_block_bytes;
  const int64_t want = static_cast<int64_t>(std::ceil((1.0 + law->headroom) * static_cast<double>(peak_kv_blocks)));
  int64_t kappa = std::max(law->kv_min_blocks, want);                                       // Eq. 6
  int64_t C = B >= static_cast<uint64_t>(kappa) * b ? static_cast<int64_t>((B - static_cast<uint64_t>(kappa) * b) / a)
                                                   : 0;
  C = std::max<int64_t>(law->cap_min, std::min<int64_t>(law->cap_max, C));                 // Eq. 7
  if (static_cast<uint64_t>(C) * a > B) return set_error(WISP_E_INVAL, "resize target: C_min does not fit B");
  kappa = static_cast<int64_t>((B - static_cast<uint64_t>(C) * a) / b);                      // Eq. 8
  *cap_out = static_cast<int32_t>(C);
  *kv_blocks_out = kappa;
  const int64_t dc = C - cap_now;
  *move_out = (dc != 0 && (dc >= law->dead_zone || -dc >= law->dead_zone)) ? 1 : 0;
  return WISP_OK;
}

wisp_status wisp_kv_pool_create(uint64_t block_bytes, int64_t blocks, wisp_kv_pool** out) {
  if (!out || block_bytes == 0 || blocks < 0) return set_error(WISP_E_INVAL, "kv pool: bad size");
  *out = nullptr;
  auto* p = new (std::nothrow) wisp_kv_pool();
  if (!p) return WISP_E_NOMEM;
  p->block_bytes = block_bytes;
  if (hipGetDevice(&p->device) != hipSuccess) {
    delete p;
    return WISP_E_HIP;
  }
  if (pool_grow(p, blocks) != WISP_OK) {
    delete p;
    return set_error(WISP_E_NOMEM, "kv pool: device allocation failed");
  }
  *out = p;
  return WISP_OK;
}

wisp_status wisp_kv_pool_blocks(const wisp_kv_pool* pool, int64_t* blocks) {
  if (!pool || !blocks) return WISP_E_INVAL;
  *blocks = pool->blocks;
  return WISP_OK;
}

wisp_status wisp_kv_pool_resize(wisp_kv_pool* pool, int64_t blocks) {
  if (!pool || blocks < 0) return set_error(WISP_E_INVAL, "kv pool: bad size");
  if (hipSetDevice(pool->device) != hipSuccess) return set_error(WISP_E_HIP, "kv pool: hipSetDevice failed");
  if (blocks > pool->blocks && pool_grow(pool, blocks) != WISP_OK)
    return set_error(WISP_E_NOMEM, "kv pool: device allocation failed; previous size kept");
  if (blocks >= pool->blocks) return WISP_OK;
  pool_shrink(pool, blocks);
  return WISP_OK;
}

wisp_status wisp_kv_pool_destroy(wisp_kv_pool* pool) {
  if (!pool) return WISP_E_INVAL;
  (void)hipSetDevice(pool->device);
  for (void* m : pool->chunks) (void)hipFree(m);
  delete pool;
  return WISP_OK;
}

wisp_status wisp_dual_resize(wisp_ctx* ctx, wisp_kv_pool* pool, int32_t cap_new, int64_t kv_blocks_new) {
  if (!ctx || !pool || kv_blocks_new < 0) return set_error(WISP_E_INVAL, "dual resize: bad argument");
  int32_t cap_old = 0;
  wisp_status s = wisp_get_cap(ctx, &cap_old);
  if (s != WISP_OK) return s;
  wisp_model_desc desc{};
  if ((s = wisp_get_desc(ctx, &desc)) != WISP_OK) return s;
  uint64_t me = 0;
  if ((s = wisp_expert_bytes(&desc, &me)) != WISP_OK) return s;
  if (cap_new < 1 || cap_new > desc.n_experts) return set_error(WISP_E_INVAL, "dual resize: cap out of [1, N]");
  const uint64_t a = static_cast<uint64_t>(desc.n_layers) * me;
  const int64_t kv_old = pool->blocks;
  if (cap_new >= cap_old) {
    // expert grow: free KV first, then grow the scratch; on failure grow KV back
    if ((s = wisp_kv_pool_resize(pool, std::min(kv_old, kv_blocks_new))) != WISP_OK) return s;
    s = wisp_set_budget(ctx, static_cast<uint64_t>(cap_new) * a, nullptr);
    if (s != WISP_OK) {
      (void)wisp_kv_pool_resize(pool, kv_old);
      return s;
    }
    if (kv_blocks_new > pool->blocks && (s = wisp_kv_pool_resize(pool, kv_blocks_new)) != WISP_OK) {
      (void)wisp_set_budget(ctx, static_cast<uint64_t>(cap_old) * a, nullptr);
      (void)wisp_kv_pool_resize(pool, kv_old);
      return s;
    }
    return WISP_OK;
  }
  // expert shrink: free slots first, then grow KV; on failure grow the scratch back
  if ((s = wisp_set_budget(ctx, static_cast<uint64_t>(cap_new) * a, nullptr)) != WISP_OK) return s;
  if ((s = wisp_kv_pool_resize(pool, kv_blocks_new)) != WISP_OK) {
    (void)wisp_set_budget(ctx, static_cast<uint64_t>(cap_old) * a, nullptr);
    return s;
  }
  return WISP_OK;
}

wisp_status wisp_controller_create(const wisp_resize_law* law, int32_t cap_now, int64_t kv_blocks_now,
                                   wisp_controller** out) {
  if (!law || !out) return set_error(WISP_E_INVAL, "controller: NULL argument");
  *out = nullptr;
  int32_t c = 0, m = 0;
  int64_t k = 0;
  // the law must be valid (checked by evaluating it once) and the current split inside the budget
  wisp_status s = wisp_resize_target(law, 0, cap_now, &c, &k, &m);
  if (s != WISP_OK) return s;
  if (cap_now < 0 || kv_blocks_now < 0 ||
      static_cast<uint64_t>(cap_now) * law->expert_set_bytes + static_cast<uint64_t>(kv_blocks_now) *
      law->kv_block_bytes > law->budget_bytes)
    return set_error(WISP_E_INVAL, "controller: the current split exceeds the budget");
  auto* ctl = new (std::nothrow) wisp_controller();
  if (!ctl) return set_error(WISP_E_NOMEM, "controller: host allocation failed");
  ctl->law = *law;
  ctl->cap = cap_now;
  ctl->kv = kv_blocks_now;
  *out = ctl;
  return WISP_OK;
}

wisp_status wisp_controller_observe(wisp_controller* ctl, int64_t kv_blocks_in_use) {
  if (!ctl || kv_blocks_in_use < 0) return set_error(WISP_E_INVAL, "controller: bad observation");
  ctl->peak = std::max(ctl->peak, kv_blocks_in_use);
  ++ctl->observed;
  return WISP_OK;
}

wisp_status wisp_controller_barrier(wisp_controller* ctl, wisp_ctx* ctx, wisp_kv_pool* pool, int32_t* cap_out,
                                    int64_t* kv_blocks_out, int32_t* moved_out, int64_t* peak_out) {
  if (!ctl) return set_error(WISP_E_INVAL, "controller: NULL controller");
  if ((ctx == nullptr) != (pool == nullptr)) return set_error(WISP_E_INVAL, "controller: ctx and pool go together");
  int32_t moved = 0;
  const int64_t peak = ctl->peak;
  if (peak >= 0) {
    int32_t cap = 0, move = 0;
    int64_t kv = 0;
    wisp_status s = wisp_resize_target(&ctl->law, peak, ctl->cap, &cap, &kv, &move);
    if (s != WISP_OK) return s;
    if (move) {
      s = ctx ? wisp_dual_resize(ctx, pool, cap, kv) : WISP_OK;
      if (s == WISP_OK) {
        ctl->cap = cap;
        ctl->kv = kv;
        moved = 1;
      } else if (s == WISP_E_NOMEM) {
        moved = -1;            // the move is skipped: the previous split stays in place (App. B)
      } else {
        return s;
      }
    }
  }
  ctl->peak = -1;
  ctl->observed = 0;
  if (cap_out) *cap_out = ctl->cap;
  if (kv_blocks_out) *kv_blocks_out = ctl->kv;
  if (moved_out) *moved_out = moved;
  if (peak_out) *peak_out = peak;
  return WISP_OK;
}

wisp_status wisp_controller_destroy(wisp_controller* ctl) {
  delete ctl;
  return WISP_OK;
}

}  // extern "C"
