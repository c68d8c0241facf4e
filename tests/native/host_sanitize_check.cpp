// Host-only sources of the library (slot table, predictor, allocator and controller, copy pool) under
// AddressSanitizer and UndefinedBehaviorSanitizer.  The few HIP runtime calls of the KV pool are
// replaced by host-memory stand-ins, and the context calls wisp_dual_resize makes by a minimal fake
// context, so that every path (including failed allocations and the rollbacks after them) runs on
// the CPU.  Random sequences check the invariants of each part.  Prints "ok" and exits 0, or stops
// at the first broken invariant (the sanitizers stop at the first error themselves).
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <string>
#include <vector>

#include "copy_pool.hpp"
#include "errors.hpp"
#include "wisp.h"
#include "wisp_mvwsa.h"
#include "wisp_predictor.h"
#include "wisp_slot_table.h"

#define CHECK(cond)                                                                  \
  do {                                                                               \
    if (!(cond)) {                                                                   \
      std::printf("check failed at line %d: %s\n", __LINE__, #cond);                 \
      std::exit(1);                                                                  \
    }                                                                                \
  } while (0)

// ---- stand-ins: HIP allocations on host memory, with an injectable failure ----------------------
static int g_fail_malloc_at = 0;   // the n-th hipMalloc from now fails (0 = never)
static int g_live_allocs = 0;

extern "C" hipError_t hipMalloc(void** p, size_t n) {
  if (g_fail_malloc_at > 0 && --g_fail_malloc_at == 0) return hipErrorOutOfMemory;
  *p = std::malloc(n ? n : 1);
  if (!*p) return hipErrorOutOfMemory;
  ++g_live_allocs;
  return hipSuccess;
}
extern "C" hipError_t hipFree(void* p) {
  if (p) --g_live_allocs;
  std::free(p);
  return hipSuccess;
}
extern "C" hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
extern "C" hipError_t hipSetDevice(int) { return hipSuccess; }
extern "C" hipError_t hipGetLastError(void) { return hipSuccess; }

// ---- a minimal context for wisp_dual_resize: the cap and the budget call ------------------------
struct wisp_ctx {
  wisp_model_desc desc{};
  int32_t cap = 0;
  int fail_budget_at = 0;          // the n-th wisp_set_budget from now fails (WISP_E_NOMEM)
};
namespace wisp {
wisp_status set_error(wisp_status s, const std::string&) { return s; }
}  // namespace wisp
extern "C" wisp_status wisp_get_cap(wisp_ctx* c, int32_t* cap) {
  *cap = c->cap;
  return WISP_OK;
}
extern "C" wisp_status wisp_get_desc(wisp_ctx* c, wisp_model_desc* d) {
  *d = c->desc;
  return WISP_OK;
}
extern "C" wisp_status wisp_expert_bytes(const wisp_model_desc*, uint64_t* b) {
  *b = 1000;
  return WISP_OK;
}
extern "C" wisp_status wisp_set_budget(wisp_ctx* c, uint64_t bytes, int32_t* cap_out) {
  if (c->fail_budget_at > 0 && --c->fail_budget_at == 0) return WISP_E_NOMEM;
  c->cap = static_cast<int32_t>(bytes / (static_cast<uint64_t>(c->desc.n_layers) * 1000));
  if (cap_out) *cap_out = c->cap;
  return WISP_OK;
}

// ---- parts ---------------------------------------------------------------------------------------
static void check_slot_table(std::mt19937& rng) {
  for (int rep = 0; rep < 200; ++rep) {
    const int N = 1 + rng() % 96, C = 1 + rng() % N;
    wisp_slot_table* t = wisp_slot_table_create(N, C);
    CHECK(t);
    std::vector<int32_t> ids(40), hi(40), ms(40), mc(40), fi(96), fs(96);
    for (int s = 0; s < 60; ++s) {
      const int op = rng() % 10;
      const int cap = wisp_slot_table_cap(t);
      if (op == 0) {
        const int nc = 1 + rng() % N;
        CHECK(wisp_slot_table_resize(t, nc) == 0);
        continue;
      }
      const int n = static_cast<int>(rng() % 12);
      for (int i = 0; i < n; ++i) ids[i] = rng() % N;
      if (op == 1) {
        std::vector<int32_t> p;
        std::set<int32_t> seen;
        for (int i = 0; i < n && static_cast<int>(p.size()) < cap; ++i)
          if (seen.insert(ids[i]).second) p.push_back(ids[i]);
        const int m = wisp_slot_table_prefetch(t, p.empty() ? nullptr : p.data(), static_cast<int32_t>(p.size()),
                                               fi.data(), fs.data());
        CHECK(m >= 0 && m <= static_cast<int>(p.size()));
        for (int32_t e : p) CHECK(wisp_slot_table_slot_of(t, e) >= 0);
        continue;
      }
      int32_t h = 0, m = 0, ch = 0;
      CHECK(wisp_slot_table_step(t, ids.data(), n, &h, &m, &ch, hi.data(), ms.data(), mc.data()) == 0);
      std::set<int32_t> u(ids.begin(), ids.begin() + n);
      CHECK(h + m == static_cast<int>(u.size()));
      if (static_cast<int>(u.size()) <= cap)
        for (int32_t e : u) CHECK(wisp_slot_table_slot_of(t, e) >= 0);
      // the map is a bijection between resident experts and occupied slots
      int resident = 0;
      for (int e = 0; e < N; ++e) {
        const int sl = wisp_slot_table_slot_of(t, e);
        if (sl >= 0) {
          ++resident;
          CHECK(sl < wisp_slot_table_cap(t) && wisp_slot_table_expert_in(t, sl) == e);
        }
      }
      CHECK(resident <= wisp_slot_table_cap(t));
    }
    int32_t bad = N, h, m, ch;
    CHECK(wisp_slot_table_step(t, &bad, 1, &h, &m, &ch, hi.data(), ms.data(), mc.data()) != 0);
    wisp_slot_table_destroy(t);
  }
}

static void check_predictor(std::mt19937& rng) {
  for (int rep = 0; rep < 20; ++rep) {
    const int L = 1 + rng() % 6, N = 2 + rng() % 40, H = 1 + rng() % 6;
    wisp_predictor* p = nullptr;
    CHECK(wisp_predictor_create(L, N, H, 0.5, &p) == WISP_OK);
    std::vector<int32_t> ids(8), out(N);
    std::vector<double> sc(N);
    for (int pass = 0; pass < 12; ++pass) {
      for (int l = 0; l < L; ++l) {
        int32_t n = 0;
        CHECK(wisp_predictor_predict(p, l, 1 + rng() % N, out.data(), &n, sc.data()) == WISP_OK);
        CHECK(n >= 0 && n <= N);
        for (int i = 1; i < n; ++i) CHECK(sc[i - 1] >= sc[i]);
        const int k = 1 + rng() % 8;
        for (int i = 0; i < k; ++i) ids[i] = rng() % N;
        CHECK(wisp_predictor_observe(p, l, ids.data(), k) == WISP_OK);
      }
      CHECK(wisp_predictor_end_pass(p) == WISP_OK);
    }
    ids[0] = N;
    CHECK(wisp_predictor_observe(p, 0, ids.data(), 1) != WISP_OK);
    CHECK(wisp_predictor_destroy(p) == WISP_OK);
  }
}

static void check_allocator(std::mt19937& rng) {
  // miss curves: monotone, between first references and all references, upper >= lower
  for (int rep = 0; rep < 50; ++rep) {
    const int N = 1 + rng() % 64, steps = rng() % 200, refs = 1 + rng() % 8;
    std::vector<int32_t> ids(static_cast<size_t>(steps) * refs);
    for (auto& v : ids) v = rng() % N;
    std::vector<uint64_t> lo(N + 1), up(N + 1);
    CHECK(wisp_miss_curve(ids.empty() ? nullptr : ids.data(), steps, refs, N, lo.data(), up.data()) ==
          (ids.empty() ? WISP_E_INVAL : WISP_OK));
    if (ids.empty()) continue;
    for (int c = 0; c < N; ++c) CHECK(lo[c] >= lo[c + 1] && up[c] >= up[c + 1] && up[c] >= lo[c]);
    CHECK(lo[0] == up[0]);
    std::set<int32_t> distinct(ids.begin(), ids.end());
    CHECK(lo[N] == distinct.size());         // at C = N only first references miss
  }
  // configurator and control law on random problems
  for (int rep = 0; rep < 500; ++rep) {
    const int N = 1 + rng() % 40;
    const uint64_t a = 1 + rng() % 50, b = 1 + rng() % 20, B = 1 + rng() % (N * a + 400 * b);
    const int64_t kv_min = rng() % 30;
    std::vector<uint64_t> m_exp(N + 1);
    for (int c = 0; c <= N; ++c) m_exp[c] = static_cast<uint64_t>(N - c) * (1 + rng() % 3);
    std::vector<double> m_kv(1 + rng() % 300);
    for (size_t i = 0; i < m_kv.size(); ++i) m_kv[i] = static_cast<double>(m_kv.size() - i);
    wisp_mvwsa_problem pr{B, a, b, kv_min, 1.0, 0.5, N, static_cast<int64_t>(m_kv.size())};
    wisp_mvwsa_split sp{};
    const wisp_status s = wisp_mvwsa_configure(&pr, m_exp.data(), m_kv.data(), &sp);
    if (s == WISP_OK) CHECK(sp.cap >= 0 && sp.cap <= N && static_cast<uint64_t>(sp.cap) * a + sp.kv_bytes <= B);
    wisp_resize_law law{B, a, b, kv_min, 0.2, 0, N, static_cast<int32_t>(rng() % 3)};
    int32_t cap = 0, mv = 0;
    int64_t kv = 0;
    if (wisp_resize_target(&law, rng() % 500, static_cast<int32_t>(rng() % (N + 1)), &cap, &kv, &mv) == WISP_OK)
      CHECK(static_cast<uint64_t>(cap) * a + static_cast<uint64_t>(kv) * b <= B);
  }
  // KV pool on host memory: sizes, slack, an injected allocation failure
  wisp_kv_pool* pool = nullptr;
  CHECK(wisp_kv_pool_create(4096, 200, &pool) == WISP_OK);
  int64_t blocks = 0;
  for (int rep = 0; rep < 300; ++rep) {
    const int64_t want = rng() % 600;
    if (rng() % 7 == 0) g_fail_malloc_at = 1 + rng() % 3;
    CHECK(wisp_kv_pool_blocks(pool, &blocks) == WISP_OK);
    const int64_t before = blocks;
    const wisp_status s = wisp_kv_pool_resize(pool, want);
    CHECK(wisp_kv_pool_blocks(pool, &blocks) == WISP_OK);
    CHECK((s == WISP_OK && blocks == want) || (s == WISP_E_NOMEM && blocks == before));
    g_fail_malloc_at = 0;
  }
  // the controller driving the drained-barrier move on the fake context, with failures on both sides
  wisp_ctx ctx;
  ctx.desc.n_layers = 3;
  ctx.desc.n_experts = 64;
  ctx.cap = 16;
  const uint64_t a = 3 * 1000, b = 4096;
  CHECK(wisp_kv_pool_resize(pool, 100) == WISP_OK);
  const uint64_t B = 16 * a + 100 * b;
  wisp_resize_law law{B, a, b, 10, 0.2, 1, 64, 2};
  wisp_controller* ctl = nullptr;
  CHECK(wisp_controller_create(&law, 16, 100, &ctl) == WISP_OK);
  for (int barrier = 0; barrier < 200; ++barrier) {
    for (int s = 0; s < 8; ++s) CHECK(wisp_controller_observe(ctl, rng() % 140) == WISP_OK);
    const int f = rng() % 6;
    if (f == 0) g_fail_malloc_at = 1;
    if (f == 1) ctx.fail_budget_at = 1;
    int32_t cap = 0, moved = 0;
    int64_t kv = 0, peak = 0;
    CHECK(wisp_controller_barrier(ctl, &ctx, pool, &cap, &kv, &moved, &peak) == WISP_OK);
    g_fail_malloc_at = 0;
    ctx.fail_budget_at = 0;
    CHECK(wisp_kv_pool_blocks(pool, &blocks) == WISP_OK);
    CHECK(ctx.cap == cap && blocks == kv && static_cast<uint64_t>(cap) * a + static_cast<uint64_t>(kv) * b <= B);
  }
  CHECK(wisp_controller_destroy(ctl) == WISP_OK);
  CHECK(wisp_kv_pool_destroy(pool) == WISP_OK);
  CHECK(g_live_allocs == 0);
}

static void check_copy_pool(std::mt19937& rng) {
  std::vector<uint8_t> src(3u << 20), dst(3u << 20);
  for (auto& v : src) v = static_cast<uint8_t>(rng());
  for (int p = 0; p < 20; ++p) {
    wisp::CopyPool pool(1 + p % 6);
    const size_t n = 1 + rng() % src.size();
    std::memset(dst.data(), 0, dst.size());
    pool.copy(dst.data(), src.data(), n);
    CHECK(std::memcmp(dst.data(), src.data(), n) == 0);
  }
}

int main() {
  std::mt19937 rng(12345);
  check_slot_table(rng);
  check_predictor(rng);
  check_allocator(rng);
  check_copy_pool(rng);
  std::printf("ok\n");
  return 0;
}
