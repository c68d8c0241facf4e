// C ABI of the paged MoE layer: context, pinned expert masters, the expert pager (Algorithm 1 of
// WiSP, arXiv 2606.21868, Sec. 3.2) and the launch sequence of one layer-step.
//
// Streams and ordering.  The caller's stream carries the router, the FFN kernels and the combine.
// The library's side stream (non-blocking, default priority) carries the host->device fills.
// Per layer: the side stream waits for the layer's last FFN before overwriting victim slots
// (write-after-read), and the caller's stream waits for the fill event before the FFN of the
// faulted experts (read-after-write).  Resident experts' FFN is issued before that wait, so it
// overlaps the fills.  When the union of a layer-step exceeds C, chunk i+1's fills wait for
// chunk i's FFN.
#include <hip/hip_runtime.h>
#include <sys/mman.h>

#include <algorithm>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "slot_table.hpp"
#include "errors.hpp"
#include "staging.hpp"
#include "wisp.h"
#include "wisp_predictor.h"

#include <thread>

using namespace wisp;

namespace {

thread_local std::string g_err;

wisp_status fail(wisp_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

}  // namespace

wisp_status wisp::set_error(wisp_status s, const std::string& msg) { return fail(s, msg); }

namespace {

#define WISP_HIP(expr, what)                                                               \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail(WISP_E_HIP, std::string(what) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr size_t kMasterAlign = 4096;

struct TimedPair {
  hipEvent_t a, b;
  int kclass;
  uint64_t bytes;
  uint64_t flops;
};

struct LayerState {
  std::unique_ptr<SlotTable> table;
  std::vector<uint8_t*> slot_mem;
  const float* wr = nullptr;
  uint8_t* shared_dev = nullptr;
  hipEvent_t use_ev = nullptr;
  bool use_ev_recorded = false;
  std::vector<hipEvent_t> fill_ev;   // [2 * chunk + half]: that half of the chunk's fills has landed
  std::vector<hipEvent_t> chunk_ev;  // [2 * chunk + half]: the chunk's compute up to that half is done
  std::vector<std::vector<uint8_t>> late;   // per chunk, per expert: a fault of the chunk's second half
  bool pending = false;
  int32_t T = 0;
  std::vector<int32_t> ids;          // the routed ids, or (from_counts) the distinct experts
  bool from_counts = false;          // paged in from the device's per-expert pair counts
  StepPlan plan;
  std::vector<std::vector<const uint8_t*>> chunk_ptrs;
  wisp_page_stats cum{};
  // speculative prefetch (host pager): copies issued since the last forward that waited for them
  hipEvent_t pf_ev = nullptr;        // the layer's last prefetch copy has landed
  bool pf_pending = false;
  std::vector<int32_t> pf_inflight;  // experts whose prefetch copy is ordered before pf_ev
  std::vector<int32_t> pf_unused;    // prefetched since the last page-in, not yet routed to
  std::vector<int32_t> pf_req;       // ids requested for this layer by the last decode step
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

struct wisp_ctx {
  wisp_model_desc desc{};
  int device = 0;
  BlobLayout blob;
  FfnShape shape;
  size_t master_stride = 0;
  std::vector<uint8_t*> masters;
  std::vector<uint8_t*> shared_master;
  bool pageable = false;             // masters in pageable memory (mapped, not pinned)
  size_t master_map_bytes = 0;       // bytes of one layer's mapping (pageable masters)
  std::unique_ptr<BounceRing> bounce;
  int32_t cap = 0;
  std::vector<LayerState> layers;
  hipStream_t side = nullptr;
  float* logits = nullptr;
  void* h = nullptr;
  float* buf = nullptr;
  uint64_t* idx_tagged = nullptr;    // host-coherent (seq << 32 | id) words written by the router
  uint64_t* cnt_tagged = nullptr;    // host-coherent (seq << 32 | pairs) words, one per expert
  std::vector<int32_t> batch_cnt;    // a token batch's pairs per expert, from cnt_tagged
  std::vector<int32_t> batch_set;    // the experts with pairs, ascending
  uint32_t route_seq = 0;
  int32_t profile_mask = 0;          // kernel classes timed when profiling
  std::vector<int32_t> ids_scratch;
  bool profiling = false;
  std::vector<TimedPair> timed;
  std::vector<hipEvent_t> ev_pool;
  double k_ms[WISP_K_NUM] = {};
  uint64_t k_n[WISP_K_NUM] = {};
  uint64_t k_bytes[WISP_K_NUM] = {};
  uint64_t k_flops[WISP_K_NUM] = {};
  // token batches: the routed ids on the device and their expert-sorted order
  int32_t* ids_up = nullptr;         // pinned staging of the ids for the upload
  int32_t* d_ids = nullptr;          // [max_tokens * k]
  int32_t* d_perm = nullptr;         // [max_tokens * k]
  int32_t* d_perm_counts = nullptr;  // [segments of the pairs][N] scratch of the permutation
  hipEvent_t ids_ev = nullptr;       // the last upload has been read
  bool ids_ev_recorded = false;
  // the permutation of a token batch, computed from the device ids right after routing (while the
  // host pages the layer in) and used by the next wisp_moe_forward of that layer with the same ids
  hipEvent_t perm_ev = nullptr;      // the last early permutation is done
  hipEvent_t perm_use_ev = nullptr;  // the last grouped launches that read d_perm are done
  bool perm_ev_recorded = false, perm_use_recorded = false;
  hipStream_t perm_stream = nullptr; // the stream the last early permutation was enqueued on
  int32_t perm_layer = -1, perm_T = 0;
  std::vector<int32_t> perm_ids;     // the ids the early permutation was computed from
  std::vector<int32_t> e_cnt, e_off; // pairs per expert and their first sorted row
  std::vector<int32_t> pair_order;   // pairs sorted by expert (host copy, for the per-item path)
  // routing-blind static offload (comparison arm)
  struct Offload {
    bool on = false;
    int32_t mode = 0;                  // wisp_offload_mode
    int32_t resident_layers = 0;       // layers 0 .. R-1 hold all N experts in HBM
    uint8_t* resident = nullptr;       // [R][N] blobs at master_stride
    uint8_t* staging[2] = {nullptr, nullptr};
    hipEvent_t filled[2] = {nullptr, nullptr};
    hipEvent_t used[2] = {nullptr, nullptr};
    bool used_rec[2] = {false, false};
    int32_t next_copy = 0;             // streamed-layer sequence number of the next copy to issue
    int32_t next_use = 0;              // sequence number of the next streamed layer to compute
  } off;
  int32_t fail_alloc_at = 0;
  int32_t alloc_counter = 0;
  bool poison = false;               // debug: victim slots overwritten with NaN bytes before each fill
  // device pager (WISP_PAGER_DEVICE): the slot tables in HBM are authoritative while it is on
  int32_t pager = WISP_PAGER_HOST;
  int32_t dev_cap = 0;               // C the device arrays are sized for
  int32_t* d_pi = nullptr;           // [L][N]
  int32_t* d_pinv = nullptr;         // [L][C]
  uint64_t* d_tau = nullptr;         // [L][C]
  uint64_t* d_clock = nullptr;       // [L]
  uint64_t* d_slot_ptr = nullptr;    // [L][C] device addresses of the slots
  FfnBatch* d_plan = nullptr;        // launch plan written by the device pager
  uint32_t* d_stats = nullptr;       // [L][2] hits, misses of the current step
  uint32_t* h_stats = nullptr;       // pinned copy
  bool fusion = true;                // fused decode kernels (route + page; down + combine)
  uint64_t* d_logit_tags = nullptr;  // [4][N] tagged logit words of the one-launch router kernels
  uint32_t logit_tag = 0;            // tag of the last such launch (never 0)
  // speculative prefetch inside wisp_decode_step (host pager)
  int32_t pf_mode = WISP_PREFETCH_OFF;
  wisp_predictor* pf_pred = nullptr;
  int32_t pf_depth = 0;
  std::vector<int32_t> pf_hints;     // [L][pf_hint_n] for the next decode step, -1 = none
  int32_t pf_hint_n = 0;
  uint64_t pf_issued = 0, pf_useful = 0;
  std::vector<uint8_t> pf_mark;      // [N] scratch

  uint8_t* master(int l, int e) const { return masters[l] + static_cast<size_t>(e) * master_stride; }
  int k() const { return desc.top_k; }
  size_t h_elem() const { return shape.h_dtype == DT_F32 ? 4 : 2; }
  size_t x_elem() const { return desc.x_dtype == DT_F32 ? 4 : 2; }
};

namespace {

// ------------------------------------------------------------------------------------------
// profiling
// ------------------------------------------------------------------------------------------
hipEvent_t pool_event(wisp_ctx* c) {
  if (!c->ev_pool.empty()) {
    hipEvent_t e = c->ev_pool.back();
    c->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

LaunchTiming timing_begin(wisp_ctx* c, int kclass) {
  LaunchTiming t;
  if (c->profiling && ((c->profile_mask >> kclass) & 1)) {
    t.start = pool_event(c);
    t.stop = pool_event(c);
  }
  return t;
}

void timing_end(wisp_ctx* c, const LaunchTiming& t, int kclass, uint64_t bytes, uint64_t flops = 0) {
  if (!c->profiling || !t.start || !t.stop) return;
  c->timed.push_back({t.start, t.stop, kclass, bytes, flops});
}

// Accumulate every finished timed pair; with wait, first wait for all of them.
void harvest(wisp_ctx* c, bool wait) {
  size_t keep = 0;
  for (size_t i = 0; i < c->timed.size(); ++i) {
    TimedPair& p = c->timed[i];
    if (wait) (void)hipEventSynchronize(p.b);
    if (hipEventQuery(p.b) != hipSuccess) {
      c->timed[keep++] = p;
      continue;
    }
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      c->k_ms[p.kclass] += ms;
      c->k_n[p.kclass] += 1;
      c->k_bytes[p.kclass] += p.bytes;
      c->k_flops[p.kclass] += p.flops;
    } else {
      (void)hipGetLastError();   // a pair that could not be timed must not leave an error for the next launch check
    }
    c->ev_pool.push_back(p.a);
    c->ev_pool.push_back(p.b);
  }
  c->timed.resize(keep);
}

// The tag of the next one-launch router kernel: a sequence number that skips 0 (the words start at 0).
uint32_t next_logit_tag(wisp_ctx* c) {
  if (++c->logit_tag == 0) ++c->logit_tag;
  return c->logit_tag;
}

// ------------------------------------------------------------------------------------------
// validation helpers
// ------------------------------------------------------------------------------------------
wisp_status check_desc(const wisp_model_desc* d) {
  if (!d) return fail(WISP_E_INVAL, "desc is NULL");
  if (d->n_layers < 1 || d->d_model < 1 || d->d_ff < 1) return fail(WISP_E_INVAL, "non-positive shape");
  if (d->n_experts < 1 || d->n_experts > 256) return fail(WISP_E_INVAL, "n_experts must be in [1, 256]");
  if (d->top_k < 1 || d->top_k > 8 || d->top_k > d->n_experts) return fail(WISP_E_INVAL, "top_k must be in [1, min(8, N)]");
  if (d->max_tokens < 1) return fail(WISP_E_INVAL, "max_tokens must be >= 1");
  if (d->route < 0 || d->route > 2) return fail(WISP_E_INVAL, "unknown route");
  if (d->route == WISP_ROUTE_SIGMOID_GROUP) {
    if (d->n_groups < 1 || d->n_groups > 32 || d->n_experts % d->n_groups)
      return fail(WISP_E_INVAL, "n_groups must divide N and be <= 32");
    if (d->topk_groups < 1 || d->topk_groups > d->n_groups ||
        d->topk_groups * (d->n_experts / d->n_groups) < d->top_k)
      return fail(WISP_E_INVAL, "topk_groups too small for top_k");
  }
  const bool ok_pair = (d->w_dtype == WISP_F32 && d->x_dtype == WISP_F32) ||
                       (d->w_dtype == WISP_BF16 && d->x_dtype == WISP_BF16) ||
                       (d->w_dtype == WISP_FP8E4M3_B128 && d->x_dtype == WISP_BF16);
  if (!ok_pair) return fail(WISP_E_INVAL, "supported (weights, inputs): (f32, f32), (bf16, bf16), (fp8, bf16)");
  if (d->d_model % 16 || d->d_ff % 16) return fail(WISP_E_INVAL, "d_model and d_ff must be multiples of 16");
  if (d->w_dtype == WISP_FP8E4M3_B128 && (d->d_model % 128 || d->d_ff % 128))
    return fail(WISP_E_INVAL, "fp8 blocks need d_model and d_ff multiples of 128");
  const int epl = d->w_dtype == WISP_F32 ? 4 : d->w_dtype == WISP_BF16 ? 8 : 16;
  if ((d->d_model / epl) % 8 || (d->d_ff / epl) % 8)
    return fail(WISP_E_INVAL, "d_model and d_ff must be multiples of 8 x 16-byte chunks");
  if (d->has_shared != 0 && d->has_shared != 1) return fail(WISP_E_INVAL, "has_shared must be 0 or 1");
  if (d->pageable_masters != 0 && d->pageable_masters != 1) return fail(WISP_E_INVAL, "pageable_masters must be 0 or 1");
  return WISP_OK;
}

wisp_status check_ctx(wisp_ctx* c) {
  if (!c) return fail(WISP_E_INVAL, "ctx is NULL");
  hipError_t e = hipSetDevice(c->device);
  if (e != hipSuccess) return fail(WISP_E_HIP, std::string("hipSetDevice: ") + hipGetErrorString(e));
  return WISP_OK;
}

wisp_status check_layer(wisp_ctx* c, int32_t l) {
  if (l < 0 || l >= c->desc.n_layers) return fail(WISP_E_INVAL, "layer out of range");
  return WISP_OK;
}

void free_offload(wisp_ctx* c) {
  auto& o = c->off;
  if (c->side) (void)hipStreamSynchronize(c->side);
  for (int b = 0; b < 2; ++b) {
    if (o.used_rec[b]) (void)hipEventSynchronize(o.used[b]);
    if (o.staging[b]) (void)hipFree(o.staging[b]);
    if (o.filled[b]) (void)hipEventDestroy(o.filled[b]);
    if (o.used[b]) (void)hipEventDestroy(o.used[b]);
  }
  if (o.resident) (void)hipFree(o.resident);
  o = wisp_ctx::Offload{};
}

void free_ctx(wisp_ctx* c) {
  if (!c) return;
  free_offload(c);
  if (c->side) (void)hipStreamSynchronize(c->side);
  for (auto& L : c->layers) {
    if (L.use_ev_recorded) (void)hipEventSynchronize(L.use_ev);
  }
  (void)hipDeviceSynchronize();
  for (auto& L : c->layers) {
    for (auto* p : L.slot_mem) if (p) (void)hipFree(p);
    if (L.shared_dev) (void)hipFree(L.shared_dev);
    if (L.use_ev) (void)hipEventDestroy(L.use_ev);
    if (L.pf_ev) (void)hipEventDestroy(L.pf_ev);
    for (auto e : L.fill_ev) (void)hipEventDestroy(e);
    for (auto e : L.chunk_ev) (void)hipEventDestroy(e);
  }
  c->bounce.reset();
  for (auto* p : c->masters)
    if (p) c->pageable ? (void)munmap(p, c->master_map_bytes) : (void)hipHostFree(p);
  for (auto* p : c->shared_master)
    if (p) c->pageable ? (void)munmap(p, c->master_stride) : (void)hipHostFree(p);
  for (auto& t : c->timed) { (void)hipEventDestroy(t.a); (void)hipEventDestroy(t.b); }
  for (auto e : c->ev_pool) (void)hipEventDestroy(e);
  if (c->side) (void)hipStreamDestroy(c->side);
  if (c->logits) (void)hipFree(c->logits);
  if (c->h) (void)hipFree(c->h);
  if (c->buf) (void)hipFree(c->buf);
  if (c->idx_tagged) (void)hipHostFree(c->idx_tagged);
  if (c->cnt_tagged) (void)hipHostFree(c->cnt_tagged);
  if (c->ids_up) (void)hipHostFree(c->ids_up);
  if (c->d_ids) (void)hipFree(c->d_ids);
  if (c->d_perm) (void)hipFree(c->d_perm);
  if (c->d_perm_counts) (void)hipFree(c->d_perm_counts);
  if (c->ids_ev) (void)hipEventDestroy(c->ids_ev);
  if (c->perm_ev) (void)hipEventDestroy(c->perm_ev);
  if (c->perm_use_ev) (void)hipEventDestroy(c->perm_use_ev);
  for (void* p : {static_cast<void*>(c->d_pi), static_cast<void*>(c->d_pinv), static_cast<void*>(c->d_tau),
                  static_cast<void*>(c->d_clock), static_cast<void*>(c->d_slot_ptr), static_cast<void*>(c->d_plan),
                  static_cast<void*>(c->d_stats)})
    if (p) (void)hipFree(p);
  if (c->h_stats) (void)hipHostFree(c->h_stats);
  if (c->d_logit_tags) (void)hipFree(c->d_logit_tags);
  delete c;
}

wisp_status ensure_events(std::vector<hipEvent_t>& v, size_t n) {
  while (v.size() < n) {
    hipEvent_t e = nullptr;
    WISP_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreateWithFlags");
    v.push_back(e);
  }
  return WISP_OK;
}

// Drained barrier: every fill and every FFN of the context has finished.
wisp_status drain(wisp_ctx* c) {
  if (c->pager == WISP_PAGER_DEVICE) WISP_HIP(hipDeviceSynchronize(), "hipDeviceSynchronize");
  WISP_HIP(hipStreamSynchronize(c->side), "hipStreamSynchronize(side)");
  for (auto& L : c->layers) {
    if (L.use_ev_recorded) WISP_HIP(hipEventSynchronize(L.use_ev), "hipEventSynchronize(layer)");
    L.pf_pending = false;
    L.pf_inflight.clear();
  }
  return WISP_OK;
}

// Copy every layer's slot table (and slot addresses) host -> device, resizing the device arrays
// to the current cap.  Synchronous.
wisp_status upload_tables(wisp_ctx* c) {
  const int L = c->desc.n_layers, N = c->desc.n_experts, C = c->cap;
  if (c->dev_cap != C) {
    for (void** p : {reinterpret_cast<void**>(&c->d_pinv), reinterpret_cast<void**>(&c->d_tau),
                     reinterpret_cast<void**>(&c->d_slot_ptr)}) {
      if (*p) (void)hipFree(*p);
      *p = nullptr;
    }
    c->dev_cap = 0;
    if (hipMalloc(reinterpret_cast<void**>(&c->d_pinv), sizeof(int32_t) * L * C) != hipSuccess ||
        hipMalloc(reinterpret_cast<void**>(&c->d_tau), sizeof(uint64_t) * L * C) != hipSuccess ||
        hipMalloc(reinterpret_cast<void**>(&c->d_slot_ptr), sizeof(uint64_t) * L * C) != hipSuccess)
      return fail(WISP_E_NOMEM, "device pager tables");
    c->dev_cap = C;
  }
  if (!c->d_pi) {
    if (hipMalloc(reinterpret_cast<void**>(&c->d_pi), sizeof(int32_t) * L * N) != hipSuccess ||
        hipMalloc(reinterpret_cast<void**>(&c->d_clock), sizeof(uint64_t) * L) != hipSuccess ||
        hipMalloc(reinterpret_cast<void**>(&c->d_plan), sizeof(FfnBatch)) != hipSuccess ||
        hipMalloc(reinterpret_cast<void**>(&c->d_stats), sizeof(uint32_t) * 2 * L) != hipSuccess ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_stats), sizeof(uint32_t) * 2 * L, hipHostMallocDefault) != hipSuccess)
      return fail(WISP_E_NOMEM, "device pager state");
  }
  std::vector<int32_t> pi(static_cast<size_t>(L) * N), pinv(static_cast<size_t>(L) * C);
  std::vector<uint64_t> tau(static_cast<size_t>(L) * C), clk(L), sp(static_cast<size_t>(L) * C);
  for (int l = 0; l < L; ++l) {
    c->layers[l].table->export_state(&pi[static_cast<size_t>(l) * N], &pinv[static_cast<size_t>(l) * C],
                                     &tau[static_cast<size_t>(l) * C], &clk[l]);
    for (int s = 0; s < C; ++s) sp[static_cast<size_t>(l) * C + s] = reinterpret_cast<uint64_t>(c->layers[l].slot_mem[s]);
  }
  WISP_HIP(hipMemcpy(c->d_pi, pi.data(), sizeof(int32_t) * pi.size(), hipMemcpyHostToDevice), "upload pi");
  WISP_HIP(hipMemcpy(c->d_pinv, pinv.data(), sizeof(int32_t) * pinv.size(), hipMemcpyHostToDevice), "upload pinv");
  WISP_HIP(hipMemcpy(c->d_tau, tau.data(), sizeof(uint64_t) * tau.size(), hipMemcpyHostToDevice), "upload tau");
  WISP_HIP(hipMemcpy(c->d_clock, clk.data(), sizeof(uint64_t) * clk.size(), hipMemcpyHostToDevice), "upload clock");
  WISP_HIP(hipMemcpy(c->d_slot_ptr, sp.data(), sizeof(uint64_t) * sp.size(), hipMemcpyHostToDevice), "upload slots");
  return WISP_OK;
}

// Copy the device slot tables back into the host tables.  Synchronous; call after drain().
wisp_status download_tables(wisp_ctx* c) {
  const int L = c->desc.n_layers, N = c->desc.n_experts, C = c->cap;
  std::vector<int32_t> pi(static_cast<size_t>(L) * N), pinv(static_cast<size_t>(L) * C);
  std::vector<uint64_t> tau(static_cast<size_t>(L) * C), clk(L);
  WISP_HIP(hipDeviceSynchronize(), "hipDeviceSynchronize");
  WISP_HIP(hipMemcpy(pi.data(), c->d_pi, sizeof(int32_t) * pi.size(), hipMemcpyDeviceToHost), "download pi");
  WISP_HIP(hipMemcpy(pinv.data(), c->d_pinv, sizeof(int32_t) * pinv.size(), hipMemcpyDeviceToHost), "download pinv");
  WISP_HIP(hipMemcpy(tau.data(), c->d_tau, sizeof(uint64_t) * tau.size(), hipMemcpyDeviceToHost), "download tau");
  WISP_HIP(hipMemcpy(clk.data(), c->d_clock, sizeof(uint64_t) * clk.size(), hipMemcpyDeviceToHost), "download clock");
  for (int l = 0; l < L; ++l)
    c->layers[l].table->import_state(&pi[static_cast<size_t>(l) * N], &pinv[static_cast<size_t>(l) * C],
                                     &tau[static_cast<size_t>(l) * C], clk[l]);
  return WISP_OK;
}

// Run `body` on the host tables: with the device pager on, move them down first and back up after.
template <typename F>
wisp_status with_host_tables(wisp_ctx* c, F body) {
  const bool dev = c->pager == WISP_PAGER_DEVICE;
  wisp_status s;
  if (dev) {
    if ((s = drain(c)) != WISP_OK) return s;
    if ((s = download_tables(c)) != WISP_OK) return s;
  }
  wisp_status r = body();
  if (dev && (s = upload_tables(c)) != WISP_OK) return s;
  return r;
}

// Enqueue the fills of chunk ci of `layer`'s pending plan on the side stream.
// host master -> device copy on `st`: one DMA copy from pinned masters, or staged through the
// pinned bounce ring from pageable ones.
wisp_status master_h2d(wisp_ctx* c, void* dst, const uint8_t* src, size_t bytes, hipStream_t st) {
  if (!c->pageable) {
    WISP_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, st), "hipMemcpyAsync(master)");
  } else {
    WISP_HIP(c->bounce->copy_to_device(dst, src, bytes, st), "staged copy(master)");
  }
  return WISP_OK;
}

// (expert, slot) blobs of `layer` into their slots on the side stream.  Token batches with pinned
// masters: the compute units stream them over the host link (one launch per up to kMaxFills blobs;
// 4 % faster than a copy-engine copy per blob on the cold prefill pass).  Decode steps: a copy-engine
// copy per blob, because the fills run beside the GEMV over the resident experts and compute-unit
// reads of host memory slow it down (8.4 -> 12 us median, and far more at the tail).  Pageable
// masters: staged through the bounce ring.
wisp_status fill_slots(wisp_ctx* c, int32_t layer, const std::vector<std::pair<int32_t, int32_t>>& fills,
                       bool by_cus) {
  LayerState& L = c->layers[layer];
  if (c->pageable || !by_cus) {
    for (const auto& f : fills) {
      wisp_status s = master_h2d(c, L.slot_mem[f.second], c->master(layer, f.first), c->blob.bytes, c->side);
      if (s != WISP_OK) return s;
    }
    return WISP_OK;
  }
  FillList fl;
  fl.n = 0;
  for (const auto& f : fills) {
    fl.src[fl.n] = c->master(layer, f.first);
    fl.dst[fl.n] = L.slot_mem[f.second];
    if (++fl.n == kMaxFills) {
      WISP_HIP(launch_fill(fl, c->blob.bytes, c->side, LaunchTiming{}), "fill launch");
      fl.n = 0;
    }
  }
  WISP_HIP(launch_fill(fl, c->blob.bytes, c->side, LaunchTiming{}), "fill launch");
  return WISP_OK;
}

// Debug hazard check: after the side stream's write-after-read wait, fill each victim slot with 0xFF
// bytes (NaN in fp32, bf16 and E4M3, and in the bf16 block scales) before its copy.  A read of a slot
// that is not ordered after its fill, or a fill not ordered after the slot's last read, then shows up
// as NaN in the outputs instead of as plausible stale weights.
wisp_status poison_slots(wisp_ctx* c, int32_t layer, const std::vector<std::pair<int32_t, int32_t>>& fills) {
  if (!c->poison) return WISP_OK;
  LayerState& L = c->layers[layer];
  for (const auto& f : fills)
    WISP_HIP(hipMemsetAsync(L.slot_mem[f.second], 0xFF, c->blob.bytes, c->side), "hipMemsetAsync(poison)");
  return WISP_OK;
}

// The fills of chunk ci on the side stream, in two halves with an event each (fill_ev[2 ci + h]).
// With several chunks in a layer-step, a fill waits only for the part of the previous chunk's compute
// that read its victim slot: that chunk's hits and first half (chunk_ev[2 (ci - 1)]) or its second
// half (chunk_ev[2 (ci - 1) + 1]).  Faults whose victim the previous chunk's second half read form
// this chunk's second half; chunk 0 splits its faults in the middle.  The link then streams a
// chunk's first half while the previous chunk's second half computes, instead of idling for the
// previous chunk's whole compute.  A single chunk keeps every fault in the first half.
wisp_status issue_fills(wisp_ctx* c, int32_t layer, size_t ci) {
  LayerState& L = c->layers[layer];
  const ChunkPlan& cp = L.plan.chunks[ci];
  const size_t nch = L.plan.chunks.size();
  std::vector<uint8_t>& late = L.late[ci];
  late.assign(cp.experts.size(), 0);
  if (cp.n_faults == 0) return WISP_OK;   // nothing waits for this chunk's fill events
  if (nch > 1 && ci == 0) {
    int32_t nf = 0;
    for (size_t i = 0; i < cp.experts.size(); ++i)
      if (cp.fault[i]) late[i] = nf++ >= (cp.n_faults + 1) / 2 ? 1 : 0;
  } else if (nch > 1) {
    const ChunkPlan& pp = L.plan.chunks[ci - 1];
    std::vector<uint8_t> read_late(static_cast<size_t>(c->cap), 0);
    for (size_t i = 0; i < pp.experts.size(); ++i)
      if (L.late[ci - 1][i]) read_late[pp.slots[i]] = 1;
    for (size_t i = 0; i < cp.experts.size(); ++i)
      if (cp.fault[i]) late[i] = read_late[cp.slots[i]];
  }
  std::vector<std::pair<int32_t, int32_t>> fills[2];
  for (size_t i = 0; i < cp.experts.size(); ++i)
    if (cp.fault[i]) fills[late[i]].push_back({cp.experts[i], cp.slots[i]});
  const bool batch = L.T >= kGroupedMinTokens && grouped_supported(c->shape, c->desc.has_shared);
  for (int h = 0; h < (nch > 1 ? 2 : 1); ++h) {   // a single chunk has one half
    if (ci == 0) {
      if (h == 0 && L.use_ev_recorded) WISP_HIP(hipStreamWaitEvent(c->side, L.use_ev, 0), "hipStreamWaitEvent(use)");
    } else {
      WISP_HIP(hipStreamWaitEvent(c->side, L.chunk_ev[2 * (ci - 1) + h], 0), "hipStreamWaitEvent(chunk)");
    }
    if (!fills[h].empty()) {
      LaunchTiming tm = timing_begin(c, WISP_K_H2D_FILL);
      if (tm.start) WISP_HIP(hipEventRecord(tm.start, c->side), "hipEventRecord");
      wisp_status s = poison_slots(c, layer, fills[h]);
      if (s != WISP_OK) return s;
      s = fill_slots(c, layer, fills[h], batch);
      if (s != WISP_OK) return s;
      if (tm.stop) WISP_HIP(hipEventRecord(tm.stop, c->side), "hipEventRecord");
      timing_end(c, tm, WISP_K_H2D_FILL, static_cast<uint64_t>(fills[h].size()) * c->blob.bytes);
    }
    WISP_HIP(hipEventRecord(L.fill_ev[2 * ci + h], c->side), "hipEventRecord(fill)");
  }
  return WISP_OK;
}

uint64_t ffn_bytes(const wisp_ctx* c, const FfnBatch& b, bool gateup) {
  const BlobLayout& B = c->blob;
  const uint64_t n = static_cast<uint64_t>(B.d) * B.I;
  const uint64_t nb = B.w_dtype == DT_FP8 ? static_cast<uint64_t>(B.d / 128) * (B.I / 128) * 2 : 0;
  uint64_t bytes = 0;
  for (int i = 0; i < b.n_items; ++i) {
    const uint64_t nt = b.items[i].ntok;
    if (gateup) bytes += 2 * n * B.elem + 2 * nb + nt * (B.d * c->x_elem() + B.I * c->h_elem());
    else bytes += n * B.elem + nb + nt * (B.I * c->h_elem() + B.d * 4);
  }
  return bytes;
}

// Launch gate/up then down for a list of (expert blob, (token, rank) pairs), in batches of up to
// kMaxItems items; the per-(token, rank) outputs land in buf.
struct Pair { int32_t t, out; };
struct Work { const uint8_t* w; std::vector<Pair> pairs; };

wisp_status run_ffn(wisp_ctx* c, const std::vector<Work>& work, const void* x, hipStream_t st, bool down = true) {
  FfnBatch b;
  b.n_items = 0;
  b.max_ntok = 0;
  auto flush = [&]() -> wisp_status {
    if (b.n_items == 0) return WISP_OK;
    LaunchTiming t1 = timing_begin(c, WISP_K_FFN_GATEUP);
    WISP_HIP(launch_ffn_gateup(b, c->shape, x, c->h, st, t1), "ffn gate/up launch");
    timing_end(c, t1, WISP_K_FFN_GATEUP, ffn_bytes(c, b, true));
    if (down) {
      LaunchTiming t2 = timing_begin(c, WISP_K_FFN_DOWN);
      WISP_HIP(launch_ffn_down(b, c->shape, c->h, c->buf, st, t2), "ffn down launch");
      timing_end(c, t2, WISP_K_FFN_DOWN, ffn_bytes(c, b, false));
    }
    b.n_items = 0;
    b.max_ntok = 0;
    return WISP_OK;
  };
  for (const Work& wk : work) {
    for (size_t p0 = 0; p0 < wk.pairs.size(); p0 += kMaxTokPerItem) {
      if (b.n_items == kMaxItems) {
        wisp_status s = flush();
        if (s != WISP_OK) return s;
      }
      FfnItem& it = b.items[b.n_items++];
      it.w = wk.w;
      it.src = nullptr;
      it.fault = 0;
      it.ntok = static_cast<int32_t>(std::min<size_t>(kMaxTokPerItem, wk.pairs.size() - p0));
      for (int q = 0; q < kMaxTokPerItem; ++q) {
        const bool on = q < it.ntok;
        it.tok[q] = on ? wk.pairs[p0 + q].t : 0;
        it.out[q] = on ? wk.pairs[p0 + q].out : 0;
      }
      b.max_ntok = std::max(b.max_ntok, it.ntok);
    }
  }
  return flush();
}

// Speculative prefetch of ids[0..n) into `layer`'s slots (host pager).  Validated by the caller.
wisp_status prefetch_layer(wisp_ctx* c, int32_t layer, const int32_t* ids, int32_t n) {
  LayerState& L = c->layers[layer];
  std::vector<std::pair<int32_t, int32_t>> fills;
  if (!L.table->prefetch(ids, n, &fills)) return fail(WISP_E_INVAL, "expert id out of range");
  if (fills.empty()) return WISP_OK;
  if (L.use_ev_recorded) WISP_HIP(hipStreamWaitEvent(c->side, L.use_ev, 0), "hipStreamWaitEvent(use)");
  LaunchTiming tm = timing_begin(c, WISP_K_H2D_FILL);
  if (tm.start) WISP_HIP(hipEventRecord(tm.start, c->side), "hipEventRecord");
  wisp_status s = poison_slots(c, layer, fills);
  if (s != WISP_OK) return s;
  s = fill_slots(c, layer, fills, false);
  if (s != WISP_OK) return s;
  for (const auto& f : fills) {
    L.pf_inflight.push_back(f.first);
    L.pf_unused.push_back(f.first);
  }
  if (tm.stop) WISP_HIP(hipEventRecord(tm.stop, c->side), "hipEventRecord");
  timing_end(c, tm, WISP_K_H2D_FILL, static_cast<uint64_t>(fills.size()) * c->blob.bytes);
  WISP_HIP(hipEventRecord(L.pf_ev, c->side), "hipEventRecord(prefetch)");
  L.pf_pending = true;
  c->pf_issued += fills.size();
  return WISP_OK;
}

// The prefetch wisp_decode_step issues for `layer` before routing it: the predictor's top `depth`
// from the layers already routed in this pass, or the hints given for this step.
wisp_status prefetch_before_route(wisp_ctx* c, int32_t layer) {
  std::vector<int32_t>& ids = c->layers[layer].pf_req;
  ids.clear();
  if (c->pf_mode == WISP_PREFETCH_OFF) return WISP_OK;
  if (c->pf_mode == WISP_PREFETCH_PREDICTOR) {
    if (layer == 0 || c->pf_depth < 1) return WISP_OK;
    ids.resize(c->pf_depth);
    int32_t n = 0;
    wisp_status s = wisp_predictor_predict(c->pf_pred, layer, c->pf_depth, ids.data(), &n, nullptr);
    if (s != WISP_OK) return s;
    ids.resize(n);
  } else {
    if (c->pf_hint_n < 1) return WISP_OK;
    const int32_t* h = &c->pf_hints[static_cast<size_t>(layer) * c->pf_hint_n];
    for (int32_t i = 0; i < c->pf_hint_n; ++i)
      if (h[i] >= 0) ids.push_back(h[i]);
  }
  if (ids.empty()) return WISP_OK;
  return prefetch_layer(c, layer, ids.data(), static_cast<int32_t>(ids.size()));
}

}  // namespace

// ==========================================================================================
// C ABI
// ==========================================================================================
extern "C" {

const char* wisp_last_error(void) { return g_err.c_str(); }

wisp_status wisp_expert_bytes(const wisp_model_desc* desc, uint64_t* bytes) {
  wisp_status s = check_desc(desc);
  if (s != WISP_OK) return s;
  if (!bytes) return fail(WISP_E_INVAL, "bytes is NULL");
  *bytes = make_blob_layout(desc->d_model, desc->d_ff, desc->w_dtype).bytes;
  return WISP_OK;
}

wisp_status wisp_create(const wisp_model_desc* desc, wisp_ctx** out) {
  if (!out) return fail(WISP_E_INVAL, "out is NULL");
  *out = nullptr;
  wisp_status s = check_desc(desc);
  if (s != WISP_OK) return s;
  auto* c = new (std::nothrow) wisp_ctx();
  if (!c) return fail(WISP_E_NOMEM, "host allocation failed");
  c->desc = *desc;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return fail(WISP_E_HIP, "hipGetDevice failed (no GPU?)");
  }
  c->blob = make_blob_layout(desc->d_model, desc->d_ff, desc->w_dtype);
  c->shape.blob = c->blob;
  c->shape.x_dtype = desc->x_dtype;
  c->shape.h_dtype = desc->w_dtype == WISP_F32 ? DT_F32 : DT_BF16;
  c->master_stride = round_up(c->blob.bytes, kMasterAlign);
  const int L = desc->n_layers, N = desc->n_experts, k = desc->top_k, T = desc->max_tokens;
  c->layers.resize(L);
  c->masters.assign(L, nullptr);
  c->shared_master.assign(L, nullptr);
  auto bail = [&](wisp_status st, const std::string& m) {
    free_ctx(c);
    return fail(st, m);
  };
  c->pageable = desc->pageable_masters != 0;
  c->master_map_bytes = static_cast<size_t>(N) * c->master_stride;
  auto host_alloc = [&](size_t bytes) -> uint8_t* {
    if (c->pageable) {
      void* m = mmap(nullptr, bytes, PROT_READ | PROT_WRITE, MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE, -1, 0);
      return m == MAP_FAILED ? nullptr : static_cast<uint8_t*>(m);
    }
    void* m = nullptr;
    if (hipHostMalloc(&m, bytes, hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    return static_cast<uint8_t*>(m);
  };
  if (c->pageable) {
    c->bounce.reset(new (std::nothrow) BounceRing());
    const int hw = static_cast<int>(std::thread::hardware_concurrency());
    if (!c->bounce || c->bounce->init(std::max(1, std::min(8, hw))) != hipSuccess)
      return bail(WISP_E_NOMEM, "pinned bounce buffers for the pageable masters");
  }
  for (int l = 0; l < L; ++l) {
    void* p = nullptr;
    c->masters[l] = host_alloc(c->master_map_bytes);
    if (!c->masters[l])
      return bail(WISP_E_NOMEM, c->pageable ? "mapping the pageable expert masters failed"
                                            : "hipHostMalloc of the expert masters failed (pinned memory limit? "
                                              "set pageable_masters)");
    if (desc->has_shared) {
      c->shared_master[l] = host_alloc(c->master_stride);
      if (!c->shared_master[l]) return bail(WISP_E_NOMEM, "allocating the shared-expert master failed");
      if (hipMalloc(&p, c->blob.bytes) != hipSuccess) return bail(WISP_E_NOMEM, "hipMalloc of a shared expert failed");
      c->layers[l].shared_dev = static_cast<uint8_t*>(p);
    }
    if (hipEventCreateWithFlags(&c->layers[l].use_ev, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&c->layers[l].pf_ev, hipEventDisableTiming) != hipSuccess)
      return bail(WISP_E_HIP, "hipEventCreate failed");
  }
  if (hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) != hipSuccess)
    return bail(WISP_E_HIP, "hipStreamCreateWithFlags failed");
  void* p = nullptr;
  if (hipMalloc(&p, sizeof(float) * kRouterMaxSplit * static_cast<size_t>(T) * N) != hipSuccess)
    return bail(WISP_E_NOMEM, "scratch");
  c->logits = static_cast<float*>(p);
  const size_t rows = static_cast<size_t>(T) * (k + 1);
  if (hipMalloc(&c->h, rows * desc->d_ff * c->h_elem()) != hipSuccess) return bail(WISP_E_NOMEM, "scratch");
  if (hipMalloc(&p, rows * desc->d_model * sizeof(float)) != hipSuccess) return bail(WISP_E_NOMEM, "scratch");
  c->buf = static_cast<float*>(p);
  if (hipHostMalloc(&p, sizeof(uint64_t) * static_cast<size_t>(T) * k, hipHostMallocCoherent) != hipSuccess)
    return bail(WISP_E_NOMEM, "pinned scratch");
  c->idx_tagged = static_cast<uint64_t*>(p);
  std::memset(c->idx_tagged, 0, sizeof(uint64_t) * static_cast<size_t>(T) * k);
  if (hipHostMalloc(&p, sizeof(uint64_t) * N, hipHostMallocCoherent) != hipSuccess)
    return bail(WISP_E_NOMEM, "pinned scratch");
  c->cnt_tagged = static_cast<uint64_t*>(p);
  std::memset(c->cnt_tagged, 0, sizeof(uint64_t) * N);
  c->batch_cnt.assign(N, 0);
  c->batch_set.reserve(N);
  c->ids_scratch.resize(static_cast<size_t>(T) * k);
  const size_t pairs_bytes = sizeof(int32_t) * static_cast<size_t>(T) * k;
  if (hipHostMalloc(&p, pairs_bytes, hipHostMallocDefault) != hipSuccess) return bail(WISP_E_NOMEM, "pinned scratch");
  c->ids_up = static_cast<int32_t*>(p);
  if (hipMalloc(&p, pairs_bytes) != hipSuccess) return bail(WISP_E_NOMEM, "scratch");
  c->d_ids = static_cast<int32_t*>(p);
  if (hipMalloc(&p, pairs_bytes) != hipSuccess) return bail(WISP_E_NOMEM, "scratch");
  c->d_perm = static_cast<int32_t*>(p);
  if (hipMalloc(&p, sizeof(int32_t) * static_cast<size_t>(permute_segments(T * k)) * N) != hipSuccess)
    return bail(WISP_E_NOMEM, "scratch");
  c->d_perm_counts = static_cast<int32_t*>(p);
  if (hipEventCreateWithFlags(&c->ids_ev, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->perm_ev, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->perm_use_ev, hipEventDisableTiming) != hipSuccess)
    return bail(WISP_E_HIP, "hipEventCreate failed");
  c->e_cnt.assign(N, 0);
  c->e_off.assign(N + 1, 0);
  c->pf_mark.assign(N, 0);
  if (hipMalloc(&p, sizeof(uint64_t) * 4 * N) != hipSuccess) return bail(WISP_E_NOMEM, "scratch");
  c->d_logit_tags = static_cast<uint64_t*>(p);
  if (hipMemset(c->d_logit_tags, 0, sizeof(uint64_t) * 4 * N) != hipSuccess)
    return bail(WISP_E_HIP, "hipMemset(logit tags)");

  c->pair_order.resize(static_cast<size_t>(T) * k);
  *out = c;
  g_err.clear();
  return WISP_OK;
}

wisp_status wisp_destroy(wisp_ctx* ctx) {
  if (!ctx) return fail(WISP_E_INVAL, "ctx is NULL");
  (void)hipSetDevice(ctx->device);
  free_ctx(ctx);
  return WISP_OK;
}

wisp_status wisp_expert_host_ptr(wisp_ctx* ctx, int32_t layer, int32_t expert, void** ptr, uint64_t* bytes) {
  if (!ctx || !ptr) return fail(WISP_E_INVAL, "NULL argument");
  wisp_status s = check_layer(ctx, layer);
  if (s != WISP_OK) return s;
  if (expert == -1) {
    if (!ctx->desc.has_shared) return fail(WISP_E_INVAL, "model has no shared expert");
    *ptr = ctx->shared_master[layer];
  } else {
    if (expert < 0 || expert >= ctx->desc.n_experts) return fail(WISP_E_INVAL, "expert out of range");
    *ptr = ctx->master(layer, expert);
  }
  if (bytes) *bytes = ctx->blob.bytes;
  return WISP_OK;
}

static wisp_status masters_ready_host(wisp_ctx* ctx) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  s = drain(ctx);
  if (s != WISP_OK) return s;
  for (auto& L : ctx->layers)
    if (L.pending) return fail(WISP_E_STATE, "a page-in is pending");
  for (int l = 0; l < ctx->desc.n_layers; ++l) {
    LayerState& L = ctx->layers[l];
    if (ctx->desc.has_shared &&
        (s = master_h2d(ctx, L.shared_dev, ctx->shared_master[l], ctx->blob.bytes, ctx->side)) != WISP_OK)
      return s;
    if (L.table) L.table->clear();
  }
  WISP_HIP(hipStreamSynchronize(ctx->side), "hipStreamSynchronize(side)");
  return WISP_OK;
}

wisp_status wisp_router_weights(wisp_ctx* ctx, int32_t layer, const float* w_r_dev) {
  if (!ctx || !w_r_dev) return fail(WISP_E_INVAL, "NULL argument");
  wisp_status s = check_layer(ctx, layer);
  if (s != WISP_OK) return s;
  ctx->layers[layer].wr = w_r_dev;
  return WISP_OK;
}

static wisp_status set_budget_host(wisp_ctx* ctx, uint64_t expert_bytes, int32_t* cap_out) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  const uint64_t a = static_cast<uint64_t>(ctx->desc.n_layers) * ctx->blob.bytes;
  const uint64_t cap64 = expert_bytes / a;
  if (cap64 < 1 || cap64 > static_cast<uint64_t>(ctx->desc.n_experts))
    return fail(WISP_E_INVAL, "budget gives a cap outside [1, N]: C = floor(B / (L * M_e)) = " + std::to_string(cap64));
  const int32_t C = static_cast<int32_t>(cap64);
  for (auto& L : ctx->layers)
    if (L.pending) return fail(WISP_E_STATE, "a page-in is pending");
  s = drain(ctx);
  if (s != WISP_OK) return s;
  if (cap_out) *cap_out = C;
  const int32_t old = ctx->cap;
  if (C == old) return WISP_OK;
  const int nl = ctx->desc.n_layers;
  if (C > old) {
    // grow: allocate every new slot first; commit only if all succeed
    std::vector<std::vector<uint8_t*>> fresh(nl);
    bool ok = true;
    std::string why;
    for (int l = 0; l < nl && ok; ++l) {
      for (int32_t i = old; i < C; ++i) {
        ++ctx->alloc_counter;
        void* p = nullptr;
        if (ctx->fail_alloc_at > 0 && ctx->alloc_counter == ctx->fail_alloc_at) {
          ctx->fail_alloc_at = 0;
          ok = false;
          why = "injected slot allocation failure";
          break;
        }
        if (hipMalloc(&p, ctx->blob.bytes) != hipSuccess) {
          ok = false;
          why = "hipMalloc of an expert slot failed";
          (void)hipGetLastError();
          break;
        }
        fresh[l].push_back(static_cast<uint8_t*>(p));
      }
    }
    if (!ok) {
      for (auto& v : fresh)
        for (auto* p : v) (void)hipFree(p);
      return fail(WISP_E_NOMEM, why + "; previous budget kept");
    }
    for (int l = 0; l < nl; ++l) {
      LayerState& L = ctx->layers[l];
      if (!L.table) {
        L.table.reset(new SlotTable(ctx->desc.n_experts, C));
      } else {
        std::vector<int32_t> map;
        L.table->resize(C, &map);
      }
      L.slot_mem.insert(L.slot_mem.end(), fresh[l].begin(), fresh[l].end());
    }
  } else {
    // shrink: keep the most recently used experts, free the rest of the slots first
    for (int l = 0; l < nl; ++l) {
      LayerState& L = ctx->layers[l];
      std::vector<int32_t> map;
      L.table->resize(C, &map);
      std::vector<uint8_t> used(old, 0);
      std::vector<uint8_t*> mem(C, nullptr);
      for (int32_t i = 0; i < C; ++i)
        if (map[i] >= 0) { mem[i] = L.slot_mem[map[i]]; used[map[i]] = 1; }
      int32_t spare = 0;
      for (int32_t i = 0; i < C; ++i) {
        if (mem[i]) continue;
        while (used[spare]) ++spare;
        mem[i] = L.slot_mem[spare];
        used[spare] = 1;
      }
      for (int32_t s2 = 0; s2 < old; ++s2)
        if (!used[s2]) (void)hipFree(L.slot_mem[s2]);
      L.slot_mem.swap(mem);
    }
  }
  ctx->cap = C;
  return WISP_OK;
}

static wisp_status preload_host(wisp_ctx* ctx) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (ctx->cap < 1) return fail(WISP_E_STATE, "no expert budget set");
  for (auto& L : ctx->layers)
    if (L.pending) return fail(WISP_E_STATE, "a page-in is pending");
  if ((s = drain(ctx)) != WISP_OK) return s;
  std::vector<int32_t> ids(ctx->cap);
  for (int32_t i = 0; i < ctx->cap; ++i) ids[i] = i;
  for (int32_t l = 0; l < ctx->desc.n_layers; ++l) {
    LayerState& L = ctx->layers[l];
    StepPlan plan;
    L.table->step(ids.data(), ctx->cap, &plan);
    for (const ChunkPlan& cp : plan.chunks)
      for (size_t i = 0; i < cp.experts.size(); ++i)
        if (cp.fault[i])
          if ((s = master_h2d(ctx, L.slot_mem[cp.slots[i]], ctx->master(l, cp.experts[i]), ctx->blob.bytes,
                              ctx->side)) != WISP_OK)
            return s;
  }
  WISP_HIP(hipStreamSynchronize(ctx->side), "hipStreamSynchronize(side)");
  return WISP_OK;
}

wisp_status wisp_masters_ready(wisp_ctx* ctx) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (ctx->pager == WISP_PAGER_DEVICE && ctx->cap > 0)
    return with_host_tables(ctx, [&] { return masters_ready_host(ctx); });
  return masters_ready_host(ctx);
}

wisp_status wisp_set_budget(wisp_ctx* ctx, uint64_t expert_bytes, int32_t* cap_out) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (ctx->pager == WISP_PAGER_DEVICE) {
    const uint64_t C = expert_bytes / (static_cast<uint64_t>(ctx->desc.n_layers) * ctx->blob.bytes);
    if (C < static_cast<uint64_t>(ctx->desc.max_tokens) * ctx->desc.top_k)
      return fail(WISP_E_INVAL, "the device pager needs C >= max_tokens * k; switch to the host pager first");
    return with_host_tables(ctx, [&] { return set_budget_host(ctx, expert_bytes, cap_out); });
  }
  return set_budget_host(ctx, expert_bytes, cap_out);
}

wisp_status wisp_preload(wisp_ctx* ctx) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (ctx->pager == WISP_PAGER_DEVICE) return with_host_tables(ctx, [&] { return preload_host(ctx); });
  return preload_host(ctx);
}

wisp_status wisp_set_fusion(wisp_ctx* ctx, int32_t on) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  for (auto& L : ctx->layers)
    if (L.pending) return fail(WISP_E_STATE, "a page-in is pending");
  ctx->fusion = on != 0;
  return WISP_OK;
}

wisp_status wisp_set_pager(wisp_ctx* ctx, int32_t pager) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (pager != WISP_PAGER_HOST && pager != WISP_PAGER_DEVICE) return fail(WISP_E_INVAL, "unknown pager");
  if (pager == ctx->pager) return WISP_OK;
  for (auto& L : ctx->layers)
    if (L.pending) return fail(WISP_E_STATE, "a page-in is pending");
  if (pager == WISP_PAGER_DEVICE) {
    const auto& d = ctx->desc;
    if (ctx->cap < 1) return fail(WISP_E_STATE, "no expert budget set");
    if (ctx->pf_mode != WISP_PREFETCH_OFF) return fail(WISP_E_STATE, "prefetch runs with the host pager; turn it off");
    if (d.max_tokens > 4) return fail(WISP_E_INVAL, "the device pager handles max_tokens <= 4");
    if (ctx->pageable) return fail(WISP_E_INVAL, "the device pager reads pinned masters; these are pageable");
    if (ctx->cap < d.max_tokens * d.top_k)
      return fail(WISP_E_INVAL, "the device pager needs C >= max_tokens * k (one Algorithm 1 step per layer-step)");
    if (!ffn_dev_supported(ctx->shape, d.max_tokens, d.top_k, d.has_shared))
      return fail(WISP_E_INVAL, "layer shape not supported by the device-planned FFN kernels");
    if ((s = drain(ctx)) != WISP_OK) return s;
    if ((s = upload_tables(ctx)) != WISP_OK) return s;
    ctx->pager = WISP_PAGER_DEVICE;
  } else {
    if ((s = drain(ctx)) != WISP_OK) return s;
    if ((s = download_tables(ctx)) != WISP_OK) return s;
    ctx->pager = WISP_PAGER_HOST;
  }
  return WISP_OK;
}

namespace {
// The router launches of a layer-step: logits and selection (one launch for T <= 4 with fusion on).
// With idx_tagged, the selection also writes each id to host-coherent memory as a word tagged seq.
wisp_status route_kernels(wisp_ctx* ctx, LayerState& L, const void* x_dev, int32_t T, int32_t* idx_dev, float* w_dev,
                          uint64_t* idx_tagged, uint32_t seq, hipStream_t st) {
  const auto& d = ctx->desc;
  if (ctx->fusion && T <= 4) {
    // logits and selection in one launch (the first workgroup selects once every row is published)
    LaunchTiming t1 = timing_begin(ctx, WISP_K_ROUTER_SELECT);
    WISP_HIP(launch_route_select(L.wr, x_dev, d.x_dtype, d.d_model, ctx->d_logit_tags, next_logit_tag(ctx),
                                 T, d.n_experts,
                                 d.top_k, d.route, d.n_groups, d.topk_groups, idx_dev, w_dev, idx_tagged, seq, st, t1),
             "router logits + select launch");
    timing_end(ctx, t1, WISP_K_ROUTER_SELECT,
               static_cast<uint64_t>(d.n_experts) * d.d_model * 4 + static_cast<uint64_t>(T) * d.d_model * ctx->x_elem());
  } else {
    LaunchTiming t1 = timing_begin(ctx, WISP_K_ROUTER_LOGITS);
    int n_split = 1;
    WISP_HIP(launch_router_logits(L.wr, x_dev, d.x_dtype, T, d.n_experts, d.d_model, ctx->logits, &n_split, st, t1),
             "router logits launch");
    timing_end(ctx, t1, WISP_K_ROUTER_LOGITS,
               static_cast<uint64_t>(d.n_experts) * d.d_model * 4 +
                   static_cast<uint64_t>(T) * d.d_model * ctx->x_elem() + static_cast<uint64_t>(T) * d.n_experts * 4);
    LaunchTiming t2 = timing_begin(ctx, WISP_K_ROUTER_SELECT);
    WISP_HIP(launch_router_select(ctx->logits, n_split, T, d.n_experts, d.top_k, d.route, d.n_groups, d.topk_groups, idx_dev,
                                  w_dev, idx_tagged, seq, st, t2),
             "router select launch");
    timing_end(ctx, t2, WISP_K_ROUTER_SELECT,
               static_cast<uint64_t>(T) * d.n_experts * 4 + static_cast<uint64_t>(T) * d.top_k * 8);
  }
  return WISP_OK;
}
}  // namespace

wisp_status wisp_route_topk(wisp_ctx* ctx, int32_t layer, const void* x_dev, int32_t T, int32_t* idx_dev,
                            float* w_dev, int32_t* idx_host, void* stream) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if ((s = check_layer(ctx, layer)) != WISP_OK) return s;
  if (!x_dev || !idx_dev || !w_dev) return fail(WISP_E_INVAL, "NULL device pointer");
  if (T < 1 || T > ctx->desc.max_tokens) return fail(WISP_E_INVAL, "T out of [1, max_tokens]");
  LayerState& L = ctx->layers[layer];
  if (!L.wr) return fail(WISP_E_STATE, "router weights not set for this layer");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const auto& d = ctx->desc;
  // the ids reach the host through host-coherent memory: the selection writes each one as a 64-bit
  // word tagged with this call's sequence number, so the host needs no copy, event or fence (a copy
  // queue's start latency was ≈10 µs of every token batch's layer-step)
  const bool publish = idx_host != nullptr;
  const uint32_t seq = publish ? ++ctx->route_seq : 0;
  if ((s = route_kernels(ctx, L, x_dev, T, idx_dev, w_dev, publish ? ctx->idx_tagged : nullptr, seq, st)) != WISP_OK)
    return s;
  if (publish) {
    const int n = T * d.top_k;
    // a token batch for the grouped FFN: its pairs are ordered by expert now, from the device ids,
    // while the host waits for the ids and pages the layer in (after the last reader of the order)
    const bool early = T >= kGroupedMinTokens && grouped_supported(ctx->shape, d.has_shared);
    if (early) {
      ctx->perm_layer = -1;
      if (ctx->perm_use_recorded) WISP_HIP(hipStreamWaitEvent(st, ctx->perm_use_ev, 0), "hipStreamWaitEvent(perm use)");
      LaunchTiming tp = timing_begin(ctx, WISP_K_PERMUTE);
      WISP_HIP(launch_permute_pairs(idx_dev, n, d.n_experts, ctx->d_perm, ctx->d_perm_counts, st, tp), "permute launch");
      timing_end(ctx, tp, WISP_K_PERMUTE, static_cast<uint64_t>(n) * 8);
      WISP_HIP(hipEventRecord(ctx->perm_ev, st), "hipEventRecord(perm)");
      ctx->perm_ev_recorded = true;
      ctx->perm_stream = st;
    }
    // spin until every entry carries this call's tag: the wait on the critical path of a layer-step
    uint64_t spins = 0;
    for (int i = 0; i < n; ++i) {
      uint64_t v;
      while (((v = __atomic_load_n(ctx->idx_tagged + i, __ATOMIC_ACQUIRE)) >> 32) != seq) {
        __builtin_ia32_pause();
        if ((++spins & 0xFFFFF) == 0) {
          hipError_t q = hipStreamQuery(st);
          if (q != hipSuccess && q != hipErrorNotReady)
            return fail(WISP_E_HIP, std::string("router stream: ") + hipGetErrorString(q));
          if (q == hipSuccess && (__atomic_load_n(ctx->idx_tagged + i, __ATOMIC_ACQUIRE) >> 32) != seq)
            return fail(WISP_E_HIP, "router finished without publishing its indices");
        }
      }
      idx_host[i] = static_cast<int32_t>(v & 0xFFFFFFFFu);
    }
    if (early) {
      ctx->perm_ids.assign(idx_host, idx_host + n);
      ctx->perm_layer = layer;
      ctx->perm_T = T;
    }
    if (ctx->profiling) harvest(ctx, false);
  }
  return WISP_OK;
}

namespace {
// Algorithm 1 for one layer-step over the n ids (the routed ids, or the distinct experts of a token
// batch whose counts came from the device: the step depends only on the set of ids), then the fills
// of its first chunk.
wisp_status page_in_ids(wisp_ctx* ctx, int32_t layer, const int32_t* ids_host, int32_t n, int32_t T, bool from_counts,
                        wisp_page_stats* st) {
  wisp_status s = WISP_OK;
  LayerState& L = ctx->layers[layer];
  if (!L.pf_unused.empty()) {
    // the prefetch bookkeeping indexes by id: validate first (otherwise the slot table's step validates
    // every id before it changes anything)
    for (int32_t i = 0; i < n; ++i)
      if (ids_host[i] < 0 || ids_host[i] >= ctx->desc.n_experts) return fail(WISP_E_INVAL, "expert id out of range");
    // prefetched experts this page-in routes to while they are still resident
    std::vector<uint8_t>& mk = ctx->pf_mark;
    for (int32_t e : L.pf_unused) mk[e] = 1;
    for (int32_t i = 0; i < n; ++i) {
      const int32_t e = ids_host[i];
      if (mk[e] == 1 && L.table->slot_of(e) >= 0) { ++ctx->pf_useful; mk[e] = 2; }
    }
    for (int32_t e : L.pf_unused) mk[e] = 0;
    L.pf_unused.clear();
  }
  if (!L.table->step(ids_host, n, &L.plan)) return fail(WISP_E_INVAL, "expert id out of range");
  L.ids.assign(ids_host, ids_host + n);
  L.from_counts = from_counts;
  L.T = T;
  const size_t nch = L.plan.chunks.size();
  if ((s = ensure_events(L.fill_ev, 2 * nch)) != WISP_OK) return s;
  if ((s = ensure_events(L.chunk_ev, 2 * nch)) != WISP_OK) return s;
  if (L.late.size() < nch) L.late.resize(nch);
  L.chunk_ptrs.assign(nch, {});
  for (size_t ci = 0; ci < nch; ++ci)
    for (int32_t sl : L.plan.chunks[ci].slots) L.chunk_ptrs[ci].push_back(L.slot_mem[sl]);
  L.pending = true;
  wisp_page_stats ps{};
  ps.hits = L.plan.hits;
  ps.misses = L.plan.misses;
  ps.chunks = static_cast<uint32_t>(nch);
  ps.steps = 1;
  ps.h2d_bytes = static_cast<uint64_t>(L.plan.misses) * ctx->blob.bytes;
  L.cum.hits += ps.hits;
  L.cum.misses += ps.misses;
  L.cum.chunks += ps.chunks;
  L.cum.steps += 1;
  L.cum.h2d_bytes += ps.h2d_bytes;
  if (st) *st = ps;
  if (nch > 0) {
    s = issue_fills(ctx, layer, 0);
    if (s != WISP_OK) return s;
  }
  return WISP_OK;
}

}  // namespace

wisp_status wisp_page_in(wisp_ctx* ctx, int32_t layer, const int32_t* ids_host, int32_t T, wisp_page_stats* st) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if ((s = check_layer(ctx, layer)) != WISP_OK) return s;
  if (!ids_host) return fail(WISP_E_INVAL, "ids_host is NULL");
  if (T < 1 || T > ctx->desc.max_tokens) return fail(WISP_E_INVAL, "T out of [1, max_tokens]");
  if (ctx->cap < 1) return fail(WISP_E_STATE, "no expert budget set");
  if (ctx->pager == WISP_PAGER_DEVICE) return fail(WISP_E_STATE, "the device pager pages inside wisp_decode_step");
  if (ctx->layers[layer].pending) return fail(WISP_E_STATE, "previous page-in of this layer not consumed by wisp_moe_forward");
  return page_in_ids(ctx, layer, ids_host, T * ctx->desc.top_k, T, false, st);
}

wisp_status wisp_moe_forward(wisp_ctx* ctx, int32_t layer, const void* x_dev, int32_t T, const float* w_dev,
                             float* y_dev, void* stream, wisp_page_stats* st) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if ((s = check_layer(ctx, layer)) != WISP_OK) return s;
  if (!x_dev || !w_dev || !y_dev) return fail(WISP_E_INVAL, "NULL device pointer");
  if (ctx->pager == WISP_PAGER_DEVICE) return fail(WISP_E_STATE, "the device pager pages inside wisp_decode_step");
  LayerState& L = ctx->layers[layer];
  if (!L.pending) return fail(WISP_E_STATE, "no pending page-in for this layer");
  if (T != L.T) return fail(WISP_E_INVAL, "T differs from the page-in");
  hipStream_t sm = static_cast<hipStream_t>(stream);
  const int k = ctx->desc.top_k;
  const int N = ctx->desc.n_experts;
  const int rows = k + 1;
  const int32_t n_pairs = T * k;
  const size_t nch = L.plan.chunks.size();
  // pairs per expert, and the pairs in (expert, pair) order
  std::vector<int32_t>& cnt = ctx->e_cnt;
  std::vector<int32_t>& off = ctx->e_off;
  if (L.from_counts) {
    cnt = ctx->batch_cnt;
  } else {
    std::fill(cnt.begin(), cnt.end(), 0);
    for (int32_t p = 0; p < n_pairs; ++p) ++cnt[L.ids[p]];
  }
  off[0] = 0;
  for (int e = 0; e < N; ++e) off[e + 1] = off[e] + cnt[e];
  const bool grouped = T >= kGroupedMinTokens && grouped_supported(ctx->shape, ctx->desc.has_shared);
  if (L.from_counts && (!grouped || ctx->perm_layer != layer || ctx->perm_T != T))
    return fail(WISP_E_STATE, "a page-in from device counts needs its layer's device permutation");
  if (!grouped) {   // the per-item launches list their pairs; the grouped ones read the device order
    std::vector<int32_t> fill(off.begin(), off.end() - 1);
    for (int32_t p = 0; p < n_pairs; ++p) ctx->pair_order[fill[L.ids[p]]++] = p;
  }
  // exactness check: every routed id is in a chunk of the plan, with a slot
  {
    std::vector<uint8_t> planned(N, 0);
    for (size_t ci = 0; ci < nch; ++ci)
      for (int32_t e : L.plan.chunks[ci].experts) planned[e] = 1;
    for (int e = 0; e < N; ++e)
      if (cnt[e] > 0 && !planned[e]) return fail(WISP_E_NOT_RESIDENT, "routed expert missing from the page-in plan");
  }
  if (L.pf_pending) {
    // a routed expert whose prefetch copy may still be in flight: the FFN waits for the copies
    bool need = false;
    for (int32_t e : L.pf_inflight) need = need || cnt[e] > 0;
    if (need) {
      WISP_HIP(hipStreamWaitEvent(sm, L.pf_ev, 0), "hipStreamWaitEvent(prefetch)");
      L.pf_pending = false;
      L.pf_inflight.clear();
    }
  }
  if (grouped) {
    // the permutation wisp_route_topk computed for this layer, if it came from the ids paged in
    // (a page-in from counts: the counts are the permutation's own)
    const bool early = ctx->perm_layer == layer && ctx->perm_T == T &&
                       (L.from_counts ||
                        std::memcmp(ctx->perm_ids.data(), L.ids.data(), sizeof(int32_t) * n_pairs) == 0);
    ctx->perm_layer = -1;   // used once; the launches below overwrite it otherwise
    // (on the permutation's own stream the launches below are ordered after it already)
    if (ctx->perm_ev_recorded && !(early && sm == ctx->perm_stream))
      WISP_HIP(hipStreamWaitEvent(sm, ctx->perm_ev, 0), "hipStreamWaitEvent(perm)");
    if (!early) {
      // the ids go to the device; the permutation kernel orders the pairs by expert there
      if (ctx->ids_ev_recorded) WISP_HIP(hipEventSynchronize(ctx->ids_ev), "hipEventSynchronize(ids)");
      std::memcpy(ctx->ids_up, L.ids.data(), sizeof(int32_t) * n_pairs);
      WISP_HIP(hipMemcpyAsync(ctx->d_ids, ctx->ids_up, sizeof(int32_t) * n_pairs, hipMemcpyHostToDevice, sm),
               "hipMemcpyAsync(ids)");
      WISP_HIP(hipEventRecord(ctx->ids_ev, sm), "hipEventRecord(ids)");
      ctx->ids_ev_recorded = true;
      LaunchTiming tp = timing_begin(ctx, WISP_K_PERMUTE);
      WISP_HIP(launch_permute_pairs(ctx->d_ids, n_pairs, N, ctx->d_perm, ctx->d_perm_counts, sm, tp), "permute launch");
      timing_end(ctx, tp, WISP_K_PERMUTE, static_cast<uint64_t>(n_pairs) * 8);
    }
  }
  const BlobLayout& B = ctx->blob;
  const uint64_t dI = static_cast<uint64_t>(B.d) * B.I;
  // grouped GEMMs over a list of (expert, slot) in launches of up to kMaxGroups experts
  auto run_grouped = [&](const std::vector<std::pair<int32_t, const uint8_t*>>& list) -> wisp_status {
    for (size_t g0 = 0; g0 < list.size(); g0 += kMaxGroups) {
      GroupedBatch gb;
      gb.n_groups = static_cast<int32_t>(std::min<size_t>(kMaxGroups, list.size() - g0));
      int32_t tiles = 0;
      uint64_t nrows = 0;
      for (int g = 0; g < gb.n_groups; ++g) {
        const int32_t e = list[g0 + g].first;
        gb.w[g] = list[g0 + g].second;
        gb.row_off[g] = off[e];
        gb.rows[g] = cnt[e];
        tiles += grouped_row_tiles(cnt[e]);
        gb.tile_end[g] = tiles;
        nrows += static_cast<uint64_t>(cnt[e]);
      }
      for (int g = gb.n_groups; g < kMaxGroups; ++g) {
        gb.w[g] = nullptr;
        gb.row_off[g] = gb.rows[g] = 0;
        gb.tile_end[g] = tiles;
      }
      const uint64_t ng = static_cast<uint64_t>(gb.n_groups);
      LaunchTiming t1 = timing_begin(ctx, WISP_K_GROUPED_GATEUP);
      WISP_HIP(launch_grouped_gateup(gb, ctx->shape, x_dev, T, ctx->d_perm, k, ctx->h, sm, t1), "grouped gate/up launch");
      timing_end(ctx, t1, WISP_K_GROUPED_GATEUP, ng * 2 * dI * B.elem + nrows * (B.d + B.I) * 2,
                 nrows * 2 * 2 * dI);
      LaunchTiming t2 = timing_begin(ctx, WISP_K_GROUPED_DOWN);
      WISP_HIP(launch_grouped_down(gb, ctx->shape, ctx->h, T, ctx->d_perm, k, reinterpret_cast<uint16_t*>(ctx->buf), sm,
                                   t2),
               "grouped down launch");
      timing_end(ctx, t2, WISP_K_GROUPED_DOWN, ng * dI * B.elem + nrows * (B.I * 2 + B.d * 2), nrows * 2 * dI);
    }
    return WISP_OK;
  };
  auto work_of = [&](int32_t e, const uint8_t* w) {
    Work wk;
    wk.w = w;
    for (int32_t q = off[e]; q < off[e + 1]; ++q) {
      const int32_t p = ctx->pair_order[q];
      wk.pairs.push_back({p / k, (p / k) * rows + p % k});
    }
    return wk;
  };
  // one token, one chunk: gate/up of the resident experts (and the shared one), then of the faulted
  // ones after their fills, then one down + combine launch over all of them
  const bool fused = !grouped && ctx->fusion && nch == 1 && T == 1 && down_combine_supported(ctx->shape);
  if (fused) {
    const ChunkPlan& cp = L.plan.chunks[0];
    std::vector<Work> hits, faults;
    FusedT1Items all{};
    for (size_t i = 0; i < cp.experts.size(); ++i) {
      (cp.fault[i] ? faults : hits).push_back(work_of(cp.experts[i], L.chunk_ptrs[0][i]));
      all.w[all.n_items] = L.chunk_ptrs[0][i];
      all.rank[all.n_items] = ctx->pair_order[off[cp.experts[i]]];   // T = 1: the pair index is the rank
      ++all.n_items;
    }
    if (ctx->desc.has_shared) {
      Work wk;
      wk.w = L.shared_dev;
      wk.pairs.push_back({0, k});
      hits.push_back(std::move(wk));
      all.w[all.n_items] = L.shared_dev;
      all.rank[all.n_items] = k;
      ++all.n_items;
    }
    if (!hits.empty() && (s = run_ffn(ctx, hits, x_dev, sm, false)) != WISP_OK) return s;
    if (!faults.empty()) {
      WISP_HIP(hipStreamWaitEvent(sm, L.fill_ev[0], 0), "hipStreamWaitEvent(fill)");
      if ((s = run_ffn(ctx, faults, x_dev, sm, false)) != WISP_OK) return s;
    }
    FfnBatch b;
    b.n_items = all.n_items;
    b.max_ntok = 1;
    for (int i = 0; i < all.n_items; ++i) b.items[i].ntok = 1;
    LaunchTiming td = timing_begin(ctx, WISP_K_DOWN_COMBINE);
    WISP_HIP(launch_down_combine_t1(all, ctx->shape, ctx->h, w_dev, y_dev, k, ctx->desc.has_shared, sm, td),
             "down+combine launch");
    timing_end(ctx, td, WISP_K_DOWN_COMBINE, ffn_bytes(ctx, b, false) + static_cast<uint64_t>(k) * 4);
  }
  for (size_t ci = 0; ci < nch && !fused; ++ci) {
    const ChunkPlan& cp = L.plan.chunks[ci];
    if (ci > 0 && (s = issue_fills(ctx, layer, ci)) != WISP_OK) return s;
    // the hits, then each half of the faults once its fills have landed (issue_fills)
    if (grouped) {
      std::vector<std::pair<int32_t, const uint8_t*>> hits, faults[2];
      for (size_t i = 0; i < cp.experts.size(); ++i)
        (cp.fault[i] ? faults[L.late[ci][i]] : hits).push_back({cp.experts[i], L.chunk_ptrs[ci][i]});
      if (!hits.empty() && (s = run_grouped(hits)) != WISP_OK) return s;
      for (int h = 0; h < 2; ++h) {
        if (!faults[h].empty()) {
          WISP_HIP(hipStreamWaitEvent(sm, L.fill_ev[2 * ci + h], 0), "hipStreamWaitEvent(fill)");
          if ((s = run_grouped(faults[h])) != WISP_OK) return s;
        }
        if (nch > 1) WISP_HIP(hipEventRecord(L.chunk_ev[2 * ci + h], sm), "hipEventRecord(chunk)");
      }
    } else {
      std::vector<Work> hits, faults[2];
      for (size_t i = 0; i < cp.experts.size(); ++i)
        (cp.fault[i] ? faults[L.late[ci][i]] : hits).push_back(work_of(cp.experts[i], L.chunk_ptrs[ci][i]));
      if (ci == 0 && ctx->desc.has_shared) {
        Work wk;
        wk.w = L.shared_dev;
        for (int32_t t = 0; t < T; ++t) wk.pairs.push_back({t, t * rows + k});
        hits.push_back(std::move(wk));
      }
      if (!hits.empty() && (s = run_ffn(ctx, hits, x_dev, sm)) != WISP_OK) return s;
      for (int h = 0; h < 2; ++h) {
        if (!faults[h].empty()) {
          WISP_HIP(hipStreamWaitEvent(sm, L.fill_ev[2 * ci + h], 0), "hipStreamWaitEvent(fill)");
          if ((s = run_ffn(ctx, faults[h], x_dev, sm)) != WISP_OK) return s;
        }
        if (nch > 1) WISP_HIP(hipEventRecord(L.chunk_ev[2 * ci + h], sm), "hipEventRecord(chunk)");
      }
    }
  }
  if (grouped) {   // the grouped GEMMs leave bf16 expert outputs (no shared expert on this path)
    LaunchTiming tc = timing_begin(ctx, WISP_K_COMBINE);
    WISP_HIP(launch_combine_bf16(T, k, ctx->desc.d_model, w_dev, reinterpret_cast<const uint16_t*>(ctx->buf), y_dev, sm,
                                 tc),
             "combine launch");
    timing_end(ctx, tc, WISP_K_COMBINE,
               static_cast<uint64_t>(T) * ctx->desc.d_model * (2 * k + 4) + static_cast<uint64_t>(T) * k * 4);
  } else if (!fused) {
    LaunchTiming tc = timing_begin(ctx, WISP_K_COMBINE);
    WISP_HIP(launch_combine(T, k, ctx->desc.d_model, ctx->desc.has_shared, w_dev, ctx->buf, y_dev, sm, tc),
             "combine launch");
    timing_end(ctx, tc, WISP_K_COMBINE,
               static_cast<uint64_t>(T) * ctx->desc.d_model * 4 * (k + ctx->desc.has_shared + 1) +
                   static_cast<uint64_t>(T) * k * 4);
  }
  WISP_HIP(hipEventRecord(L.use_ev, sm), "hipEventRecord(use)");
  L.use_ev_recorded = true;
  if (grouped) {
    WISP_HIP(hipEventRecord(ctx->perm_use_ev, sm), "hipEventRecord(perm use)");
    ctx->perm_use_recorded = true;
  }
  L.pending = false;
  if (st) {
    st->hits = L.plan.hits;
    st->misses = L.plan.misses;
    st->chunks = static_cast<uint32_t>(nch);
    st->steps = 1;
    st->h2d_bytes = static_cast<uint64_t>(L.plan.misses) * ctx->blob.bytes;
  }
  return WISP_OK;
}

namespace {
// Routing and page-in of a token batch for the grouped FFN with the ids left on the device: the
// permutation kernel, which orders the pairs by expert right after the selection, hands every
// expert's pair count to the host as a word tagged with this call's sequence number (host-coherent
// memory).  The host pages in the experts with pairs (Algorithm 1 depends only on that set) and
// sizes the grouped launches from the counts, so it reads N words instead of T * k ids and does no
// per-pair work.
wisp_status route_page_batch(wisp_ctx* ctx, int32_t layer, const void* x_dev, int32_t T, int32_t* idx_dev,
                             float* w_dev, hipStream_t st, wisp_page_stats* ps) {
  wisp_status s = WISP_OK;
  LayerState& L = ctx->layers[layer];
  if (!L.wr) return fail(WISP_E_STATE, "router weights not set for this layer");
  if (L.pending) return fail(WISP_E_STATE, "previous page-in of this layer not consumed by wisp_moe_forward");
  const auto& d = ctx->desc;
  const int N = d.n_experts, n = T * d.top_k;
  const uint32_t seq = ++ctx->route_seq;
  if ((s = route_kernels(ctx, L, x_dev, T, idx_dev, w_dev, nullptr, 0, st)) != WISP_OK) return s;
  ctx->perm_layer = -1;
  if (ctx->perm_use_recorded) WISP_HIP(hipStreamWaitEvent(st, ctx->perm_use_ev, 0), "hipStreamWaitEvent(perm use)");
  LaunchTiming tp = timing_begin(ctx, WISP_K_PERMUTE);
  WISP_HIP(launch_permute_pairs(idx_dev, n, N, ctx->d_perm, ctx->d_perm_counts, st, tp, ctx->cnt_tagged, seq),
           "permute launch");
  timing_end(ctx, tp, WISP_K_PERMUTE, static_cast<uint64_t>(n) * 8);
  WISP_HIP(hipEventRecord(ctx->perm_ev, st), "hipEventRecord(perm)");
  ctx->perm_ev_recorded = true;
  ctx->perm_stream = st;
  // spin until every count carries this call's tag
  std::vector<int32_t>& R = ctx->batch_set;
  R.clear();
  uint64_t spins = 0;
  int32_t total = 0;
  for (int e = 0; e < N; ++e) {
    uint64_t v;
    while (((v = __atomic_load_n(ctx->cnt_tagged + e, __ATOMIC_ACQUIRE)) >> 32) != seq) {
      __builtin_ia32_pause();
      if ((++spins & 0xFFFFF) == 0) {
        hipError_t q = hipStreamQuery(st);
        if (q != hipSuccess && q != hipErrorNotReady)
          return fail(WISP_E_HIP, std::string("router stream: ") + hipGetErrorString(q));
        if (q == hipSuccess && (__atomic_load_n(ctx->cnt_tagged + e, __ATOMIC_ACQUIRE) >> 32) != seq)
          return fail(WISP_E_HIP, "permutation finished without publishing its counts");
      }
    }
    const int32_t c = static_cast<int32_t>(v & 0xFFFFFFFFu);
    ctx->batch_cnt[e] = c;
    total += c;
    if (c > 0) R.push_back(e);
  }
  if (total != n) return fail(WISP_E_HIP, "expert counts do not add up to the routed pairs");
  ctx->perm_layer = layer;
  ctx->perm_T = T;
  if (ctx->profiling) harvest(ctx, false);
  return page_in_ids(ctx, layer, R.data(), static_cast<int32_t>(R.size()), T, true, ps);
}
}  // namespace

wisp_status wisp_decode_step(wisp_ctx* ctx, const void* x_dev, int32_t T, int32_t* idx_dev, float* w_dev,
                             float* y_dev, void* stream, wisp_page_stats* st) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (!x_dev || !idx_dev || !w_dev || !y_dev) return fail(WISP_E_INVAL, "NULL device pointer");
  if (T < 1 || T > ctx->desc.max_tokens) return fail(WISP_E_INVAL, "T out of [1, max_tokens]");
  const auto& d = ctx->desc;
  const size_t xs = static_cast<size_t>(T) * d.d_model * ctx->x_elem();
  if (ctx->pager == WISP_PAGER_DEVICE) {
    hipStream_t sm = static_cast<hipStream_t>(stream);
    const int max_items = T * d.top_k + d.has_shared;
    const int C = ctx->cap;
    const bool dc = ctx->fusion && T == 1 && down_combine_supported(ctx->shape);
    for (int32_t l = 0; l < d.n_layers; ++l) {
      LayerState& L = ctx->layers[l];
      if (!L.wr) return fail(WISP_E_STATE, "router weights not set for this layer");
      const void* xl = static_cast<const uint8_t*>(x_dev) + l * xs;
      int32_t* il = idx_dev + static_cast<size_t>(l) * T * d.top_k;
      float* wl = w_dev + static_cast<size_t>(l) * T * d.top_k;
      float* yl = y_dev + static_cast<size_t>(l) * T * d.d_model;
      int32_t* pi_l = ctx->d_pi + static_cast<size_t>(l) * d.n_experts;
      int32_t* pinv_l = ctx->d_pinv + static_cast<size_t>(l) * C;
      uint64_t* tau_l = ctx->d_tau + static_cast<size_t>(l) * C;
      const uint64_t* slot_l = ctx->d_slot_ptr + static_cast<size_t>(l) * C;
      if (ctx->fusion) {
        LaunchTiming t1 = timing_begin(ctx, WISP_K_ROUTER_SELECT);
        WISP_HIP(launch_route_page(L.wr, xl, d.x_dtype, d.d_model, ctx->d_logit_tags, next_logit_tag(ctx),
                                   T, d.n_experts, d.top_k,
                                   d.route, d.n_groups, d.topk_groups, il, wl, pi_l, pinv_l, tau_l, ctx->d_clock + l, C,
                                   slot_l, ctx->masters[l], ctx->master_stride, L.shared_dev, d.has_shared,
                                   ctx->d_plan, ctx->d_stats + 2 * l, sm, t1),
                 "device route + pager launch");
        timing_end(ctx, t1, WISP_K_ROUTER_SELECT, static_cast<uint64_t>(d.n_experts) * d.d_model * 4);
      } else {
        LaunchTiming t1 = timing_begin(ctx, WISP_K_ROUTER_LOGITS);
        int n_split = 1;   // decode sizes: one slice (the device pager's selection reads plain logits)
        WISP_HIP(launch_router_logits(L.wr, xl, d.x_dtype, T, d.n_experts, d.d_model, ctx->logits, &n_split, sm, t1),
                 "router logits launch");
        timing_end(ctx, t1, WISP_K_ROUTER_LOGITS, static_cast<uint64_t>(d.n_experts) * d.d_model * 4);
        LaunchTiming t2 = timing_begin(ctx, WISP_K_ROUTER_SELECT);
        WISP_HIP(launch_select_page(ctx->logits, T, d.n_experts, d.top_k, d.route, d.n_groups, d.topk_groups, il, wl,
                                    pi_l, pinv_l, tau_l, ctx->d_clock + l, C, slot_l, ctx->masters[l],
                                    ctx->master_stride, L.shared_dev, d.has_shared, ctx->d_plan, ctx->d_stats + 2 * l,
                                    sm, t2),
                 "device pager launch");
        timing_end(ctx, t2, WISP_K_ROUTER_SELECT, 0);
      }
      LaunchTiming t3 = timing_begin(ctx, WISP_K_FFN_GATEUP);
      LaunchTiming t4 = dc ? LaunchTiming{} : timing_begin(ctx, WISP_K_FFN_DOWN);
      WISP_HIP(launch_ffn_dev(ctx->d_plan, max_items, ctx->shape, xl, ctx->h, ctx->buf, !dc, sm, t3, t4),
               "device-planned FFN launch");
      timing_end(ctx, t3, WISP_K_FFN_GATEUP, 0);
      if (!dc) timing_end(ctx, t4, WISP_K_FFN_DOWN, 0);
      if (dc) {
        LaunchTiming t5 = timing_begin(ctx, WISP_K_DOWN_COMBINE);
        WISP_HIP(launch_down_combine_dev(ctx->d_plan, max_items, ctx->shape, ctx->h, wl, yl, d.top_k, d.has_shared, sm,
                                         t5),
                 "device-planned down+combine launch");
        timing_end(ctx, t5, WISP_K_DOWN_COMBINE, 0);
      } else {
        LaunchTiming t5 = timing_begin(ctx, WISP_K_COMBINE);
        WISP_HIP(launch_combine(T, d.top_k, d.d_model, d.has_shared, wl, ctx->buf, yl, sm, t5), "combine launch");
        timing_end(ctx, t5, WISP_K_COMBINE, 0);
      }
    }
    WISP_HIP(hipMemcpyAsync(ctx->h_stats, ctx->d_stats, sizeof(uint32_t) * 2 * d.n_layers, hipMemcpyDeviceToHost, sm),
             "stats copy");
    WISP_HIP(hipStreamSynchronize(sm), "hipStreamSynchronize");
    if (ctx->profiling) harvest(ctx, false);
    for (int32_t l = 0; l < d.n_layers; ++l) {
      wisp_page_stats ps{};
      ps.hits = ctx->h_stats[2 * l];
      ps.misses = ctx->h_stats[2 * l + 1];
      ps.chunks = (ps.hits + ps.misses) > 0 ? 1 : 0;
      ps.steps = 1;
      ps.h2d_bytes = static_cast<uint64_t>(ps.misses) * ctx->blob.bytes;
      LayerState& L = ctx->layers[l];
      L.cum.hits += ps.hits;
      L.cum.misses += ps.misses;
      L.cum.chunks += ps.chunks;
      L.cum.steps += 1;
      L.cum.h2d_bytes += ps.h2d_bytes;
      if (st) st[l] = ps;
    }
    return WISP_OK;
  }
  // a token batch for the grouped FFN pages in from the device's per-expert counts (no prefetch
  // bookkeeping needs its ids)
  const bool batch_counts = T >= kGroupedMinTokens && grouped_supported(ctx->shape, d.has_shared) &&
                            ctx->pf_mode == WISP_PREFETCH_OFF && ctx->cap >= 1;
  for (int32_t l = 0; l < d.n_layers; ++l) {
    const void* xl = static_cast<const uint8_t*>(x_dev) + l * xs;
    int32_t* il = idx_dev + static_cast<size_t>(l) * T * d.top_k;
    float* wl = w_dev + static_cast<size_t>(l) * T * d.top_k;
    float* yl = y_dev + static_cast<size_t>(l) * T * d.d_model;
    if ((s = prefetch_before_route(ctx, l)) != WISP_OK) return s;
    if (batch_counts) {
      if ((s = check_layer(ctx, l)) != WISP_OK) return s;
      if ((s = route_page_batch(ctx, l, xl, T, il, wl, static_cast<hipStream_t>(stream), st ? st + l : nullptr)) !=
          WISP_OK)
        return s;
      if ((s = wisp_moe_forward(ctx, l, xl, T, wl, yl, stream, nullptr)) != WISP_OK) return s;
      continue;
    }
    if ((s = wisp_route_topk(ctx, l, xl, T, il, wl, ctx->ids_scratch.data(), stream)) != WISP_OK) return s;
    if (ctx->pf_mode == WISP_PREFETCH_PREDICTOR &&
        (s = wisp_predictor_observe(ctx->pf_pred, l, ctx->ids_scratch.data(), T * d.top_k)) != WISP_OK)
      return s;
    if ((s = wisp_page_in(ctx, l, ctx->ids_scratch.data(), T, st ? st + l : nullptr)) != WISP_OK) return s;
    if ((s = wisp_moe_forward(ctx, l, xl, T, wl, yl, stream, nullptr)) != WISP_OK) return s;
  }
  if (ctx->pf_mode == WISP_PREFETCH_PREDICTOR && (s = wisp_predictor_end_pass(ctx->pf_pred)) != WISP_OK) return s;
  if (ctx->pf_mode == WISP_PREFETCH_HINTS) ctx->pf_hint_n = 0;
  return WISP_OK;
}

// ------------------------------------------------------------------------------------------
// Speculative prefetch (the experiment of Sec. 4 with the predictor of App. E)
// ------------------------------------------------------------------------------------------
wisp_status wisp_prefetch(wisp_ctx* ctx, int32_t layer, const int32_t* ids, int32_t n) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if ((s = check_layer(ctx, layer)) != WISP_OK) return s;
  if (n < 0 || (n > 0 && !ids)) return fail(WISP_E_INVAL, "bad id list");
  if (ctx->cap < 1) return fail(WISP_E_STATE, "no expert budget set");
  if (ctx->pager != WISP_PAGER_HOST) return fail(WISP_E_STATE, "prefetch runs with the host pager");
  if (ctx->off.on) return fail(WISP_E_STATE, "static offload is active");
  if (ctx->layers[layer].pending) return fail(WISP_E_STATE, "a page-in of this layer is pending");
  for (int32_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= ctx->desc.n_experts) return fail(WISP_E_INVAL, "expert id out of range");
  return prefetch_layer(ctx, layer, ids, n);
}

wisp_status wisp_set_prefetch(wisp_ctx* ctx, int32_t mode, wisp_predictor* predictor, int32_t depth) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (mode != WISP_PREFETCH_OFF && mode != WISP_PREFETCH_PREDICTOR && mode != WISP_PREFETCH_HINTS)
    return fail(WISP_E_INVAL, "unknown prefetch mode");
  if (mode != WISP_PREFETCH_OFF && ctx->pager != WISP_PAGER_HOST)
    return fail(WISP_E_STATE, "prefetch runs with the host pager");
  if (mode == WISP_PREFETCH_PREDICTOR) {
    if (!predictor) return fail(WISP_E_INVAL, "predictor is NULL");
    int32_t L = 0, N = 0;
    if ((s = wisp_predictor_shape(predictor, &L, &N)) != WISP_OK) return s;
    if (L != ctx->desc.n_layers || N != ctx->desc.n_experts)
      return fail(WISP_E_INVAL, "predictor shape differs from the model");
    if (depth < 1 || depth > ctx->desc.n_experts) return fail(WISP_E_INVAL, "depth out of [1, N]");
  }
  ctx->pf_mode = mode;
  ctx->pf_pred = mode == WISP_PREFETCH_PREDICTOR ? predictor : nullptr;
  ctx->pf_depth = mode == WISP_PREFETCH_PREDICTOR ? depth : 0;
  ctx->pf_hint_n = 0;
  return WISP_OK;
}

wisp_status wisp_set_prefetch_hints(wisp_ctx* ctx, const int32_t* ids, int32_t n) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (ctx->pf_mode != WISP_PREFETCH_HINTS) return fail(WISP_E_STATE, "prefetch mode is not HINTS");
  if (n < 0 || n > ctx->desc.n_experts || (n > 0 && !ids)) return fail(WISP_E_INVAL, "bad hint list");
  const size_t tot = static_cast<size_t>(ctx->desc.n_layers) * n;
  for (size_t i = 0; i < tot; ++i)
    if (ids[i] < -1 || ids[i] >= ctx->desc.n_experts) return fail(WISP_E_INVAL, "hint id out of range");
  ctx->pf_hints.assign(ids, ids + tot);
  ctx->pf_hint_n = n;
  return WISP_OK;
}

wisp_status wisp_prefetch_requests(wisp_ctx* ctx, int32_t layer, int32_t* ids_out, int32_t cap, int32_t* n_out) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if ((s = check_layer(ctx, layer)) != WISP_OK) return s;
  if (!n_out || cap < 0 || (cap > 0 && !ids_out)) return fail(WISP_E_INVAL, "bad output buffer");
  const std::vector<int32_t>& r = ctx->layers[layer].pf_req;
  if (static_cast<size_t>(cap) < r.size()) return fail(WISP_E_INVAL, "output buffer too small");
  std::copy(r.begin(), r.end(), ids_out);
  *n_out = static_cast<int32_t>(r.size());
  return WISP_OK;
}

wisp_status wisp_prefetch_stats(wisp_ctx* ctx, uint64_t* issued, uint64_t* useful) {
  if (!ctx || !issued || !useful) return fail(WISP_E_INVAL, "NULL argument");
  *issued = ctx->pf_issued;
  *useful = ctx->pf_useful;
  return WISP_OK;
}

// ------------------------------------------------------------------------------------------
// Routing-blind static offload at a VRAM expert budget (the comparison arm of Sec. 5.2)
// ------------------------------------------------------------------------------------------
namespace {

// Streamed layers are R .. L-1, visited in order every step; sequence number q (counting across
// steps) is layer R + q % S and uses staging buffer q % 2.
wisp_status offload_issue_copy(wisp_ctx* c) {
  auto& o = c->off;
  const int32_t L = c->desc.n_layers, S = L - o.resident_layers;
  const int32_t q = o.next_copy++;
  const int b = q & 1;
  const int32_t layer = o.resident_layers + q % S;
  if (o.used_rec[b]) WISP_HIP(hipStreamWaitEvent(c->side, o.used[b], 0), "hipStreamWaitEvent(staging use)");
  wisp_status s = master_h2d(c, o.staging[b], c->masters[layer], c->master_map_bytes, c->side);
  if (s != WISP_OK) return s;
  WISP_HIP(hipEventRecord(o.filled[b], c->side), "hipEventRecord(staging fill)");
  return WISP_OK;
}

}  // namespace

wisp_status wisp_offload_begin(wisp_ctx* ctx, uint64_t expert_bytes, int32_t mode, int32_t* resident_layers_out) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (ctx->off.on) return fail(WISP_E_STATE, "static offload already active");
  if (mode != WISP_OFFLOAD_BULK && mode != WISP_OFFLOAD_ZERO_COPY) return fail(WISP_E_INVAL, "unknown offload mode");
  if (mode == WISP_OFFLOAD_ZERO_COPY && ctx->pageable)
    return fail(WISP_E_INVAL, "zero-copy offload reads pinned masters; these are pageable");
  if (ctx->pager == WISP_PAGER_DEVICE) return fail(WISP_E_STATE, "switch to the host pager first");
  for (auto& L : ctx->layers) {
    if (L.pending) return fail(WISP_E_STATE, "a page-in is pending");
    if (!L.wr) return fail(WISP_E_STATE, "router weights not set for every layer");
  }
  const uint64_t layer_bytes = static_cast<uint64_t>(ctx->master_map_bytes);
  const int32_t L = ctx->desc.n_layers;
  int32_t R = 0, staging = 0;
  if (expert_bytes >= layer_bytes * static_cast<uint64_t>(L)) {
    R = L;                                              // everything fits: no streaming
  } else if (mode == WISP_OFFLOAD_ZERO_COPY) {
    R = static_cast<int32_t>(expert_bytes / layer_bytes);   // no staging: the kernels read host memory
  } else if (expert_bytes >= 2 * layer_bytes) {
    R = static_cast<int32_t>((expert_bytes - 2 * layer_bytes) / layer_bytes);
    staging = 2;
  } else {
    return fail(WISP_E_INVAL, "static offload needs a budget of at least two layers of experts");
  }
  if ((s = drain(ctx)) != WISP_OK) return s;
  auto& o = ctx->off;
  auto bail = [&](wisp_status st, const char* m) {
    free_offload(ctx);
    return fail(st, m);
  };
  if (R > 0 && hipMalloc(&o.resident, layer_bytes * R) != hipSuccess) {
    (void)hipGetLastError();
    return bail(WISP_E_NOMEM, "hipMalloc of the resident layers failed");
  }
  for (int b = 0; b < staging; ++b) {
    void* p = nullptr;
    if (hipMalloc(&p, layer_bytes) != hipSuccess) {
      (void)hipGetLastError();
      return bail(WISP_E_NOMEM, "hipMalloc of a staging buffer failed");
    }
    o.staging[b] = static_cast<uint8_t*>(p);
    if (hipEventCreateWithFlags(&o.filled[b], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&o.used[b], hipEventDisableTiming) != hipSuccess)
      return bail(WISP_E_HIP, "hipEventCreate failed");
  }
  o.resident_layers = R;
  o.mode = mode;
  for (int32_t l = 0; l < R; ++l)
    if ((s = master_h2d(ctx, o.resident + layer_bytes * l, ctx->masters[l], layer_bytes, ctx->side)) != WISP_OK)
      return bail(s, "copying a resident layer failed");
  o.on = true;
  // two copies in flight from the start (with one streamed layer both are that layer)
  for (int i = 0; i < 2 && R < L && mode == WISP_OFFLOAD_BULK; ++i)
    if ((s = offload_issue_copy(ctx)) != WISP_OK) return s;
  WISP_HIP(hipStreamSynchronize(ctx->side), "hipStreamSynchronize(side)");
  if (resident_layers_out) *resident_layers_out = R;
  return WISP_OK;
}

wisp_status wisp_offload_step(wisp_ctx* ctx, const void* x_dev, int32_t T, int32_t* idx_dev, float* w_dev,
                              float* y_dev, void* stream) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  auto& o = ctx->off;
  if (!o.on) return fail(WISP_E_STATE, "static offload not active");
  if (!x_dev || !idx_dev || !w_dev || !y_dev) return fail(WISP_E_INVAL, "NULL device pointer");
  if (T < 1 || T > ctx->desc.max_tokens) return fail(WISP_E_INVAL, "T out of [1, max_tokens]");
  const auto& d = ctx->desc;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  const size_t xs = static_cast<size_t>(T) * d.d_model * ctx->x_elem();
  const int k = d.top_k, rows = k + 1;
  const int32_t S = d.n_layers - o.resident_layers;
  for (int32_t l = 0; l < d.n_layers; ++l) {
    const void* xl = static_cast<const uint8_t*>(x_dev) + l * xs;
    int32_t* il = idx_dev + static_cast<size_t>(l) * T * k;
    float* wl = w_dev + static_cast<size_t>(l) * T * k;
    float* yl = y_dev + static_cast<size_t>(l) * T * d.d_model;
    int32_t* ids = ctx->ids_scratch.data();
    if ((s = wisp_route_topk(ctx, l, xl, T, il, wl, ids, stream)) != WISP_OK) return s;
    const uint8_t* base;
    int b = -1;
    if (l < o.resident_layers) {
      base = o.resident + ctx->master_map_bytes * static_cast<size_t>(l);
    } else if (o.mode == WISP_OFFLOAD_ZERO_COPY) {
      base = ctx->masters[l];          // the expert kernels read the routed experts over the host link
    } else {
      const int32_t q = o.next_use++;
      b = q & 1;
      if (o.resident_layers + q % S != l) return fail(WISP_E_STATE, "static offload out of step");
      base = o.staging[b];
      WISP_HIP(hipStreamWaitEvent(sm, o.filled[b], 0), "hipStreamWaitEvent(staging fill)");
    }
    // the routed experts of the layer, ascending, each with its (token, rank) pairs
    std::vector<Work> work;
    for (int e = 0; e < d.n_experts; ++e) {
      Work wk;
      for (int32_t t = 0; t < T; ++t)
        for (int j = 0; j < k; ++j)
          if (ids[t * k + j] == e) wk.pairs.push_back({t, t * rows + j});
      if (wk.pairs.empty()) continue;
      wk.w = base + static_cast<size_t>(e) * ctx->master_stride;
      work.push_back(std::move(wk));
    }
    if (d.has_shared) {
      Work wk;
      wk.w = ctx->layers[l].shared_dev;
      for (int32_t t = 0; t < T; ++t) wk.pairs.push_back({t, t * rows + k});
      work.push_back(std::move(wk));
    }
    if ((s = run_ffn(ctx, work, xl, sm)) != WISP_OK) return s;
    LaunchTiming tc = timing_begin(ctx, WISP_K_COMBINE);
    WISP_HIP(launch_combine(T, k, d.d_model, d.has_shared, wl, ctx->buf, yl, sm, tc), "combine launch");
    timing_end(ctx, tc, WISP_K_COMBINE, 0);
    if (b >= 0) {
      WISP_HIP(hipEventRecord(o.used[b], sm), "hipEventRecord(staging use)");
      o.used_rec[b] = true;
      if ((s = offload_issue_copy(ctx)) != WISP_OK) return s;   // two streamed layers ahead, same buffer
    }
  }
  return WISP_OK;
}

wisp_status wisp_offload_end(wisp_ctx* ctx) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (!ctx->off.on) return fail(WISP_E_STATE, "static offload not active");
  free_offload(ctx);
  return WISP_OK;
}

wisp_status wisp_get_desc(wisp_ctx* ctx, wisp_model_desc* desc) {
  if (!ctx || !desc) return fail(WISP_E_INVAL, "NULL argument");
  *desc = ctx->desc;
  return WISP_OK;
}

wisp_status wisp_get_stats(wisp_ctx* ctx, int32_t layer, wisp_page_stats* cumulative) {
  if (!ctx || !cumulative) return fail(WISP_E_INVAL, "NULL argument");
  wisp_status s = check_layer(ctx, layer);
  if (s != WISP_OK) return s;
  *cumulative = ctx->layers[layer].cum;
  return WISP_OK;
}

wisp_status wisp_reset_stats(wisp_ctx* ctx) {
  if (!ctx) return fail(WISP_E_INVAL, "ctx is NULL");
  for (auto& L : ctx->layers) L.cum = wisp_page_stats{};
  ctx->pf_issued = ctx->pf_useful = 0;
  return WISP_OK;
}

wisp_status wisp_get_cap(wisp_ctx* ctx, int32_t* cap) {
  if (!ctx || !cap) return fail(WISP_E_INVAL, "NULL argument");
  *cap = ctx->cap;
  return WISP_OK;
}

wisp_status wisp_slot_of(wisp_ctx* ctx, int32_t layer, int32_t expert, int32_t* slot) {
  if (!ctx || !slot) return fail(WISP_E_INVAL, "NULL argument");
  wisp_status s = check_layer(ctx, layer);
  if (s != WISP_OK) return s;
  if (expert < 0 || expert >= ctx->desc.n_experts) return fail(WISP_E_INVAL, "expert out of range");
  if (ctx->pager == WISP_PAGER_DEVICE) {
    if ((s = check_ctx(ctx)) != WISP_OK || (s = drain(ctx)) != WISP_OK || (s = download_tables(ctx)) != WISP_OK) return s;
  }
  const auto& t = ctx->layers[layer].table;
  *slot = t ? t->slot_of(expert) : -1;
  return WISP_OK;
}

wisp_status wisp_expert_in_slot(wisp_ctx* ctx, int32_t layer, int32_t slot, int32_t* expert) {
  if (!ctx || !expert) return fail(WISP_E_INVAL, "NULL argument");
  wisp_status s = check_layer(ctx, layer);
  if (s != WISP_OK) return s;
  if (slot < 0 || slot >= ctx->cap) return fail(WISP_E_INVAL, "slot out of range");
  if (ctx->pager == WISP_PAGER_DEVICE) {
    if ((s = check_ctx(ctx)) != WISP_OK || (s = drain(ctx)) != WISP_OK || (s = download_tables(ctx)) != WISP_OK) return s;
  }
  *expert = ctx->layers[layer].table->expert_in(slot);
  return WISP_OK;
}

wisp_status wisp_read_slot(wisp_ctx* ctx, int32_t layer, int32_t slot, void* dst) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if ((s = check_layer(ctx, layer)) != WISP_OK) return s;
  if (!dst) return fail(WISP_E_INVAL, "dst is NULL");
  if (slot < 0 || slot >= ctx->cap) return fail(WISP_E_INVAL, "slot out of range");
  if ((s = drain(ctx)) != WISP_OK) return s;
  WISP_HIP(hipMemcpy(dst, ctx->layers[layer].slot_mem[slot], ctx->blob.bytes, hipMemcpyDeviceToHost),
           "hipMemcpy(read slot)");
  return WISP_OK;
}

wisp_status wisp_set_profiling(wisp_ctx* ctx, int32_t class_mask) {
  if (!ctx) return fail(WISP_E_INVAL, "ctx is NULL");
  if (!class_mask) harvest(ctx, true);
  ctx->profiling = class_mask != 0;
  ctx->profile_mask = class_mask;
  return WISP_OK;
}

wisp_status wisp_kernel_times(wisp_ctx* ctx, int32_t kclass, double* total_ms, uint64_t* launches, uint64_t* bytes,
                              uint64_t* flops) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (kclass < 0 || kclass >= WISP_K_NUM) return fail(WISP_E_INVAL, "kernel class out of range");
  harvest(ctx, true);
  if (total_ms) *total_ms = ctx->k_ms[kclass];
  if (launches) *launches = ctx->k_n[kclass];
  if (bytes) *bytes = ctx->k_bytes[kclass];
  if (flops) *flops = ctx->k_flops[kclass];
  return WISP_OK;
}

wisp_status wisp_reset_kernel_times(wisp_ctx* ctx) {
  if (!ctx) return fail(WISP_E_INVAL, "ctx is NULL");
  harvest(ctx, true);
  for (int i = 0; i < WISP_K_NUM; ++i) { ctx->k_ms[i] = 0; ctx->k_n[i] = 0; ctx->k_bytes[i] = 0; ctx->k_flops[i] = 0; }
  return WISP_OK;
}

wisp_status wisp_probe_h2d(wisp_ctx* ctx, int32_t count, int32_t reps, double* gbps) {
  return wisp_probe_h2d_engine(ctx, count, reps, WISP_LINK_COPY_ENGINE, gbps);
}

wisp_status wisp_probe_h2d_engine(wisp_ctx* ctx, int32_t count, int32_t reps, int32_t engine, double* gbps) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  if (count < 1 || reps < 1 || !gbps) return fail(WISP_E_INVAL, "count, reps >= 1 and gbps required");
  if (engine != WISP_LINK_COPY_ENGINE && engine != WISP_LINK_CUS) return fail(WISP_E_INVAL, "unknown engine");
  if (engine == WISP_LINK_CUS && ctx->pageable)
    return fail(WISP_E_INVAL, "compute-unit fills read pinned masters; these are pageable");
  if ((s = drain(ctx)) != WISP_OK) return s;
  void* scratch = nullptr;
  const size_t B = ctx->blob.bytes;
  if (hipMalloc(&scratch, B * count) != hipSuccess) {
    (void)hipGetLastError();
    return fail(WISP_E_NOMEM, "probe scratch allocation failed");
  }
  hipEvent_t a = nullptr, b = nullptr;
  std::vector<double> rates;
  hipError_t e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  const int nl = ctx->desc.n_layers, ne = ctx->desc.n_experts;
  int src = 0;
  for (int r = 0; r < reps && e == hipSuccess; ++r) {
    e = hipEventRecord(a, ctx->side);
    if (engine == WISP_LINK_CUS) {
      FillList fl;
      fl.n = 0;
      for (int i = 0; i < count && e == hipSuccess; ++i, ++src) {
        const int l = (src / ne) % nl, x = src % ne;
        fl.src[fl.n] = ctx->master(l, x);
        fl.dst[fl.n] = static_cast<uint8_t*>(scratch) + static_cast<size_t>(i) * B;
        if (++fl.n == 32 || i + 1 == count) {
          e = launch_fill(fl, B, ctx->side, LaunchTiming{});
          fl.n = 0;
        }
      }
    }
    for (int i = 0; i < count && e == hipSuccess && engine == WISP_LINK_COPY_ENGINE; ++i, ++src) {
      const int l = (src / ne) % nl, x = src % ne;
      if (!ctx->pageable)
        e = hipMemcpyAsync(static_cast<uint8_t*>(scratch) + static_cast<size_t>(i) * B, ctx->master(l, x), B,
                           hipMemcpyHostToDevice, ctx->side);
      else
        e = ctx->bounce->copy_to_device(static_cast<uint8_t*>(scratch) + static_cast<size_t>(i) * B,
                                        ctx->master(l, x), B, ctx->side);
    }
    if (e == hipSuccess) e = hipEventRecord(b, ctx->side);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
    if (e == hipSuccess) rates.push_back(static_cast<double>(B) * count / (ms * 1e-3) / 1e9);
  }
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  (void)hipFree(scratch);
  if (e != hipSuccess) return fail(WISP_E_HIP, std::string("probe: ") + hipGetErrorString(e));
  std::sort(rates.begin(), rates.end());
  *gbps = rates[rates.size() / 2];
  return WISP_OK;
}

wisp_status wisp_hbm_copy(const void* src, void* dst, uint64_t bytes, void* stream) {
  if (!src || !dst) return fail(WISP_E_INVAL, "NULL pointer");
  if (bytes % 16 || reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16)
    return fail(WISP_E_INVAL, "bytes and pointers must be 16-byte aligned");
  WISP_HIP(launch_hbm_copy(src, dst, bytes, static_cast<hipStream_t>(stream)), "copy launch");
  return WISP_OK;
}

wisp_status wisp_probe_hbm_read(uint64_t bytes, int32_t launches, double* us_per_launch) {
  if (bytes < 16 || bytes % 16 || bytes > (1ull << 32) || launches < 1 || !us_per_launch)
    return fail(WISP_E_INVAL, "bytes in [16, 4 GiB] and a multiple of 16, launches >= 1, result pointer required");
  // enough windows that a launch never reads what the last-level cache (256 MB) still holds
  const uint64_t nwin = std::max<uint64_t>(4, ((2ull << 30) + bytes - 1) / bytes);
  void* buf = nullptr;
  uint32_t* sink = nullptr;
  if (hipMalloc(&buf, nwin * bytes) != hipSuccess || hipMalloc(reinterpret_cast<void**>(&sink), 256) != hipSuccess) {
    (void)hipGetLastError();
    if (buf) (void)hipFree(buf);
    return fail(WISP_E_NOMEM, "read probe allocation failed");
  }
  hipStream_t st = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  if (e == hipSuccess) e = hipMemsetAsync(buf, 0, nwin * bytes, st);
  const uint8_t* base = static_cast<const uint8_t*>(buf);
  uint64_t w = 0;
  for (int i = 0; i < 8 && e == hipSuccess; ++i, ++w) e = launch_hbm_read(base + (w % nwin) * bytes, bytes, sink, st);
  if (e == hipSuccess) e = hipEventRecord(a, st);
  for (int i = 0; i < launches && e == hipSuccess; ++i, ++w)
    e = launch_hbm_read(base + (w % nwin) * bytes, bytes, sink, st);
  if (e == hipSuccess) e = hipEventRecord(b, st);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  if (st) (void)hipStreamSynchronize(st);
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (st) (void)hipStreamDestroy(st);
  (void)hipFree(sink);
  (void)hipFree(buf);
  if (e != hipSuccess) return fail(WISP_E_HIP, std::string("read probe: ") + hipGetErrorString(e));
  *us_per_launch = static_cast<double>(ms) * 1e3 / launches;
  return WISP_OK;
}

wisp_status wisp_probe_mfma(int32_t launches, double* tflops) {
  if (launches < 1 || !tflops) return fail(WISP_E_INVAL, "launches >= 1 and a result pointer required");
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return fail(WISP_E_HIP, "device attributes");
  const int wgs = cus * 8, iters = 2048;   // eight waves per SIMD, ≈1 ms per launch
  float* sink = nullptr;
  if (hipMalloc(reinterpret_cast<void**>(&sink), 256) != hipSuccess) {
    (void)hipGetLastError();
    return fail(WISP_E_NOMEM, "probe sink allocation failed");
  }
  hipStream_t st = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  for (int i = 0; i < 2 && e == hipSuccess; ++i) e = launch_mfma_peak(wgs, iters, sink, st);
  if (e == hipSuccess) e = hipEventRecord(a, st);
  for (int i = 0; i < launches && e == hipSuccess; ++i) e = launch_mfma_peak(wgs, iters, sink, st);
  if (e == hipSuccess) e = hipEventRecord(b, st);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  if (st) (void)hipStreamSynchronize(st);
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (st) (void)hipStreamDestroy(st);
  (void)hipFree(sink);
  if (e != hipSuccess) return fail(WISP_E_HIP, std::string("matrix-core probe: ") + hipGetErrorString(e));
  const double flops = static_cast<double>(launches) * wgs * 4 /* waves */ * iters * 4 /* chains */ * 2.0 * 32 * 32 * 16;
  *tflops = flops / (static_cast<double>(ms) * 1e-3) / 1e12;
  return WISP_OK;
}

wisp_status wisp_decode_fp8(const uint8_t* codes_dev, float* out_dev, int32_t n, void* stream) {
  if (!codes_dev || !out_dev || n < 0) return fail(WISP_E_INVAL, "bad argument");
  WISP_HIP(launch_decode_fp8(codes_dev, out_dev, n, static_cast<hipStream_t>(stream)), "decode launch");
  return WISP_OK;
}

wisp_status wisp_debug_poison_victims(wisp_ctx* ctx, int32_t on) {
  wisp_status s = check_ctx(ctx);
  if (s != WISP_OK) return s;
  ctx->poison = on != 0;
  return WISP_OK;
}

wisp_status wisp_debug_fail_slot_alloc(wisp_ctx* ctx, int32_t n) {
  if (!ctx || n < 0) return fail(WISP_E_INVAL, "bad argument");
  ctx->fail_alloc_at = n > 0 ? ctx->alloc_counter + n : 0;
  return WISP_OK;
}

}  // extern "C"
