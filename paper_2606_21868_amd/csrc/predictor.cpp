// The co-activation predictor of WiSP (App. E): online co-firing counts between a source layer and
// the later layers within a horizon, and the decayed, source-normalised score of a target layer's
// candidates from the layers already routed in the current pass.  Host code.
#include <algorithm>
#include <cmath>
#include <new>
#include <vector>

#include "errors.hpp"
#include "wisp_predictor.h"

using wisp::set_error;

struct wisp_predictor {
  int32_t L = 0, N = 0, H = 0;
  double gamma = 1.0;
  // counts[((l' * H + d - 1) * N + e) * N + e']: e at layer l' - d and e' at layer l' in one pass
  std::vector<uint32_t> counts;
  // row[(l' * H + d - 1) * N + e] = sum over e' of the counts above (the source marginal)
  std::vector<uint64_t> row;
  std::vector<std::vector<int32_t>> cur;   // the current pass's routed set per layer
  std::vector<uint8_t> seen;               // scratch, per layer
};

namespace {

size_t cidx(const wisp_predictor* p, int32_t lt, int32_t d, int32_t e, int32_t et) {
  return ((static_cast<size_t>(lt) * p->H + (d - 1)) * p->N + e) * p->N + et;
}

size_t ridx(const wisp_predictor* p, int32_t lt, int32_t d, int32_t e) {
  return (static_cast<size_t>(lt) * p->H + (d - 1)) * p->N + e;
}

}  // namespace

extern "C" {

wisp_status wisp_predictor_create(int32_t n_layers, int32_t n_experts, int32_t horizon, double gamma,
                                  wisp_predictor** out) {
  if (!out) return set_error(WISP_E_INVAL, "predictor: out is NULL");
  *out = nullptr;
  if (n_layers < 1 || n_experts < 1 || n_experts > 4096 || horizon < 1 || !(gamma > 0.0 && gamma <= 1.0))
    return set_error(WISP_E_INVAL, "predictor: bad shape, horizon or gamma (0 < gamma <= 1)");
  const int32_t H = std::min(horizon, std::max(1, n_layers - 1));
  const double cells = static_cast<double>(n_layers) * H * n_experts * n_experts;
  if (cells > 1.5e9) return set_error(WISP_E_INVAL, "predictor: tables too large (lower the horizon)");
  auto* p = new (std::nothrow) wisp_predictor();
  if (!p) return set_error(WISP_E_NOMEM, "predictor: host allocation failed");
  try {
    p->L = n_layers;
    p->N = n_experts;
    p->H = H;
    p->gamma = gamma;
    p->counts.assign(static_cast<size_t>(cells), 0u);
    p->row.assign(static_cast<size_t>(n_layers) * H * n_experts, 0u);
    p->cur.assign(n_layers, {});
    p->seen.assign(n_experts, 0);
  } catch (...) {
    delete p;
    return set_error(WISP_E_NOMEM, "predictor: host allocation failed");
  }
  *out = p;
  return WISP_OK;
}

wisp_status wisp_predictor_destroy(wisp_predictor* p) {
  if (!p) return set_error(WISP_E_INVAL, "predictor: NULL");
  delete p;
  return WISP_OK;
}

wisp_status wisp_predictor_shape(const wisp_predictor* p, int32_t* n_layers, int32_t* n_experts) {
  if (!p || !n_layers || !n_experts) return set_error(WISP_E_INVAL, "predictor: NULL argument");
  *n_layers = p->L;
  *n_experts = p->N;
  return WISP_OK;
}

wisp_status wisp_predictor_observe(wisp_predictor* p, int32_t layer, const int32_t* ids, int32_t n) {
  if (!p || (!ids && n > 0) || n < 0) return set_error(WISP_E_INVAL, "predictor: bad argument");
  if (layer < 0 || layer >= p->L) return set_error(WISP_E_INVAL, "predictor: layer out of range");
  for (int32_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= p->N) return set_error(WISP_E_INVAL, "predictor: expert id out of range");
  auto& s = p->cur[layer];
  s.clear();
  for (int32_t i = 0; i < n; ++i)
    if (!p->seen[ids[i]]) {
      p->seen[ids[i]] = 1;
      s.push_back(ids[i]);
    }
  for (int32_t e : s) p->seen[e] = 0;
  std::sort(s.begin(), s.end());
  return WISP_OK;
}

wisp_status wisp_predictor_end_pass(wisp_predictor* p) {
  if (!p) return set_error(WISP_E_INVAL, "predictor: NULL");
  for (int32_t lt = 1; lt < p->L; ++lt) {
    const auto& tgt = p->cur[lt];
    if (tgt.empty()) continue;
    for (int32_t d = 1; d <= p->H && lt - d >= 0; ++d) {
      for (int32_t e : p->cur[lt - d]) {
        for (int32_t et : tgt) ++p->counts[cidx(p, lt, d, e, et)];
        p->row[ridx(p, lt, d, e)] += tgt.size();
      }
    }
  }
  for (auto& s : p->cur) s.clear();
  return WISP_OK;
}

wisp_status wisp_predictor_predict(wisp_predictor* p, int32_t layer, int32_t depth, int32_t* ids_out, int32_t* n_out,
                                   double* scores_out) {
  if (!p || !n_out || depth < 0 || (depth > 0 && !ids_out)) return set_error(WISP_E_INVAL, "predictor: bad argument");
  if (layer < 0 || layer >= p->L) return set_error(WISP_E_INVAL, "predictor: layer out of range");
  std::vector<double> score(p->N, 0.0);
  double decay = 1.0;
  for (int32_t d = 1; d <= p->H && layer - d >= 0; ++d) {
    decay *= p->gamma;
    for (int32_t e : p->cur[layer - d]) {
      const uint64_t rs = p->row[ridx(p, layer, d, e)];
      if (rs == 0) continue;
      const double scale = decay / static_cast<double>(rs);
      const uint32_t* c = &p->counts[cidx(p, layer, d, e, 0)];
      for (int32_t et = 0; et < p->N; ++et)
        if (c[et]) score[et] += scale * static_cast<double>(c[et]);
    }
  }
  std::vector<int32_t> order;
  for (int32_t et = 0; et < p->N; ++et)
    if (score[et] > 0.0) order.push_back(et);
  const size_t keep = std::min(order.size(), static_cast<size_t>(depth));
  std::partial_sort(order.begin(), order.begin() + keep, order.end(), [&](int32_t a, int32_t b) {
    return score[a] > score[b] || (score[a] == score[b] && a < b);
  });
  for (size_t i = 0; i < keep; ++i) {
    ids_out[i] = order[i];
    if (scores_out) scores_out[i] = score[order[i]];
  }
  *n_out = static_cast<int32_t>(keep);
  return WISP_OK;
}

}  // extern "C"
