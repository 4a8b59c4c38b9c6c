// Temporal scheduler: shared-stage path rotation with a slack guard and a
// long-path admission cap (HorizonServe §4.2 "Remaining-slack ratio", §4.3;
// Algorithm 1, steps 1 and 2).  Host-only C++.
//
// Per scheduling step the caller passes the queue as request views (path,
// waiting prefill or decode continuation, deadline, remaining-time estimate)
// and receives one visibility flag per request: the temporary queue view the
// base scheduler then batches from.  The queue itself is never reordered;
// hidden requests are simply visible again at the next step.
//   slack       u_i = (d_i - t) / r_hat_i; protected when u_i < u_guard
//   ratio       N = round(N_min + f (N_max - N_min)), f the protected share of
//               the waiting short-path prefills (0 when none wait)
//   rotation    step k is a short-path phase when k mod (N + M) < N
//   view        decode continuations and protected requests stay visible;
//               ordinary prefills of the other path are hidden
//   cap         at most long_cap ordinary long-path prefills stay visible,
//               earliest deadlines first (ties: earlier queue position)
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "horizon.h"
#include "plan.h"

struct hs_temporal {
  hs_temporal_cfg cfg;
  int64_t k = 0;  // scheduling steps taken
};

extern "C" {

hs_status hs_temporal_create(const hs_temporal_cfg* cfg, hs_temporal** out) {
  hs::clear_error();
  if (!cfg || !out) return hs::fail(HS_ERR_INVALID_ARG, "config or output pointer is null");
  *out = nullptr;
  if (!(1 <= cfg->n_min && cfg->n_min <= cfg->n_max))
    return hs::fail(HS_ERR_INVALID_ARG, "need 1 <= N_min (%d) <= N_max (%d)", cfg->n_min, cfg->n_max);
  if (cfg->m < 1) return hs::fail(HS_ERR_INVALID_ARG, "M = %d must be >= 1", cfg->m);
  if (!(cfg->u_guard > 0.0) || !std::isfinite(cfg->u_guard))
    return hs::fail(HS_ERR_INVALID_ARG, "u_guard must be a positive finite number");
  auto* s = new hs_temporal;
  s->cfg = *cfg;
  *out = s;
  return HS_OK;
}

hs_status hs_temporal_step(hs_temporal* s, double now, const hs_request_view* reqs, int32_t n_reqs,
                           uint8_t* visible, hs_temporal_step_info* info) {
  hs::clear_error();
  if (!s) return hs::fail(HS_ERR_INVALID_ARG, "scheduler is null");
  if (n_reqs < 0) return hs::fail(HS_ERR_INVALID_ARG, "n_reqs %d < 0", n_reqs);
  if (n_reqs > 0 && (!reqs || !visible)) return hs::fail(HS_ERR_INVALID_ARG, "request or visibility array is null");
  if (!std::isfinite(now)) return hs::fail(HS_ERR_INVALID_ARG, "time is not finite");
  for (int32_t i = 0; i < n_reqs; ++i) {
    const hs_request_view& r = reqs[i];
    if ((r.path != HS_PATH_SHORT && r.path != HS_PATH_LONG) || (r.work != HS_WORK_PREFILL && r.work != HS_WORK_DECODE))
      return hs::fail(HS_ERR_INVALID_ARG, "request %d: path %d / work %d unknown", i, r.path, r.work);
    if (!std::isfinite(r.deadline) || !(r.remaining > 0.0) || !std::isfinite(r.remaining))
      return hs::fail(HS_ERR_INVALID_ARG, "request %d: deadline must be finite and remaining > 0", i);
  }
  const hs_temporal_cfg& c = s->cfg;
  // Step 1: slack and the protected bit.
  std::vector<uint8_t> prot(static_cast<size_t>(n_reqs));
  int32_t short_wait = 0, short_prot = 0, n_prot = 0;
  for (int32_t i = 0; i < n_reqs; ++i) {
    const hs_request_view& r = reqs[i];
    prot[i] = (r.deadline - now) / r.remaining < c.u_guard;
    n_prot += prot[i];
    if (r.work == HS_WORK_PREFILL && r.path == HS_PATH_SHORT) {
      ++short_wait;
      short_prot += prot[i];
    }
  }
  // Adaptive ratio and the phase of step k.
  const double frac = short_wait ? double(short_prot) / double(short_wait) : 0.0;
  const int32_t N = int32_t(std::floor(double(c.n_min) + frac * double(c.n_max - c.n_min) + 0.5));
  const int32_t phase = (s->k % int64_t(N + c.m)) < N ? HS_PATH_SHORT : HS_PATH_LONG;
  // Step 2: the temporary view.
  int32_t n_hidden = 0;
  std::vector<int32_t> cand;
  for (int32_t i = 0; i < n_reqs; ++i) {
    const hs_request_view& r = reqs[i];
    visible[i] = r.work == HS_WORK_DECODE || prot[i] || r.path == phase;
    n_hidden += !visible[i];
    if (visible[i] && r.work == HS_WORK_PREFILL && r.path == HS_PATH_LONG && !prot[i]) cand.push_back(i);
  }
  int32_t n_capped = 0;
  if (c.long_cap >= 0 && int32_t(cand.size()) > c.long_cap) {
    std::stable_sort(cand.begin(), cand.end(),
                     [&](int32_t a, int32_t b) { return reqs[a].deadline < reqs[b].deadline; });
    for (size_t j = size_t(c.long_cap); j < cand.size(); ++j) {
      visible[cand[j]] = 0;
      ++n_capped;
    }
  }
  if (info) {
    info->step = s->k;
    info->n = N;
    info->phase = phase;
    info->n_protected = n_prot;
    info->n_hidden = n_hidden;
    info->n_capped = n_capped;
  }
  ++s->k;
  return HS_OK;
}

hs_status hs_temporal_destroy(hs_temporal* s) {
  delete s;
  return HS_OK;
}

}  // extern "C"
