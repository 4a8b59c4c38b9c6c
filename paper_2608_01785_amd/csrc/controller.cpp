// Spatial controller: bandwidth-guided shared-stage CU cap (HorizonServe
// §4.4, Eq. (1); Algorithm 1, steps 1 and 3).  Host-only C++.
//
// Per scheduling step the caller passes the downstream activity A(t) and one
// sample B(t) of memory-system activity.  The controller smooths the sample
// with an EWMA, maps the normalised pressure rho = clamp(B_hat / B_sat, 0, 1)
// onto the co-running ladder S_min..S_cap (nearest level, ties upward), and
// applies the new level only if it is at least hysteresis_steps ladder levels
// away from the current one; with no downstream activity it returns the
// aggressive cap.  The downstream stage gets S_tot - s_shared.  The chosen
// counts are ladder levels of a context, so switching is the selection of a
// pre-built stream pair (§5), not the creation of one.  The sample itself
// comes from pressure.cpp.
#include <cmath>
#include <cstdint>
#include <vector>

#include "horizon.h"
#include "plan.h"

struct hs_controller {
  int32_t total = 0, aggressive = 0;
  std::vector<int32_t> ladder;
  double gamma = 0.0, saturation = 0.0;
  int32_t step_min = 1;
  bool have_sample = false;
  double b_hat = 0.0;
  bool have_prev = false;
  int32_t prev_shared = 0, prev_level = -1;
};

namespace {

// Index of the ladder level nearest to x; a tie goes to the larger level.
int32_t snap_level(const std::vector<int32_t>& ladder, double x) {
  int32_t best = 0;
  for (int32_t i = 0; i < int32_t(ladder.size()); ++i)
    if (std::fabs(ladder[i] - x) <= std::fabs(ladder[best] - x)) best = i;
  return best;
}

}  // namespace

extern "C" {

hs_status hs_controller_create(const hs_controller_cfg* cfg, hs_controller** out) {
  hs::clear_error();
  if (!cfg || !out) return hs::fail(HS_ERR_INVALID_ARG, "config or output pointer is null");
  *out = nullptr;
  if (!cfg->ladder || cfg->n_ladder < 1) return hs::fail(HS_ERR_INVALID_ARG, "the co-running ladder is empty");
  for (int32_t i = 0; i < cfg->n_ladder; ++i) {
    if (cfg->ladder[i] < 1) return hs::fail(HS_ERR_INVALID_ARG, "ladder level %d is %d < 1", i, cfg->ladder[i]);
    if (i > 0 && cfg->ladder[i] <= cfg->ladder[i - 1])
      return hs::fail(HS_ERR_INVALID_ARG, "ladder levels must increase strictly (level %d)", i);
  }
  const int32_t s_cap = cfg->ladder[cfg->n_ladder - 1];
  if (!(s_cap < cfg->aggressive_cus && cfg->aggressive_cus <= cfg->total_cus))
    return hs::fail(HS_ERR_INVALID_ARG, "need S_cap (%d) < S_aggr (%d) <= S_tot (%d)", s_cap, cfg->aggressive_cus,
                    cfg->total_cus);
  if (!(cfg->ewma_weight > 0.0 && cfg->ewma_weight <= 1.0))
    return hs::fail(HS_ERR_INVALID_ARG, "EWMA weight %g outside (0, 1]", cfg->ewma_weight);
  if (!(cfg->saturation > 0.0)) return hs::fail(HS_ERR_INVALID_ARG, "saturation pressure must be > 0");
  if (cfg->hysteresis_steps < 1) return hs::fail(HS_ERR_INVALID_ARG, "hysteresis_steps must be >= 1");
  auto* c = new hs_controller;
  c->total = cfg->total_cus;
  c->aggressive = cfg->aggressive_cus;
  c->ladder.assign(cfg->ladder, cfg->ladder + cfg->n_ladder);
  c->gamma = cfg->ewma_weight;
  c->saturation = cfg->saturation;
  c->step_min = cfg->hysteresis_steps;
  *out = c;
  return HS_OK;
}

hs_status hs_controller_step(hs_controller* c, int32_t downstream_active, double sample, hs_split* out) {
  hs::clear_error();
  if (!c || !out) return hs::fail(HS_ERR_INVALID_ARG, "controller or output pointer is null");
  if (!std::isfinite(sample)) return hs::fail(HS_ERR_INVALID_ARG, "pressure sample is not finite");
  // Step 1: EWMA of the pressure signal (the first sample initialises it).
  c->b_hat = c->have_sample ? c->gamma * sample + (1.0 - c->gamma) * c->b_hat : sample;
  c->have_sample = true;
  const double rho = std::fmin(std::fmax(c->b_hat / c->saturation, 0.0), 1.0);
  // Eq. (1).
  int32_t level = -1, target = c->aggressive;
  if (downstream_active) {
    const double s_min = c->ladder.front(), s_cap = c->ladder.back();
    level = snap_level(c->ladder, s_min + rho * (s_cap - s_min));
    target = c->ladder[level];
  }
  // Step 3: hysteresis on the ladder level.
  const bool apply = !downstream_active || !c->have_prev || c->prev_level < 0 ||
                     std::abs(level - c->prev_level) >= c->step_min;
  bool changed = false;
  if (apply) {
    changed = !c->have_prev || c->prev_shared != target;
    c->prev_shared = target;
    c->prev_level = level;
    c->have_prev = true;
  }
  out->shared_cus = c->prev_shared;
  out->down_cus = c->total > c->prev_shared ? c->total - c->prev_shared : 0;
  out->level = c->prev_level;
  out->changed = changed ? 1 : 0;
  out->pressure = c->b_hat;
  out->rho = rho;
  return HS_OK;
}

hs_status hs_controller_destroy(hs_controller* c) {
  delete c;
  return HS_OK;
}

}  // extern "C"
