// Spatial controller: bandwidth-guided shared-stage CU cap (HorizonServe
// §4.4, Eq. (1); Algorithm 1, steps 1 and 3) and the memory-pressure sample
// it feeds on.  Host-only C++.
//
// Per scheduling step the caller passes the downstream activity A(t) and one
// sample B(t) of memory-system activity.  The controller smooths the sample
// with an EWMA, maps the normalised pressure rho = clamp(B_hat / B_sat, 0, 1)
// onto the co-running ladder S_min..S_cap (nearest level, ties upward), and
// applies the new level only if it is at least hysteresis_steps ladder levels
// away from the current one; with no downstream activity it returns the
// aggressive cap.  The downstream stage gets S_tot - s_shared.  The chosen
// counts are ladder levels of a context, so switching is the selection of a
// pre-built stream pair (§5), not the creation of one.
#include <dlfcn.h>

#include <cmath>
#include <cstdint>
#include <mutex>
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

// ---------------------------------------------------------------------------
// Memory-controller activity through the AMD SMI library, loaded on first use
// so that the library does not depend on it at link time.

struct AmdSmiStatics {
  std::once_flag once;
  bool ok = false;
  std::vector<void*> gpus;  // processor handles in enumeration order
  int (*get_activity)(void*, void*) = nullptr;
};
AmdSmiStatics g_smi;

constexpr uint64_t kAmdSmiInitGpus = 1ull << 1;  // AMDSMI_INIT_AMD_GPUS

void smi_load() {
  void* h = dlopen("libamd_smi.so", RTLD_NOW | RTLD_LOCAL);
  if (!h) h = dlopen("/opt/rocm/lib/libamd_smi.so", RTLD_NOW | RTLD_LOCAL);
  if (!h) return;
  auto init = reinterpret_cast<int (*)(uint64_t)>(dlsym(h, "amdsmi_init"));
  auto sockets = reinterpret_cast<int (*)(uint32_t*, void**)>(dlsym(h, "amdsmi_get_socket_handles"));
  auto procs = reinterpret_cast<int (*)(void*, uint32_t*, void**)>(dlsym(h, "amdsmi_get_processor_handles"));
  g_smi.get_activity = reinterpret_cast<int (*)(void*, void*)>(dlsym(h, "amdsmi_get_gpu_activity"));
  if (!init || !sockets || !procs || !g_smi.get_activity) return;
  if (init(kAmdSmiInitGpus) != 0) return;
  uint32_t n_sock = 0;
  if (sockets(&n_sock, nullptr) != 0 || n_sock == 0) return;
  std::vector<void*> socks(n_sock);
  if (sockets(&n_sock, socks.data()) != 0) return;
  for (uint32_t s = 0; s < n_sock; ++s) {
    uint32_t n = 0;
    if (procs(socks[s], &n, nullptr) != 0 || n == 0) continue;
    std::vector<void*> p(n);
    if (procs(socks[s], &n, p.data()) != 0) continue;
    g_smi.gpus.insert(g_smi.gpus.end(), p.begin(), p.begin() + n);
  }
  g_smi.ok = !g_smi.gpus.empty();
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

hs_status hs_pressure_sample(int32_t device, double* activity) {
  hs::clear_error();
  if (!activity) return hs::fail(HS_ERR_INVALID_ARG, "output pointer is null");
  std::call_once(g_smi.once, smi_load);
  if (!g_smi.ok) return hs::fail(HS_ERR_UNSUPPORTED, "AMD SMI is not available");
  if (device < 0 || device >= int32_t(g_smi.gpus.size()))
    return hs::fail(HS_ERR_INVALID_ARG, "device %d outside the %zu GPUs AMD SMI lists", device, g_smi.gpus.size());
  // amdsmi_engine_usage_t: gfx_activity, umc_activity, mm_activity (percent), reserved[13].
  uint32_t usage[16] = {0};
  if (g_smi.get_activity(g_smi.gpus[device], usage) != 0)
    return hs::fail(HS_ERR_UNSUPPORTED, "AMD SMI could not read the activity of device %d", device);
  *activity = double(usage[1]) / 100.0;
  return HS_OK;
}

}  // extern "C"
