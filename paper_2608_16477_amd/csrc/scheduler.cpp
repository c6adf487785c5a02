// Scheduler Engine: the prefetching-window model (Section 4.1) and its
// online selection (Section 4.2, Algorithm 1), admission, telemetry
// smoothing and the stale-preparation bound (Section 4.4).  Host-only
// scalar code: a decision evaluates O(T_limit / dt) candidates and takes
// microseconds, next to the prefill it schedules.
#include <cmath>
#include <cstdint>
#include <string>

#include "pallas.h"

namespace {

bool valid(const pallas_window_params* p) {
  return p && p->r_p > 0.0 && p->r_d >= 0.0 && p->goodput > 0.0 && p->s_kv >= 0.0 && p->t_load >= 0.0 &&
         p->t_0 >= 0.0 && p->alpha >= 0.0 && p->alpha <= 1.0 && p->t_max >= 0.0 && p->dt > 0.0 &&
         std::isfinite(p->r_p) && std::isfinite(p->r_d) && std::isfinite(p->goodput) &&
         std::isfinite(p->s_kv) && std::isfinite(p->t_load) && std::isfinite(p->t_0) &&
         std::isfinite(p->t_max) && std::isfinite(p->dt);
}

// Eqs. 3-9 at window t_w.
void model(const pallas_window_params& p, double k_curr, double t_remain, double t_w,
           pallas_window_decision* d) {
  const double l_hist = k_curr + p.r_d * (t_remain - t_w);       // Eq. 9
  const double t_hist = p.t_load + l_hist / p.r_p;                // Eq. 4
  const double s_inc = p.r_d * t_w * p.s_kv;                      // Eq. 3
  const double t_res = std::fmax(0.0, s_inc / p.goodput - t_w);   // Eq. 5
  const double t_sit = p.t_0 + std::fmax(0.0, std::fmax(t_hist - t_w, t_res));  // Eq. 6
  const double t_early = std::fmax(0.0, t_w - t_hist);            // Eq. 7
  d->t_w = t_w;
  d->l_hist = l_hist;
  d->t_hist = t_hist;
  d->t_res = t_res;
  d->t_sit = t_sit;
  d->t_early = t_early;
  d->cost = p.alpha * t_sit + (1.0 - p.alpha) * t_early;          // Eq. 8
  d->n_candidates = 1;
  d->trigger = 0;
}

}  // namespace

extern "C" {

int pallas_window_evaluate(const pallas_window_params* p, double k_curr, double t_remain, double t_w,
                           pallas_window_decision* out) {
  if (!valid(p) || !out || !(t_w >= 0.0) || !std::isfinite(t_w) || !std::isfinite(k_curr) ||
      !std::isfinite(t_remain))
    return PALLAS_ERR_INVALID_ARG;
  model(*p, k_curr, t_remain, t_w, out);
  return PALLAS_OK;
}

int pallas_window_select(const pallas_window_params* p, double k_curr, double t_remain,
                         pallas_window_decision* out) {
  if (!valid(p) || !out || !std::isfinite(k_curr) || !std::isfinite(t_remain))
    return PALLAS_ERR_INVALID_ARG;
  const double t_limit = std::fmin(p->t_max, std::fmax(t_remain, 0.0));
  const double steps = std::floor(t_limit / p->dt);
  if (steps > 1e7) return PALLAS_ERR_INVALID_ARG;
  const int64_t last_k = static_cast<int64_t>(steps);
  pallas_window_decision best, cur;
  model(*p, k_curr, t_remain, 0.0, &best);
  int64_t n = 1;
  double last = 0.0;
  for (int64_t k = 1; k <= last_k; ++k) {
    last = std::fmin(static_cast<double>(k) * p->dt, t_limit);
    model(*p, k_curr, t_remain, last, &cur);
    ++n;
    if (cur.cost < best.cost) best = cur;
  }
  // T_limit closes the grid when it is not a multiple of dt.
  if (t_limit - last > 1e-12 * std::fmax(1.0, t_limit)) {
    model(*p, k_curr, t_remain, t_limit, &cur);
    ++n;
    if (cur.cost < best.cost) best = cur;
  }
  best.n_candidates = static_cast<int32_t>(n);
  best.trigger = t_remain <= best.t_w ? 1 : 0;
  *out = best;
  return PALLAS_OK;
}

double pallas_ewma_update(pallas_ewma* e, double sample, double weight) {
  if (!e || !(weight > 0.0) || weight > 1.0) return std::nan("");
  if (!e->primed) {
    e->value = sample;
    e->primed = 1;
  } else {
    e->value = weight * sample + (1.0 - weight) * e->value;
  }
  return e->value;
}

int32_t pallas_admit(int32_t model_compatible, double vram_free_bytes, double s_kv, double k_curr,
                     double r_d, double t_remain) {
  if (!model_compatible) return 0;
  const double need = s_kv * (k_curr + r_d * std::fmax(t_remain, 0.0));
  return vram_free_bytes >= need ? 1 : 0;
}

double pallas_waste_bound(double t_max, double e_early, double t_avail) {
  return std::fmax(t_max + e_early - t_avail, 0.0);
}

}  // extern "C"
