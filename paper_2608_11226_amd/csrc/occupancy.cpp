// Power metrics and threshold policy of the occupancy controller (section 4.5,
// eqs. (1)-(3), (5), (8)).  Host code; the window means sum the window in
// sample order every time, so the streaming monitor and the series functions
// give the same doubles.
#include "occupancy.h"

#include <algorithm>
#include <cmath>
#include <mutex>
#include <new>
#include <vector>

namespace {

constexpr int32_t kOk = 0;
constexpr int32_t kInval = -1;

int64_t window_samples(double dt_s, double window_s) { return std::max<int64_t>(1, std::llround(window_s / dt_s)); }

// mean of p[max(0, i - k + 1) .. i]
double window_mean(const double* p, int64_t i, int64_t k) {
  const int64_t lo = std::max<int64_t>(0, i - k + 1);
  double s = 0.0;
  for (int64_t j = lo; j <= i; ++j) s += p[j];
  return s / (double)(i + 1 - lo);
}

}  // namespace

struct occ_monitor {
  double dt_s, budget_w;
  int64_t k10, k30, back5;
  std::vector<double> p;
  int64_t n_viol = 0;
  double excess_ws = 0.0, p10 = 0.0, p30 = 0.0, peak30 = 0.0;
  mutable std::mutex mu;
};

extern "C" {

int32_t occ_rolling_mean(const double* p, int64_t n, double dt_s, double window_s, double* out) {
  if (n < 0 || !(dt_s > 0.0) || !(window_s >= dt_s) || (n > 0 && (!p || !out))) return kInval;
  const int64_t k = window_samples(dt_s, window_s);
  for (int64_t i = 0; i < n; ++i) out[i] = window_mean(p, i, k);
  return kOk;
}

int32_t occ_violation(const double* p30, int64_t n, double budget_w, double dt_s, double* rate, double* excess_ws) {
  if (n < 0 || !(dt_s > 0.0) || !rate || !excess_ws || (n > 0 && !p30)) return kInval;
  int64_t v = 0;
  double x = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    if (p30[i] > budget_w) ++v;
    x += std::max(0.0, p30[i] - budget_w);
  }
  *rate = n ? (double)v / (double)n : 0.0;
  *excess_ws = x * dt_s;
  return kOk;
}

double occ_normalize_budget(double budget_cal_w, double p4_new_w, double p4_cal_w) {
  return p4_cal_w > 0.0 ? budget_cal_w * p4_new_w / p4_cal_w : 0.0;
}

int32_t occ_hysteresis_step(int32_t level_idx, int32_t n_levels, double p30_w, double p10_w, double drop_w,
                            double climb30_w, double climb10_w) {
  if (n_levels < 1 || level_idx < 0 || level_idx >= n_levels) return kInval;
  if (p30_w > drop_w) return std::max(0, level_idx - 1);
  if (p30_w < climb30_w && p10_w < climb10_w) return std::min(n_levels - 1, level_idx + 1);
  return level_idx;
}

occ_monitor* occ_monitor_create(double dt_s, double budget_w) {
  if (!(dt_s > 0.0)) return nullptr;
  occ_monitor* m = new (std::nothrow) occ_monitor();
  if (!m) return nullptr;
  m->dt_s = dt_s;
  m->budget_w = budget_w;
  m->k10 = window_samples(dt_s, 10.0);
  m->k30 = window_samples(dt_s, 30.0);
  m->back5 = window_samples(dt_s, 5.0);
  return m;
}

int32_t occ_monitor_push(occ_monitor* m, double power_w) {
  if (!m) return kInval;
  std::lock_guard<std::mutex> g(m->mu);
  try {
    m->p.push_back(power_w);
  } catch (...) {
    return kInval;
  }
  const int64_t i = (int64_t)m->p.size() - 1;
  m->p10 = window_mean(m->p.data(), i, m->k10);
  m->p30 = window_mean(m->p.data(), i, m->k30);
  if (m->p30 > m->budget_w) ++m->n_viol;
  m->excess_ws += std::max(0.0, m->p30 - m->budget_w) * m->dt_s;
  m->peak30 = i == 0 ? m->p30 : std::max(m->peak30, m->p30);
  return kOk;
}

int32_t occ_monitor_read(const occ_monitor* m, occ_reading* out) {
  if (!m || !out) return kInval;
  std::lock_guard<std::mutex> g(m->mu);
  const int64_t n = (int64_t)m->p.size();
  out->n = n;
  out->p_now_w = n ? m->p[n - 1] : 0.0;
  out->p_5s_ago_w = n ? m->p[std::max<int64_t>(0, n - 1 - m->back5)] : 0.0;
  out->p10_w = m->p10;
  out->p30_w = m->p30;
  out->violation_rate = n ? (double)m->n_viol / (double)n : 0.0;
  out->excess_ws = m->excess_ws;
  out->peak30_w = m->peak30;
  return kOk;
}

int32_t occ_monitor_state(const occ_monitor* m, int32_t level, int32_t prev_level, double prev_duration_s,
                          double out[8]) {
  if (!m || !out) return kInval;
  occ_reading r;
  occ_monitor_read(m, &r);
  if (r.n == 0 || !(m->budget_w > 0.0)) return kInval;
  const double B = m->budget_w;
  out[0] = r.p_now_w / B;
  out[1] = r.p10_w / B;
  out[2] = r.p30_w / B;
  out[3] = (B - r.p30_w) / B;
  out[4] = (r.p_now_w - r.p_5s_ago_w) / B;
  out[5] = level / 8.0;
  out[6] = prev_level / 8.0;
  out[7] = prev_duration_s / 20.0;
  return kOk;
}

void occ_monitor_destroy(occ_monitor* m) { delete m; }

}  // extern "C"
