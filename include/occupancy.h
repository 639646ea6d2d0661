/* Occupancy actuation: the power metrics and the threshold policy of the
 * paper's occupancy controller (section 4.5, "Occupancy-controller
 * methodology"), for a loop that picks the rollout's generation batch level
 * (groups in flight) at wave boundaries from sampled device power.
 *
 * Host code only: no device memory, no HIP calls.  Power is in watts, time in
 * seconds, samples are taken every dt_s seconds (the paper samples at 0.5 s).
 * Functions return 0 on success and -1 (ROLLOUT_EINVAL) for invalid arguments,
 * writing nothing in that case.  Pointers are caller-owned.
 */
#pragma once

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Eq. (1) over a series: out[i] = mean of p[max(0, i - k + 1) .. i] with
 * k = round(window_s / dt_s), i.e. the trailing window_s seconds (the mean of
 * the samples so far while fewer than k exist).  p and out hold n doubles and
 * may not overlap.  Errors: n < 0, dt_s <= 0, window_s < dt_s, NULL pointers. */
int32_t occ_rolling_mean(const double* p, int64_t n, double dt_s, double window_s, double* out);

/* Eqs. (2) and (3) over a series of 30 s means: *rate = share of samples with
 * p30[i] > budget_w (0 for n = 0), *excess_ws = dt_s * sum(max(0, p30[i] - budget_w)).
 * Errors: n < 0, dt_s <= 0, NULL pointers. */
int32_t occ_violation(const double* p30, int64_t n, double budget_w, double dt_s, double* rate, double* excess_ws);

/* Eq. (8): budget_cal_w * p4_new_w / p4_cal_w, the budget that keeps the
 * calibration plant's ratio of batch-4 mean power to budget.  Returns 0 when
 * p4_cal_w <= 0. */
double occ_normalize_budget(double budget_cal_w, double p4_new_w, double p4_cal_w);

/* The threshold baseline of section 4.5 over n_levels ordered batch levels:
 * one level down when p30_w > drop_w; else one level up when p30_w < climb30_w
 * and p10_w < climb10_w; else unchanged.  The result stays in [0, n_levels).
 * Returns -1 when level_idx is outside [0, n_levels) or n_levels < 1. */
int32_t occ_hysteresis_step(int32_t level_idx, int32_t n_levels, double p30_w, double p10_w, double drop_w,
                            double climb30_w, double climb10_w);

/* Streaming monitor: one power sample per dt_s.  After each push it holds the
 * eq. (1) means over the trailing 10 s and 30 s and accumulates eqs. (2)-(3)
 * over every sample pushed so far, with the same arithmetic as the series
 * functions above.  A monitor may be used from several threads. */
typedef struct occ_monitor occ_monitor;

typedef struct {
  int64_t n;                   /* samples pushed */
  double p_now_w, p_5s_ago_w;  /* latest sample, and the one 5 s earlier (first sample while fewer exist) */
  double p10_w, p30_w;         /* eq. (1) at the latest sample */
  double violation_rate;       /* eq. (2) over all samples */
  double excess_ws;            /* eq. (3) over all samples */
  double peak30_w;             /* largest 30 s mean so far */
} occ_reading;

/* NULL on invalid arguments (dt_s <= 0) or allocation failure. */
occ_monitor* occ_monitor_create(double dt_s, double budget_w);
int32_t occ_monitor_push(occ_monitor* m, double power_w);
int32_t occ_monitor_read(const occ_monitor* m, occ_reading* out);
/* Eq. (5) at the latest sample: [P/B, P10/B, P30/B, (B - P30)/B, (P - P(t-5 s))/B, level/8,
 * prev_level/8, prev_duration_s/20] (levels in batch units).  Error when no sample was pushed. */
int32_t occ_monitor_state(const occ_monitor* m, int32_t level, int32_t prev_level, double prev_duration_s,
                          double out[8]);
void occ_monitor_destroy(occ_monitor* m);

#ifdef __cplusplus
}
#endif
