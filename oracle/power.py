"""Power metrics and the hysteresis occupancy rule of the occupancy controller.

TEST INFRASTRUCTURE ONLY (see the package header): the library implements the
same definitions natively (``include/occupancy.h``); this module is what the
tests hold it against.

Definitions, section 4.5 "Occupancy-controller methodology":
  rolling_mean        eq. (1): mean power over the trailing window of w seconds
  violation_rate      eq. (2): fraction of samples whose 30 s rolling mean exceeds the budget B
  integrated_excess   eq. (3): sum of the 30 s rolling mean's excess over B, times the sample period
  state_vector        eq. (5): the eight budget-normalised features at a batch boundary
  normalize_budget    eq. (8): a budget carried to a new plant in proportion to its batch-4 mean power
  hysteresis_step     the threshold baseline of section 4.5: drop one batch level when the 30 s mean
                      exceeds the drop threshold, climb one when the 30 s mean is below the climb
                      threshold and the 10 s mean below its own

Readings (also listed in the design notes):
  * eq. (1) sums tau from t - w to t with the factor dt / w: read as the mean of the w / dt samples
    ending at t (the trailing w seconds); while fewer than w / dt samples exist, the mean of those so far.
  * Batch levels are positions in an ordered list (the paper's {1, 2, 4, 8}); the rule never leaves it.
  * P(t - 5) in eq. (5) is the sample 5 s earlier, or the first sample while fewer exist.

Parity: pinned in tests/test_oracle_power.py against closed forms (constant and step series, a ramp's
excess), hand-traced hysteresis sequences, and the paper's own calibration figures for eq. (8).
"""
from __future__ import annotations

import math

import numpy as np

LEVELS = (1, 2, 4, 8)


def rolling_mean(p, dt: float, window_s: float) -> np.ndarray:
    """Eq. (1) at every sample: mean of the samples in the trailing window_s seconds."""
    p = np.asarray(p, dtype=np.float64)
    k = int(round(window_s / dt))
    out = np.empty_like(p)
    for i in range(len(p)):
        lo = max(0, i - k + 1)
        out[i] = math.fsum(p[lo:i + 1]) / (i + 1 - lo)  # correctly rounded window sum
    return out


def violation_rate(p30, budget_w: float) -> float:
    """Eq. (2): share of samples whose 30 s mean exceeds the budget."""
    p30 = np.asarray(p30, dtype=np.float64)
    return float(np.sum(p30 > budget_w)) / len(p30) if len(p30) else 0.0


def integrated_excess(p30, budget_w: float, dt: float) -> float:
    """Eq. (3): watt-seconds of the 30 s mean above the budget."""
    p30 = np.asarray(p30, dtype=np.float64)
    return math.fsum(np.maximum(0.0, p30 - budget_w)) * dt


def state_vector(p, dt: float, budget_w: float, level: int, prev_level: int, prev_duration_s: float) -> np.ndarray:
    """Eq. (5) at the last sample of p (levels in batch units, e.g. 4 for batch level 4)."""
    p = np.asarray(p, dtype=np.float64)
    p10 = rolling_mean(p, dt, 10.0)[-1]
    p30 = rolling_mean(p, dt, 30.0)[-1]
    back = int(round(5.0 / dt))
    p_prev = p[max(0, len(p) - 1 - back)]
    return np.array([p[-1] / budget_w, p10 / budget_w, p30 / budget_w, (budget_w - p30) / budget_w,
                     (p[-1] - p_prev) / budget_w, level / 8.0, prev_level / 8.0, prev_duration_s / 20.0])


def normalize_budget(budget_cal_w: float, p4_new_w: float, p4_cal_w: float) -> float:
    """Eq. (8): the budget that keeps the batch-4-to-budget ratio of the calibration plant."""
    return budget_cal_w * p4_new_w / p4_cal_w


def hysteresis_step(level_idx: int, n_levels: int, p30: float, p10: float, drop_w: float, climb30_w: float,
                    climb10_w: float) -> int:
    """Next level index under the threshold rule (section 4.5)."""
    if p30 > drop_w:
        return max(0, level_idx - 1)
    if p30 < climb30_w and p10 < climb10_w:
        return min(n_levels - 1, level_idx + 1)
    return level_idx
