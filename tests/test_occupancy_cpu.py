"""The native occupancy metrics (include/occupancy.h, host code) against the oracle's definitions."""
import numpy as np
import pytest

import paper_2608_11226_amd as R
from oracle import power as O


def _trace(n, seed):
    rng = np.random.default_rng(seed)
    base = 900.0 + 120.0 * np.sin(np.arange(n) / 37.0)
    return base + rng.normal(0.0, 35.0, n)


@pytest.mark.parametrize("window", [0.5, 5.0, 10.0, 30.0, 31.3])
def test_rolling_mean_matches_oracle(window):
    p = _trace(500, 1)
    # the library sums each window in sample order, the oracle rounds the exact sum once
    assert np.allclose(R.occ_rolling_mean(p, 0.5, window), O.rolling_mean(p, 0.5, window), rtol=1e-12, atol=0)


def test_violation_matches_oracle():
    p30 = O.rolling_mean(_trace(800, 2), 0.5, 30.0)
    for budget in (850.0, 900.0, 950.0, 2000.0):
        assert np.min(np.abs(p30 - budget)) > 1e-6
        rate, excess = R.occ_violation(p30, budget, 0.5)
        assert rate == O.violation_rate(p30, budget)
        assert excess == pytest.approx(O.integrated_excess(p30, budget, 0.5), rel=1e-12, abs=1e-9)


def test_monitor_streams_the_series_definitions():
    p = _trace(300, 3)
    m = R.OccMonitor(0.5, 920.0)
    for i, x in enumerate(p):
        m.push(x)
        r = m.read()
        assert r.n == i + 1
    p10 = O.rolling_mean(p, 0.5, 10.0)
    p30 = O.rolling_mean(p, 0.5, 30.0)
    assert r.p10_w == pytest.approx(p10[-1], rel=1e-12) and r.p30_w == pytest.approx(p30[-1], rel=1e-12)
    assert r.violation_rate == O.violation_rate(p30, 920.0)  # no 30 s mean lies within 1e-9 of the budget here
    assert np.min(np.abs(p30 - 920.0)) > 1e-6
    assert r.excess_ws == pytest.approx(O.integrated_excess(p30, 920.0, 0.5), rel=1e-12)
    assert r.peak30_w == pytest.approx(p30.max(), rel=1e-12)
    s = m.state(level=4, prev_level=8, prev_duration_s=12.0)
    assert np.allclose(s, O.state_vector(p, 0.5, 920.0, 4, 8, 12.0), rtol=0, atol=1e-12)
    m.close()


def test_hysteresis_and_budget_match_oracle():
    rng = np.random.default_rng(4)
    for _ in range(2000):
        idx = int(rng.integers(0, 4))
        p30, p10 = rng.uniform(480, 540, 2)
        assert R.occ_hysteresis_step(idx, 4, p30, p10, 512, 510, 525) == O.hysteresis_step(idx, 4, p30, p10, 512, 510, 525)
    assert R.occ_normalize_budget(520, 498.4, 462) == pytest.approx(O.normalize_budget(520, 498.4, 462))


def test_argument_errors():
    with pytest.raises(R.RolloutError):
        R.occ_rolling_mean(np.ones(4), 0.0, 30.0)
    with pytest.raises(R.RolloutError):
        R.occ_rolling_mean(np.ones(4), 0.5, 0.1)
    with pytest.raises(R.RolloutError):
        R.occ_hysteresis_step(4, 4, 0, 0, 1, 1, 1)
    with pytest.raises(R.RolloutError):
        R.OccMonitor(0.0, 500.0)
    m = R.OccMonitor(0.5, 500.0)
    with pytest.raises(R.RolloutError):
        m.state(4, 4, 1.0)  # no sample yet
    m.close()
