"""Pins for oracle/power.py: closed forms, hand-traced sequences and the paper's calibration figures."""
import numpy as np
import pytest

from conftest import read_golden
from oracle import power as O


def golden():
    return {k: float(v) for k, v in read_golden("occupancy_budget.txt")}


def test_rolling_mean_constant_and_warmup():
    p = np.full(200, 400.0)
    assert np.allclose(O.rolling_mean(p, 0.5, 30.0), 400.0)
    q = np.arange(1, 11, dtype=float)  # 1..10 at dt 0.5, window 2 s = 4 samples
    got = O.rolling_mean(q, 0.5, 2.0)
    want = [1, 1.5, 2, 2.5, 3.5, 4.5, 5.5, 6.5, 7.5, 8.5]  # warm-up means, then (i-2 .. i+1) means by hand
    assert np.allclose(got, want)


def test_rolling_mean_step_series():
    # 0 W for 30 s then 100 W: the 30 s mean rises by 100/60 per sample until it saturates
    dt = 0.5
    p = np.concatenate([np.zeros(60), np.full(90, 100.0)])
    m = O.rolling_mean(p, dt, 30.0)
    assert m[59] == 0.0
    for j in range(60):
        assert m[60 + j] == pytest.approx(100.0 * (j + 1) / 60)
    assert np.allclose(m[119:], 100.0)


def test_violation_rate_and_excess_closed_forms():
    dt = 0.5
    p30 = np.full(100, 400.0)
    assert O.violation_rate(p30, 500.0) == 0.0
    assert O.violation_rate(p30, 300.0) == 1.0
    assert O.integrated_excess(p30, 300.0, dt) == pytest.approx(100.0 * dt * 100)
    # a ramp 0..99 W over 100 samples against B = 49.5: excess = dt * sum_{k=50}^{99} (k - 49.5)
    ramp = np.arange(100, dtype=float)
    assert O.violation_rate(ramp, 49.5) == 0.5
    assert O.integrated_excess(ramp, 49.5, dt) == pytest.approx(dt * sum(k - 49.5 for k in range(50, 100)))
    # equality is not a violation (strict ">")
    assert O.violation_rate(np.full(4, 500.0), 500.0) == 0.0


def test_state_vector_features():
    dt = 0.5
    p = np.concatenate([np.full(100, 300.0), np.full(20, 500.0)])  # last 10 s at 500 W
    s = O.state_vector(p, dt, 600.0, level=4, prev_level=2, prev_duration_s=15.0)
    p30 = (40 * 300.0 + 20 * 500.0) / 60
    assert s[0] == pytest.approx(500.0 / 600)
    assert s[1] == pytest.approx(500.0 / 600)
    assert s[2] == pytest.approx(p30 / 600)
    assert s[3] == pytest.approx((600 - p30) / 600)
    assert s[4] == pytest.approx(0.0)  # 5 s ago was also 500 W
    assert list(s[5:]) == pytest.approx([0.5, 0.25, 0.75])


def test_budget_rule_against_the_paper():
    g = golden()
    assert g["p4_cal_w"] / g["budget_cal_w"] == pytest.approx(g["ratio"], abs=5e-4)
    # the hardware budget keeps that ratio: the plant's batch-4 power it implies, carried back, gives 561 W
    p4_new = g["budget_new_w"] * g["p4_cal_w"] / g["budget_cal_w"]
    assert O.normalize_budget(g["budget_cal_w"], p4_new, g["p4_cal_w"]) == pytest.approx(g["budget_new_w"])
    assert p4_new / O.normalize_budget(g["budget_cal_w"], p4_new, g["p4_cal_w"]) == pytest.approx(g["ratio"], abs=5e-4)


def test_hysteresis_sequences_by_hand():
    g = golden()
    drop, c30, c10 = g["drop_w"], g["climb30_w"], g["climb10_w"]
    step = lambda i, p30, p10: O.hysteresis_step(i, 4, p30, p10, drop, c30, c10)
    assert step(2, 513, 400) == 1           # above the drop threshold: one level down
    assert step(0, 600, 600) == 0           # never below the lowest level
    assert step(1, 505, 520) == 2           # both climb conditions hold: one level up
    assert step(3, 505, 520) == 3           # never above the highest level
    assert step(1, 505, 530) == 1           # 10 s mean too high to climb
    assert step(1, 511, 500) == 1           # inside the dead band 510..512
    assert step(1, 512, 500) == 1           # "exceeds" is strict
    # a trace: rising power walks down, falling power walks back up
    idx, path = 3, []
    for p30, p10 in [(520, 530), (515, 514), (511, 505), (509, 520), (500, 500), (480, 490)]:
        idx = step(idx, p30, p10)
        path.append(idx)
    assert path == [2, 1, 1, 2, 3, 3]
