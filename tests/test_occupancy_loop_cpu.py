"""The occupancy loop's logic on a simulated plant (no GPU): a power model per batch level, a fake clock."""
import pytest

import paper_2608_11226_amd as R
from paper_2608_11226_amd import occupancy as OC
from oracle import power as O


class Plant:
    """Waves of fixed duration whose power depends on the level; samples every dt into the attached monitor."""

    def __init__(self, watts, wave_s=2.0, dt=0.5):
        self.watts, self.wave_s, self.dt = watts, wave_s, dt
        self.t, self.fn, self.trace = 0.0, None, []

    def clock(self):
        return self.t

    def attach(self, fn):
        self.fn = fn

    def run_wave(self, level):
        for _ in range(int(round(self.wave_s / self.dt))):
            self.t += self.dt
            p = self.watts[level]
            self.trace.append(p)
            if self.fn:
                self.fn(p)
        return level * 8 * 100


def test_static_arms_and_metrics_match_the_oracle():
    plant = Plant({1: 400.0, 2: 450.0, 4: 500.0, 8: 600.0})
    rec, r = OC.run_arm("uncontrolled", plant.run_wave, OC.Static(8), 60.0, plant.attach, 560.0, clock=plant.clock)
    assert rec["levels"] == {"1": 0, "2": 0, "4": 0, "8": 30}
    p30 = O.rolling_mean(plant.trace, 0.5, 30.0)
    assert rec["violation_rate_30s"] == pytest.approx(O.violation_rate(p30, 560.0), abs=1e-5)
    assert r.excess_ws == pytest.approx(O.integrated_excess(p30, 560.0, 0.5), rel=1e-9)
    assert rec["tokens"] == 30 * 8 * 8 * 100


def test_hysteresis_holds_the_budget_where_level_8_breaks_it():
    # level 8 draws above the budget, level 4 well below: the rule must oscillate between them and keep
    # the 30 s mean near the drop threshold, while the uncontrolled arm violates on most samples
    watts = {1: 300.0, 2: 380.0, 4: 480.0, 8: 620.0}
    budget = 561.0
    hy = Plant(watts)
    rec_h, _ = OC.run_arm("hysteresis", hy.run_wave, OC.Hysteresis(4), 600.0, hy.attach, budget, clock=hy.clock)
    un = Plant(watts)
    rec_u, _ = OC.run_arm("uncontrolled", un.run_wave, OC.Static(8), 600.0, un.attach, budget, clock=un.clock)
    assert rec_u["violation_rate_30s"] > 0.8
    assert rec_h["violation_rate_30s"] < 0.1
    assert rec_h["levels"]["8"] > 0 and rec_h["levels"]["4"] > 0
    st = Plant(watts)
    rec_s, _ = OC.run_arm("static4", st.run_wave, OC.Static(4), 600.0, st.attach, budget, clock=st.clock)
    assert rec_s["violation_rate_30s"] == 0.0
    assert rec_h["tokens"] > rec_s["tokens"]  # the rule spends headroom at level 8
    # its level decisions are exactly the threshold rule applied to the oracle's means at each boundary
    p = Plant(watts)
    idx, decisions = OC.LEVELS.index(4), []
    for _ in range(40):
        p.run_wave(OC.LEVELS[idx])
        p10 = O.rolling_mean(p.trace, 0.5, 10.0)[-1]
        p30 = O.rolling_mean(p.trace, 0.5, 30.0)[-1]
        idx = O.hysteresis_step(idx, 4, p30, p10, OC.DROP * budget, OC.CLIMB30 * budget, OC.CLIMB10 * budget)
        decisions.append(idx)
    q = Plant(watts)
    seen = []

    class Spy(OC.Hysteresis):
        def next(self, idx, reading, budget_w):
            n = super().next(idx, reading, budget_w)
            seen.append(n)
            return n

    OC.run_arm("hysteresis", q.run_wave, Spy(4), 80.0, q.attach, budget, clock=q.clock)
    assert seen == decisions


def test_budget_rule_reproduces_the_paper_ratio():
    assert OC.CALIB_RATIO == pytest.approx(0.888, abs=5e-4)
    assert R.occ_normalize_budget(520.0, 498.4, 462.0) == pytest.approx(561.0, abs=0.1)
