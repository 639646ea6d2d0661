"""Occupancy actuation on the rollout engine: the paper's live power-budget loop.

    python -m paper_2608_11226_amd.occupancy [--workload 7b] [--arm-seconds 60] [--calib-seconds 30]
        [--out occupancy.jsonl]

The actuator is generation concurrency: at every wave boundary the loop picks
the batch level b (whole prompt groups in flight, b in {1, 2, 4, 8}, so
b x G sequences) and runs one rollout wave at that level (section 4.5 and the
live study of section 6).  Device power is sampled every 0.5 s into an
occupancy monitor (``OccMonitor``: eq. (1) rolling means, eqs. (2)-(3) 30 s
violation rate and integrated excess, all in the library).  Arms:

  uncontrolled  static level 8
  static4       static level 4 (the paper's static safe baseline)
  hysteresis    the section 4.5 threshold rule (drop one level when the 30 s
                mean exceeds 512/561 of the budget; climb one when it is below
                510/561 and the 10 s mean below 525/561)

The budget follows eq. (8)'s rule: a calibration run at level 4 measures this
plant's batch-4 mean power P4, and B = P4 / 0.888, the paper's calibration
ratio of batch-4 power to budget (462 W / 520 W); --budget-w sets it instead
(a demand-response budget).  The learned PPO controller
is not part of this loop (its training environment is the paper's measured
transition bank).  Each arm prints one JSON line: tokens, tokens/s, 30 s
violation rate, integrated excess, Wh per 1k tokens, mean power and the
levels visited; with --out every telemetry sample is written as JSONL.
"""
from __future__ import annotations

import argparse
import json
import sys
import time

LEVELS = (1, 2, 4, 8)
CALIB_RATIO = 462.0 / 520.0      # batch-4 mean power / budget at calibration (eq. (8) keeps it)
DROP, CLIMB30, CLIMB10 = 512.0 / 561.0, 510.0 / 561.0, 525.0 / 561.0  # threshold rule, as fractions of the budget


class Static:
    def __init__(self, level: int):
        self.start_idx = LEVELS.index(level)

    def next(self, idx, reading, budget_w):
        return idx


class Hysteresis:
    """The section 4.5 threshold rule, thresholds scaled to the budget (the paper's watts at 561 W)."""

    def __init__(self, start_level: int = 4):
        self.start_idx = LEVELS.index(start_level)

    def next(self, idx, reading, budget_w):
        import paper_2608_11226_amd as R

        return R.occ_hysteresis_step(idx, len(LEVELS), reading.p30_w, reading.p10_w, DROP * budget_w,
                                     CLIMB30 * budget_w, CLIMB10 * budget_w)


def run_arm(name, run_wave, policy, seconds, attach, budget_w, dt=0.5, clock=time.perf_counter, log=None):
    """Run waves for ``seconds``; ``run_wave(level)`` blocks and returns its token count, ``attach(fn)`` routes
    power samples to fn (None detaches).  Returns the arm's record and the monitor's final reading."""
    import paper_2608_11226_amd as R

    mon = R.OccMonitor(dt, budget_w)
    attach(mon.push)
    t0 = clock()
    idx, tokens, waves = policy.start_idx, 0, []
    try:
        while clock() - t0 < seconds:
            level = LEVELS[idx]
            tw = clock()
            n = run_wave(level)
            d = clock() - tw
            tokens += n
            waves.append((level, d, n))
            r = mon.read()
            idx = policy.next(idx, r, budget_w)
            if log and len(waves) % 8 == 0:
                log(f"{name}: {clock() - t0:.0f} s, level {level}, P30 {r.p30_w:.0f} W, tokens {tokens}")
    finally:
        attach(None)
    elapsed = clock() - t0
    r = mon.read()
    mon.close()
    levels = {str(b): sum(1 for w in waves if w[0] == b) for b in LEVELS}
    rec = {"arm": name, "seconds": round(elapsed, 2), "waves": len(waves), "tokens": tokens,
           "tokens_per_s": round(tokens / elapsed, 1) if elapsed > 0 else None, "budget_w": round(budget_w, 1),
           "violation_rate_30s": round(r.violation_rate, 5), "integrated_excess_ws": round(r.excess_ws, 1),
           "peak_p30_w": round(r.peak30_w, 1), "samples": r.n, "levels": levels}
    return rec, r


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="7b", choices=["7b", "14b", "tiny"])
    ap.add_argument("--arm-seconds", type=float, default=60.0)
    ap.add_argument("--calib-seconds", type=float, default=30.0)
    ap.add_argument("--new-tokens", type=int, default=256)
    ap.add_argument("--arms", default="uncontrolled,static4,hysteresis")
    ap.add_argument("--budget-w", type=float, default=None,
                    help="explicit budget in watts (default: eq. (8) rule from the level-4 calibration)")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()

    import numpy as np
    import torch

    import paper_2608_11226_amd as R
    import workload as W
    from paper_2608_11226_amd.telemetry import PowerSampler, energy_joules

    def log(msg):
        print(f"[occupancy] {msg}", file=sys.stderr, flush=True)

    shape, P, G, dtype = {"7b": ("7b", 256, 8, R.DTYPE_BF16), "14b": ("14b", 512, 16, R.DTYPE_BF16),
                          "tiny": ("tiny", 16, 4, R.DTYPE_FP32)}[args.workload]
    N = args.new_tokens
    S_max = LEVELS[-1] * G
    eng = R.Engine(R.model_config(shape, dtype, P, N, S_max), group_size=G)
    V = eng.cfg.vocab
    dev = torch.device("cuda:0")
    prompts = torch.from_numpy(W.prompts(LEVELS[-1], P, V)).to(dev)
    uniforms = torch.from_numpy(W.uniforms(S_max, N)).to(dev)
    out = torch.empty((S_max, N), dtype=torch.int32, device=dev)

    def run_wave(level):
        R.rollout_generate(eng.ctx, prompts, level, P, G, level * G, N, 0.9, 0.95, uniforms, out)
        eng.synchronize()
        return level * G * N

    sampler = PowerSampler(0.5)
    if not sampler.ok:
        log("amd-smi power is not available: nothing to control")
        sys.exit(2)

    def attach(fn):
        sampler.listener = fn

    sampler.phase = "rollout"
    sampler.start()
    run_wave(4)  # warm-up (graph capture, clocks)
    # calibration at level 4 -> the plant's batch-4 mean power -> the budget (eq. (8) rule)
    t0 = time.perf_counter()
    calib, _ = run_arm("calibration", run_wave, Static(4), args.calib_seconds, attach, 1e9, log=log)
    t1 = time.perf_counter()
    e = energy_joules(sampler.samples, t0, t1)
    p4 = e / (t1 - t0)
    budget = args.budget_w if args.budget_w else R.occ_normalize_budget(520.0, p4, 462.0)
    log(f"calibration: batch-4 mean power {p4:.1f} W -> budget {budget:.1f} W"
        + (" (given)" if args.budget_w else " (eq. (8) rule)"))
    print(json.dumps({**calib, "mean_power_w": round(p4, 1), "budget_w": round(budget, 1)}), flush=True)
    policies = {"uncontrolled": Static(8), "static4": Static(4), "hysteresis": Hysteresis(4)}
    for name in args.arms.split(","):
        t0 = time.perf_counter()
        rec, _ = run_arm(name, run_wave, policies[name], args.arm_seconds, attach, budget, log=log)
        t1 = time.perf_counter()
        e = energy_joules(sampler.samples, t0, t1)
        rec["mean_power_w"] = round(e / (t1 - t0), 1)
        rec["wh_per_1k_tokens"] = round(e / 3600.0 / (rec["tokens"] / 1000.0), 5) if rec["tokens"] else None
        rec["power_field"] = sampler.field
        print(json.dumps(rec), flush=True)
    sampler.stop()
    if args.out:
        with open(args.out, "w") as f:
            for rec in sampler.records:
                f.write(json.dumps(rec) + "\n")
    eng.close()


if __name__ == "__main__":
    main()
