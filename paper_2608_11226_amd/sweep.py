"""Actuator sweep on the 7B-class rollout: power authority of group size and of concurrency.

    python -m paper_2608_11226_amd.sweep [--seconds 12] [--out sweep_7b.jsonl]

The paper's actuator-authority study (section 6.4, Table 4) varies one knob at
a time and reports the mean-power swing, the 30 s peak swing and the
throughput ratio across its range.  The same two concurrency knobs on this
engine, at a fixed total of 65,536 generated tokens per point (256 completions
of 256 new tokens after 256-token prompts, T = 0.9, top-p 0.95):

* arm "group": G in {4, 8, 16, 32} with 8 prompts per wave, so S = 8 G
  sequences in flight and 256 / S waves;
* arm "concurrency": S in {16, 32, 64, 128, 256} sequences in flight at G = 8
  (32 prompts, 256 / S waves).

Each point repeats its rollout until ``--seconds`` have passed while amd-smi
socket power is sampled every 0.5 s, and reports tokens/s, mean power, J per
token, the 30 s rolling-mean peak (eq. (1), over the point's own samples) and
the decode projections' HBM roofline fraction from HIP events around each
launch of one instrumented decode step at mid-completion context.  Per arm it
adds the paper's three authority figures.  Inputs are the seeded synthetic
workload (random-init weights, uniform prompt tokens).
"""
from __future__ import annotations

import argparse
import json
import sys
import time

HBM_PEAK_GBS = 8000.0
TOTAL_COMPLETIONS = 256
P = 256
N = 256


def points():
    for G in (4, 8, 16, 32):
        yield "group", G, 8 * G
    for S in (16, 32, 64, 128, 256):
        yield "concurrency", 8, S


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--seconds", type=float, default=12.0)
    ap.add_argument("--out", default=None)
    args = ap.parse_args()

    import numpy as np
    import torch

    import paper_2608_11226_amd as R
    import workload as W
    from paper_2608_11226_amd.telemetry import PowerSampler, energy_joules

    def log(msg):
        print(f"[sweep] {msg}", file=sys.stderr, flush=True)

    dev = torch.device("cuda:0")
    eng = R.Engine(R.model_config("7b", R.DTYPE_BF16, P, N, 256), group_size=4)
    V = eng.cfg.vocab
    prompts = torch.from_numpy(W.prompts(TOTAL_COMPLETIONS // 4, P, V)).to(dev)
    uniforms = torch.from_numpy(W.uniforms(TOTAL_COMPLETIONS, N)).to(dev)
    out = torch.empty((TOTAL_COMPLETIONS, N), dtype=torch.int32, device=dev)
    logits = torch.empty((256, V), dtype=torch.float32, device=dev)
    sampler = PowerSampler(0.5)
    if not sampler.ok:
        log("amd-smi power is not available")
    recs = []
    sampler.start()
    for arm, G, S in points():
        n_prompts = TOTAL_COMPLETIONS // G

        def rollout():
            R.rollout_generate(eng.ctx, prompts, n_prompts, P, G, S, N, 0.9, 0.95, uniforms, out)
            eng.synchronize()

        rollout()  # warm-up: graph capture, clocks
        sampler.phase = f"{arm} G={G} S={S}"
        t0 = time.perf_counter()
        n = 0
        while True:
            rollout()
            n += 1
            if time.perf_counter() - t0 >= args.seconds:
                break
        t1 = time.perf_counter()
        tokens = n * TOTAL_COMPLETIONS * N
        rec = {"arm": arm, "G": G, "seqs_in_flight": S, "waves": TOTAL_COMPLETIONS // S, "rollouts": n,
               "seconds": round(t1 - t0, 2), "tokens_per_s": round(tokens / (t1 - t0), 1)}
        win = [(t, p) for t, p in sampler.samples if t0 <= t <= t1]
        if win:
            e = energy_joules(sampler.samples, t0, t1)
            p = np.array([w for _, w in win])
            m30 = R.occ_rolling_mean(p, 0.5, 30.0)
            rec.update({"mean_power_w": round(e / (t1 - t0), 1), "j_per_token": round(e / tokens, 5),
                        "peak30_w": round(float(m30.max()), 1), "samples": len(win)})
        # instrumented decode step of one wave at mid-completion context
        R.rollout_prefill(eng.ctx, prompts, S // G, P, G, logits)
        for t in range(N // 2):
            R.rollout_decode_step(eng.ctx, out[:S, t].contiguous(), logits)
        prof = R.rollout_profile_decode_step(eng.ctx, out[:S, N // 2].contiguous(), logits)
        eng.synchronize()
        gbs = prof.bytes[0] / (prof.ms[0] * 1e-3) / 1e9
        rec.update({"gemm_gbs": round(gbs, 1), "gemm_hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                    "attention_gbs": round(prof.bytes[1] / (prof.ms[1] * 1e-3) / 1e9, 1),
                    "step_ms": round(sum(prof.ms), 3)})
        log(json.dumps(rec))
        print(json.dumps(rec), flush=True)
        recs.append(rec)
    sampler.stop()
    for arm in ("group", "concurrency"):
        rs = [r for r in recs if r["arm"] == arm]
        tps = [r["tokens_per_s"] for r in rs]
        summary = {"arm": arm, "summary": True, "throughput_ratio": round(max(tps) / min(tps), 3)}
        if all("mean_power_w" in r for r in rs):
            pw = [r["mean_power_w"] for r in rs]
            pk = [r["peak30_w"] for r in rs]
            summary.update({"mean_power_swing": round(max(pw) / min(pw) - 1, 4),
                            "peak30_swing": round(max(pk) / min(pk) - 1, 4)})
        print(json.dumps(summary), flush=True)
        recs.append(summary)
    if args.out:
        with open(args.out, "w") as f:
            for r in recs:
                f.write(json.dumps(r) + "\n")
            for r in sampler.records:
                f.write(json.dumps(r) + "\n")
    eng.close()


if __name__ == "__main__":
    main()
