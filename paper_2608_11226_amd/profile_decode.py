"""Short driver for hardware-counter runs of the decode step.

    rocprofv3 --pmc FETCH_SIZE --kernel-trace --output-format csv -d DIR -o run -- \
        python3 -m paper_2608_11226_amd.profile_decode [--workload 7b] [--steps 3]

Builds the workload's engine, prefills its prompts, runs a few decode steps
eagerly (the same kernels and launch shapes the rollout replays), then
copies a buffer of known size with a plain device copy so that byte counters
can be calibrated: that copy reads and writes exactly COPY_BYTES.
"""
from __future__ import annotations

import argparse
import sys

import numpy as np

COPY_BYTES = 1 << 30

# shape name, prompts, prompt length, G, sequences in flight, new tokens, int4 layer projections
WORKLOADS = {
    "7b": ("7b", 8, 256, 8, 64, 512, False),
    "14b": ("14b", 16, 512, 16, 256, 1024, False),
    "72b": ("72b", 8, 512, 8, 64, 512, False),
    "72b-int4": ("72b", 8, 512, 8, 64, 512, True),
}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="7b", choices=sorted(WORKLOADS))
    ap.add_argument("--steps", type=int, default=3)
    args = ap.parse_args()

    import torch

    import paper_2608_11226_amd as R
    import workload as W

    shape, n_prompts, P, G, S, N, q4 = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    eng = R.Engine(R.model_config(shape, R.DTYPE_INT4 if q4 else R.DTYPE_BF16, P, N, S), group_size=G)
    V = R.SHAPES[shape][6]
    prompts = torch.from_numpy(W.prompts(n_prompts, P, V)).to(dev)
    logits = torch.empty((S, V), dtype=torch.float32, device=dev)
    R.rollout_prefill(eng.ctx, prompts, n_prompts, P, G, logits)
    tok = torch.from_numpy(np.zeros(S, dtype=np.int32)).to(dev)
    for _ in range(args.steps):
        R.rollout_decode_step(eng.ctx, tok, logits)
    eng.synchronize()
    print(f"[profile_decode] {args.steps} decode steps of {S} sequences done", file=sys.stderr, flush=True)
    a = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    print(f"[profile_decode] calibration copy of {COPY_BYTES} bytes done", file=sys.stderr, flush=True)
    eng.close()


if __name__ == "__main__":
    main()
