"""Shared helpers of the GPU parity tests (inputs come from the seeded workload;
expected values come from the oracle only)."""
import sys

import numpy as np

import workload as W


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(arr, torch, device="cuda:0"):
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def shape_of(cfg):
    return W.ModelShape(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff, cfg.vocab,
                        cfg.rms_eps, cfg.rope_theta)


def guarded_token_compare(gpu_tokens, oracle_tokens, oracle_margins, guard=1e-5):
    """Compare free-running token streams sequence by sequence.

    Tokens must agree up to and including the first draw whose oracle margin is
    below ``guard`` (a legitimate near-tie); a mismatch exactly at that draw is
    allowed and later draws are not compared.  Returns (compared, skipped).
    """
    compared = skipped = 0
    for s in range(oracle_tokens.shape[0]):
        for t in range(oracle_tokens.shape[1]):
            near_tie = oracle_margins[s, t] < guard
            if gpu_tokens[s, t] != oracle_tokens[s, t]:
                assert near_tie, f"sequence {s} step {t}: gpu {gpu_tokens[s, t]} oracle {oracle_tokens[s, t]} " \
                                 f"(margin {oracle_margins[s, t]:.3g})"
                skipped += oracle_tokens.shape[1] - t
                break
            compared += 1
            if near_tie:
                skipped += oracle_tokens.shape[1] - t - 1
                break
    return compared, skipped
