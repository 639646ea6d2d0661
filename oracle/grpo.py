"""Oracle group-relative advantages.

TEST INFRASTRUCTURE ONLY (see the package header).

Section 3 ("Background") of the paper: each candidate's advantage is its
reward compared against the mean of its own group of G; GRPO normalises by the
group's standard deviation as well.  Definition used here, per group of G
rewards r (fp32 in, float64 arithmetic, fp32 out):

* G == 1, or max r == min r (tested exactly, not through a computed
  standard deviation): every advantage is 0 and the group counts as
  zero-variance (the zero-variance-group statistic of section 4.2).
* Otherwise mu = mean r, sigma = sqrt(sum (r - mu)^2 / (G - ddof)),
  A = (r - mu) / (sigma + eps).

Defaults ddof = 1, eps = 0.  Parity: pinned by closed forms (sum A = 0,
sample std 1, G = 2 gives +-1/sqrt(2) for ddof 1 and +-1 for ddof 0, equal
rewards give exactly 0) in ``tests/test_oracle_grpo.py``.
"""
from __future__ import annotations

import numpy as np


def grpo_advantages(rewards, group_size: int, eps: float = 0.0, ddof: int = 1):
    """Return (advantages fp32 [n], zero-variance group count)."""
    r = np.asarray(rewards, dtype=np.float32).astype(np.float64)
    if group_size < 1 or r.size % group_size:
        raise ValueError("rewards must hold whole groups")
    if ddof not in (0, 1):
        raise ValueError("ddof must be 0 or 1")
    groups = r.reshape(-1, group_size)
    out = np.zeros_like(groups)
    zero_var = 0
    for g in range(groups.shape[0]):
        x = groups[g]
        if group_size == 1 or x.max() == x.min():
            zero_var += 1
            continue
        mu = x.sum() / group_size
        sigma = np.sqrt(np.sum((x - mu) ** 2) / (group_size - ddof))
        out[g] = (x - mu) / (sigma + eps)
    return out.reshape(-1).astype(np.float32), zero_var
