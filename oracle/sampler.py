"""Oracle sampler: temperature, nucleus (top-p) truncation, inverse-CDF draw.

TEST INFRASTRUCTURE ONLY (see the package header).

The paper samples G completions per prompt (section 3, "Background") but
names no sampler; temperature and top-p are the workload's knobs.  The
definition taken here, per row of logits z (length V), temperature T >= 0,
top_p in (0, 1] and one uniform u in [0, 1):

* T == 0: greedy, the arg max of z, lowest token id among equal maxima.
* Otherwise the decision values are fp32: y = fp32(z / T), m = max y,
  e_i = fp32 exp(y_i - m), S = sum(e) accumulated exactly (float64).
* top_p < 1: order tokens by (e descending, id ascending) and keep the
  shortest prefix whose mass reaches top_p * S (the crossing token is kept,
  at least one token).  top_p >= 1 keeps every token.
* Draw: walk the kept tokens in ascending id, accumulating c; return the
  first id with c > u * S_kept; if rounding leaves none, the largest kept id.

Where floating point decides the token, the decision is taken on the fp32
values e_i, which is the precision the GPU kernel uses; the logits feeding it
are the oracle's own.  Each draw also reports a margin: how close the decision
came to flipping (relative to the mass involved), so a comparison can tell a
legitimate near-tie from a real mismatch.

Parity: pinned by brute force on tiny vocabularies (every kept id is drawn
for exactly the fraction of the 2**-24 uniform grid its probability predicts),
the greedy limit, and a full-sort check of the kept set in
``tests/test_oracle_sampler.py``.
"""
from __future__ import annotations

import numpy as np


def _greedy(z: np.ndarray) -> tuple[int, float]:
    z = np.asarray(z, dtype=np.float32)
    tok = int(np.argmax(z))  # numpy returns the first (lowest-id) maximum
    if z.size > 1:
        top2 = np.partition(z.astype(np.float64), -2)[-2:]
        gap = float(top2[1] - top2[0])
    else:
        gap = np.inf
    return tok, gap


def decision_values(z: np.ndarray, temperature: float) -> np.ndarray:
    """e_i = fp32 exp(fp32(z_i / T) - max): the fp32 values the draw is decided on."""
    y = (np.asarray(z, dtype=np.float32) / np.float32(temperature)).astype(np.float32)
    return np.exp(y - y.max()).astype(np.float32)


def _kept(e: np.ndarray, top_p: float):
    """(nucleus mask, top-p margin relative to S, the kept set the nearest flip would give)."""
    e64 = e.astype(np.float64)
    total = e64.sum()
    if top_p >= 1.0:
        return np.ones(e.size, dtype=bool), np.inf, None
    order = np.lexsort((np.arange(e.size), -e64))  # e descending, then id ascending
    cum = np.cumsum(e64[order])
    target = top_p * total
    k = int(np.searchsorted(cum, target, side="left"))  # first prefix with cum >= target
    k = min(k, e.size - 1)
    keep = np.zeros(e.size, dtype=bool)
    keep[order[: k + 1]] = True
    before = cum[k - 1] if k > 0 else 0.0
    over, under = abs(cum[k] - target), abs(target - before)
    alt = keep.copy()
    if over <= under and k + 1 < e.size:
        alt[order[k + 1]] = True  # the crossing prefix judged one token short
    elif k > 0:
        alt[order[k]] = False  # the prefix before the crossing judged long enough
    return keep, float(min(over, under) / total), alt


def kept_set(e: np.ndarray, top_p: float) -> tuple[np.ndarray, float]:
    """Boolean mask of the nucleus and the top-p margin (relative to S)."""
    keep, margin, _ = _kept(e, top_p)
    return keep, margin


def _draw(e: np.ndarray, keep: np.ndarray, u: float) -> tuple[int, float]:
    """Inverse-CDF draw over the kept ids in ascending order; (token, CDF-edge margin)."""
    ids = np.nonzero(keep)[0]  # ascending id
    w = e[ids].astype(np.float64)
    mass = w.sum()
    c = np.cumsum(w)
    thresh = float(u) * mass
    j = int(np.searchsorted(c, thresh, side="right"))  # first c > thresh
    if j >= ids.size:
        j = ids.size - 1
    lo = c[j - 1] if j > 0 else 0.0
    return int(ids[j]), float(min(abs(c[j] - thresh), abs(thresh - lo)) / mass)


def sample_row(z, temperature: float, top_p: float, u: float) -> tuple[int, float]:
    """Return (token id, margin) for one row of logits.

    margin is the top-2 logit gap for greedy rows, otherwise the smallest
    relative distance of the decision from flipping: the CDF edges around the
    draw and, when flipping the top-p crossing would change the drawn token,
    the top-p crossing itself.
    """
    if temperature == 0.0:
        return _greedy(z)
    e = decision_values(z, temperature)
    keep, m_top, alt = _kept(e, top_p)
    tok, m_cdf = _draw(e, keep, u)
    if alt is None or not alt.any():
        return tok, min(m_top, m_cdf)
    tok_alt, m_alt = _draw(e, alt, u)
    if tok_alt == tok:  # either reading of the crossing draws the same token
        return tok, min(m_cdf, m_alt)
    return tok, min(m_top, m_cdf)


def sample_batch(logits: np.ndarray, temperature: float, top_p: float, u: np.ndarray):
    """Rows of logits [S, V] with uniforms u [S]: (tokens int32 [S], margins float64 [S])."""
    logits = np.asarray(logits)
    toks = np.empty(logits.shape[0], dtype=np.int32)
    margins = np.empty(logits.shape[0], dtype=np.float64)
    for s in range(logits.shape[0]):
        toks[s], margins[s] = sample_row(logits[s], temperature, top_p, float(u[s]))
    return toks, margins
