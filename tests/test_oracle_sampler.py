"""Pins of the oracle sampler: greedy limit, brute force over the uniform grid, kept-set properties."""
import numpy as np
from scipy.special import softmax

from oracle import sampler as S


def test_greedy_lowest_id_on_ties():
    z = np.array([0.1, 3.0, -2.0, 3.0, 1.0], dtype=np.float32)
    tok, gap = S.sample_row(z, 0.0, 1.0, 0.7)
    assert tok == 1 and gap == 0.0
    z[3] = 2.5
    assert S.sample_row(z, 0.0, 0.3, 0.1) == (1, 0.5)


def test_low_temperature_limit_is_argmax():
    rng = np.random.default_rng(0)
    for _ in range(20):
        z = rng.standard_normal(50).astype(np.float32)
        for u in (0.0, 0.5, 0.999999):
            assert S.sample_row(z, 1e-4, 1.0, u)[0] == int(np.argmax(z))


def _grid_counts(z, temperature, top_p, bits=14):
    n = 1 << bits
    counts = np.zeros(z.size, dtype=np.int64)
    for k in range(n):
        counts[S.sample_row(z, temperature, top_p, k / n)[0]] += 1
    return counts


def test_brute_force_grid_reproduces_softmax():
    z = np.array([0.3, -1.2, 2.0, 0.0, 0.7, -0.4, 1.1, 0.05], dtype=np.float32)
    for temperature in (1.0, 0.7):
        counts = _grid_counts(z, temperature, 1.0)
        p = softmax(z.astype(np.float64) / temperature)
        # each token owns a CDF interval of width p_i: its share of 2^14 grid points is within one
        assert np.all(np.abs(counts - p * (1 << 14)) <= 1.0)


def test_cdf_runs_in_ascending_token_id():
    z = np.array([0.0, 5.0, 0.0, 1.0], dtype=np.float32)
    assert S.sample_row(z, 1.0, 1.0, 0.0)[0] == 0  # smallest id first
    assert S.sample_row(z, 1.0, 1.0, 1.0 - 2**-24)[0] == 3  # largest id last


def test_top_p_kept_set_properties_and_draws():
    rng = np.random.default_rng(1)
    for trial in range(200):
        v = int(rng.integers(2, 12))
        z = np.round(rng.standard_normal(v), 1).astype(np.float32)  # rounding makes ties common
        top_p = float(rng.uniform(0.05, 0.99))
        e = S.decision_values(z, 1.0).astype(np.float64)
        keep, _ = S.kept_set(e.astype(np.float32), top_p)
        total = e.sum()
        kept = np.nonzero(keep)[0]
        assert e[kept].sum() >= top_p * total * (1 - 1e-12)
        # no outside token beats a kept one; among equal values lower ids are kept first
        lo = e[kept].min()
        assert np.all(e[~keep] <= lo)
        tied_out = np.nonzero((~keep) & (e == lo))[0]
        if tied_out.size:
            assert tied_out.min() > kept[e[kept] == lo].max()
        # minimal: dropping the last-ranked kept token falls short of the target
        last = kept[e[kept] == lo].max()
        assert e[kept].sum() - e[last] < top_p * total
    # draws only ever return kept tokens, in proportion to their renormalised mass
    z = np.array([2.0, 1.0, 0.5, 0.0, -1.0, 1.0], dtype=np.float32)
    e = S.decision_values(z, 1.0).astype(np.float64)
    keep, _ = S.kept_set(e.astype(np.float32), 0.7)
    counts = _grid_counts(z, 1.0, 0.7, bits=13)
    assert np.all(counts[~keep] == 0)
    p = np.where(keep, e, 0) / e[keep].sum()
    assert np.all(np.abs(counts - p * (1 << 13)) <= 1.0)


def test_tiny_top_p_returns_the_mode():
    rng = np.random.default_rng(2)
    z = rng.standard_normal(100).astype(np.float32)
    for u in (0.0, 0.3, 0.99):
        assert S.sample_row(z, 0.8, 1e-9, u)[0] == int(np.argmax(z))


def test_margin_reports_near_edges():
    z = np.zeros(4, dtype=np.float32)  # four equal tokens: CDF edges at 0.25, 0.5, 0.75
    assert S.sample_row(z, 1.0, 1.0, 0.5)[1] < 1e-12
    tok, m = S.sample_row(z, 1.0, 1.0, 0.375)
    assert tok == 1 and abs(m - 0.125) < 1e-12
