"""Pins of the seeded input generator (the counter-based SplitMix64 hash)."""
import numpy as np

import workload as W
from conftest import read_golden


def test_splitmix64_known_answers():
    want = [int(r[0], 16) for r in read_golden("splitmix64_seed0.txt")]
    # stream 0 under seed 0 is the sequential generator
    got_int = [W.hash_int(0, 0, i) for i in range(len(want))]
    got_np = [int(v) for v in W.hash_range(0, 0, 0, len(want))]
    assert got_int == want
    assert got_np == want


def test_vectorised_matches_integer_reference():
    for seed, stream in [(0, 5), (7, 0x100000), (2**63 + 3, 12345)]:
        idx = np.array([0, 1, 2, 1000, 2**31 + 7, 2**40 + 1], dtype=np.uint64)
        got = W.hash_indices(seed, stream, idx)
        want = [W.hash_int(seed, stream, int(i)) for i in idx]
        assert [int(g) for g in got] == want
        rng = W.hash_range(seed, stream, 1000, 3)
        assert [int(v) for v in rng] == [W.hash_int(seed, stream, i) for i in (1000, 1001, 1002)]


def test_weight_distribution_moments():
    n = 1 << 21
    w = W.weight_values(0, 7, 0, n, std=0.02).astype(np.float64)
    # Irwin-Hall(4) of uniform 16-bit limbs, centred and scaled: variance
    # std^2 * (1 - 2^-32); support +-sqrt(3) * 2 * std
    se = 0.02 / np.sqrt(n)
    assert abs(w.mean()) < 4 * se
    assert abs(w.std() - 0.02) < 4 * 0.02 / np.sqrt(2 * n) * 1.5
    assert np.abs(w).max() <= 0.02 * 2 * np.sqrt(3) + 1e-9
    # the chunked and threaded paths agree with element access
    idx = np.array([0, 5, n - 1, 123457])
    assert np.array_equal(W.weight_elements(0, 7, idx), w[idx].astype(np.float32))


def test_weight_extreme_limbs():
    # all four limbs 0xFFFF -> s = 262140 -> (131070/65536)*sqrt(3)*std; all zero -> the negative
    v = np.array([0xFFFFFFFFFFFFFFFF, 0], dtype=np.uint64)
    w = W._weight_from_hash(v, 0.02)
    top = np.float32((131070 / 65536.0) * 1.7320508075688772 * 0.02)
    assert w[0] == top and w[1] == -top


def test_rows_and_matrix_agree():
    m = W.weight_matrix(0, 3, 16, 40)
    r = W.weight_rows(0, 3, [2, 15, 0], 40)
    assert np.array_equal(r, m[[2, 15, 0]])


def test_prompts_uniforms_rewards_ranges():
    p = W.prompts(4, 300, 1024)
    assert p.dtype == np.int32 and p.shape == (4, 300)
    assert p.min() >= 0 and p.max() < 1024
    # roughly uniform over the vocabulary
    counts = np.bincount(p.ravel(), minlength=1024)
    assert counts.max() < 12
    u = W.uniforms(8, 16)
    assert u.dtype == np.float32 and u.min() >= 0.0 and u.max() < 1.0
    assert np.all(np.floor(u.astype(np.float64) * 2**24) == u.astype(np.float64) * 2**24)
    # waves: offsetting the first completion index continues the same stream
    assert np.array_equal(W.uniforms(4, 16, first_seq=4), u[4:])
    r = W.rewards(64)
    assert r.min() >= 0 and r.max() < 1 and np.array_equal(W.rewards(32, first=32), r[32:])
