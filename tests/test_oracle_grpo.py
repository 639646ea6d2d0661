"""Pins of the oracle group-relative advantages: worked closed forms and invariants."""
import numpy as np
import pytest

from conftest import read_golden
from oracle.grpo import grpo_advantages


def test_worked_examples():
    for ddof, rewards, adv in read_golden("grpo_worked.txt"):
        r = np.array([float(x) for x in rewards.split(",")], dtype=np.float32)
        want = np.array([float(x) for x in adv.split(",")])
        got, zv = grpo_advantages(r, r.size, ddof=int(ddof))
        np.testing.assert_allclose(got, want, rtol=1e-6)
        assert zv == 0


@pytest.mark.parametrize("g", [2, 3, 4, 8, 16, 64, 100])
@pytest.mark.parametrize("ddof", [0, 1])
def test_zero_mean_unit_std(g, ddof):
    r = np.random.default_rng(g).uniform(0, 1, 40 * g).astype(np.float32)
    a, zv = grpo_advantages(r, g, ddof=ddof)
    a = a.reshape(-1, g).astype(np.float64)
    np.testing.assert_allclose(a.sum(1), 0, atol=1e-5)
    np.testing.assert_allclose(a.std(1, ddof=ddof), 1, rtol=1e-6)
    assert zv == 0


def test_equal_rewards_give_exact_zero():
    # 0.9 repeated: its float32 mean can differ from 0.9 by an ulp; the explicit
    # max == min test must still return exact zeros
    for g in (3, 6, 7, 12):
        a, zv = grpo_advantages(np.full(2 * g, 0.9, np.float32), g)
        assert np.all(a == 0) and zv == 2
    a, zv = grpo_advantages(np.array([0.1, 0.5, 0.5, 0.5], np.float32), 2)
    assert zv == 1 and np.all(a[2:] == 0) and a[0] < 0 < a[1]


def test_group_of_one_and_eps():
    a, zv = grpo_advantages(np.array([0.3, 0.7], np.float32), 1)
    assert np.all(a == 0) and zv == 2
    r = np.array([0.0, 1.0, 0.25, 0.5], np.float32)
    sig = np.std(r.astype(np.float64), ddof=1)
    a, _ = grpo_advantages(r, 4, eps=0.1)
    np.testing.assert_allclose(np.std(a.astype(np.float64), ddof=1), sig / (sig + 0.1), rtol=1e-6)


def test_rejects_partial_groups():
    with pytest.raises(ValueError):
        grpo_advantages(np.zeros(5, np.float32), 2)
