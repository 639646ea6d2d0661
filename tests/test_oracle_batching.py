"""Pins of the stop-token / continuous-batching oracle (oracle/batching.py)."""
import numpy as np
import pytest

import workload as W
from conftest import read_golden
from oracle import OracleModel, rollout
from oracle.batching import (PAD, continuous_schedule, length_target_reward, rollout_eos, sequence_schedule,
                             simulate_sequence_slots, simulate_slots)


def _ints(s):
    return [int(v) for v in s.split(",")]


def test_schedule_matches_hand_worked_cases():
    rows = read_golden("batching_schedule.txt")
    assert len(rows) == 5
    for G, ranges, R, lengths, admit, free, steps in rows:
        for fn in (continuous_schedule, simulate_slots):
            got = fn(_ints(lengths), int(G), int(ranges), int(R))
            assert list(got["admit"]) == _ints(admit), (fn.__name__, lengths)
            assert list(got["free"]) == _ints(free), (fn.__name__, lengths)
            assert got["steps"] == int(steps), (fn.__name__, lengths)


def test_schedule_event_form_equals_step_simulation():
    rng = np.random.default_rng(7)
    for _ in range(300):
        G = int(rng.choice([1, 2, 3, 4]))
        n_groups = int(rng.integers(1, 9))
        ranges = int(rng.integers(1, 6))
        R = int(rng.choice([1, 2, 3, 8]))
        lengths = rng.integers(1, 40, size=n_groups * G)
        a = continuous_schedule(lengths, G, ranges, R)
        b = simulate_slots(lengths, G, ranges, R)
        assert np.array_equal(a["admit"], b["admit"]) and np.array_equal(a["free"], b["free"])
        assert a["steps"] == b["steps"]


def test_schedule_invariants():
    rng = np.random.default_rng(8)
    lengths = rng.integers(1, 30, size=6 * 4)
    # every group fits at once: all admitted at step 0, the rollout lasts as long as the longest group
    s = continuous_schedule(lengths, 4, 6, 1)
    assert np.all(s["admit"] == 0)
    assert s["steps"] == max(1, int(lengths.max()) - 1)
    # one range and R = 1: groups run back to back
    s = continuous_schedule(lengths, 4, 1, 1)
    spans = np.maximum(1, lengths.reshape(6, 4).max(axis=1) - 1)
    assert list(s["admit"]) == [0] + list(np.cumsum(spans)[:-1])
    # admissions follow prompt order and never precede the range's previous group ending
    s = continuous_schedule(lengths, 4, 2, 3)
    assert np.all(np.diff(s["admit"]) >= 0)
    assert np.all(s["admit"] % 3 == 0) and np.all(s["free"] % 3 == 0)


def _tiny_plain(temperature, top_p, N=16):
    model = OracleModel(W.TINY, mode="fp32")
    prompts = W.prompts(2, 12, W.TINY.vocab, seed=5)
    u = W.uniforms(8, N, seed=6)
    plain = rollout(model, prompts, 4, N, temperature, top_p, u, keep_logits=False)
    return model, prompts, u, plain


@pytest.mark.parametrize("temperature,top_p", [(1.0, 1.0), (0.8, 0.9), (0.0, 1.0)])
def test_rollout_eos_is_plain_rollout_truncated_at_first_stop(temperature, top_p):
    N = 16
    model, prompts, u, plain = _tiny_plain(temperature, top_p, N)
    pt = plain["tokens"]
    stop = sorted({int(pt[0, 3]), int(pt[5, 0]), int(pt[6, 9])})
    got = rollout_eos(model, prompts, 4, N, temperature, top_p, u, stop)
    for s in range(8):
        hits = [t for t in range(N) if pt[s, t] in stop]
        L = hits[0] + 1 if hits else N
        assert got["lengths"][s] == L
        assert np.array_equal(got["tokens"][s, :L], pt[s, :L])
        assert np.all(got["tokens"][s, L:] == PAD)
    assert got["lengths"][0] <= 4 and got["lengths"][5] == 1


def test_rollout_eos_empty_and_full_stop_sets():
    N = 10
    model, prompts, u, plain = _tiny_plain(1.0, 1.0, N)
    none = rollout_eos(model, prompts, 4, N, 1.0, 1.0, u, [])
    assert np.all(none["lengths"] == N) and np.array_equal(none["tokens"], plain["tokens"])
    full = rollout_eos(model, prompts, 4, N, 1.0, 1.0, u, np.arange(W.TINY.vocab))
    assert np.all(full["lengths"] == 1)
    assert np.array_equal(full["tokens"][:, 0], plain["tokens"][:, 0]) and np.all(full["tokens"][:, 1:] == PAD)


def test_length_target_reward_closed_form():
    L = np.array([128, 64, 192, 256, 1, 1000, 0])
    want = np.array([1.0, 0.5, 0.5, 0.0, 1.0 / 128.0, 0.0, 0.0])
    assert np.allclose(length_target_reward(L, 128), want, rtol=0, atol=1e-15)
    assert length_target_reward([10], 10)[0] == 1.0 and length_target_reward([15], 10)[0] == 0.5


def test_single_completion_schedule_equals_simulation():
    rng = np.random.default_rng(9)
    for _ in range(200):
        G = int(rng.choice([1, 2, 4, 8]))
        n = G * int(rng.integers(1, 7))
        slots = int(rng.integers(1, 12))
        R = int(rng.choice([1, 2, 5]))
        lengths = rng.integers(1, 30, size=n)
        a = sequence_schedule(lengths, slots, R)
        b = simulate_sequence_slots(lengths, G, slots, R)
        assert np.array_equal(a["admit"], b["admit"]) and np.array_equal(a["free"], b["free"])
        assert a["steps"] == b["steps"]
        # a live prompt record per group with a completion in a slot, plus one being admitted
        assert b["most_records"] <= min(slots, n) + 1


def test_single_completion_schedule_hand_worked():
    # slots 2, R 1, lengths 3,1,2,2: s0 -> slot 0 (ends step 2), s1 -> slot 1 (ends at 0, seen at 1)
    # step 1: slot 1 -> s2 (ends 1 + 1 = 2); step 2: slot 0 -> s3 (ends 3), slot 1 seen free (s2); step 3: s3 seen
    got = sequence_schedule([3, 1, 2, 2], 2, 1)
    assert list(got["admit"]) == [0, 0, 1, 2] and list(got["free"]) == [2, 1, 2, 3] and got["steps"] == 3
    # fewer decode steps than refilling whole groups of 2 over the same slots
    assert continuous_schedule([3, 1, 2, 2], 2, 1, 1)["steps"] == 3
    assert sequence_schedule([5, 1, 1, 5, 1, 1], 2, 1)["steps"] < continuous_schedule([5, 1, 1, 5, 1, 1], 2, 1, 1)["steps"]
