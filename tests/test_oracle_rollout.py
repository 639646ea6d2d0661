"""Oracle rollout on the tiny fp32 configuration: cached rollout against brute-force recompute."""
import numpy as np
import pytest

import workload as W
from oracle import OracleModel, rollout


@pytest.fixture(scope="module")
def tiny_run():
    model = OracleModel(W.TINY, mode="fp32")
    prompts = W.prompts(2, 16, W.TINY.vocab)
    u = W.uniforms(8, 16)
    r = W.rewards(8)
    out = rollout(model, prompts, 4, 16, 1.0, 1.0, u, rewards=r)
    return model, prompts, u, out


def test_shapes_and_ranges(tiny_run):
    _, _, _, out = tiny_run
    assert out["tokens"].shape == (8, 16) and out["logits"].shape == (16, 8, 1024)
    assert out["tokens"].min() >= 0 and out["tokens"].max() < 1024
    assert out["advantages"].shape == (8,)


def test_every_step_equals_full_recompute(tiny_run):
    model, prompts, _, out = tiny_run
    for s in (0, 5, 7):
        seq = np.concatenate([prompts[s // 4], out["tokens"][s, :-1]])
        full = model.forward_full(seq)
        np.testing.assert_allclose(out["logits"][:, s, :], full[15:], atol=1e-10, rtol=0)


def test_group_shares_prompt_logits_then_diverges(tiny_run):
    _, _, _, out = tiny_run
    lg0 = out["logits"][0]
    for p in range(2):
        for g in range(1, 4):
            assert np.array_equal(lg0[p * 4 + g], lg0[p * 4])
    assert len({tuple(t) for t in out["tokens"]}) == 8


def test_prompt_sharing_equals_replicated_prompts(tiny_run):
    model, prompts, u, out = tiny_run
    rep = np.repeat(prompts, 4, axis=0)
    alone = rollout(model, rep, 1, 16, 1.0, 1.0, u, keep_logits=False)
    assert np.array_equal(alone["tokens"], out["tokens"])


def test_greedy_rollout_is_argmax_chain(tiny_run):
    model, prompts, u, _ = tiny_run
    out = rollout(model, prompts[:1], 2, 5, 0.0, 1.0, u[:2, :5])
    assert np.array_equal(out["tokens"][0], out["tokens"][1])
    for t in range(5):
        assert out["tokens"][0, t] == int(np.argmax(out["logits"][t, 0].astype(np.float32)))
