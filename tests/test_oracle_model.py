"""Pins of the oracle transformer against library routines, closed forms and brute force."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workload as W
from conftest import read_golden
from oracle import model as M


def test_bf16_round_golden_cases():
    for src, want, *_ in read_golden("bf16_rne.txt"):
        x = np.array([int(src, 16)], dtype=np.uint32).view(np.float32)
        got = M.bf16_round(x).astype(np.float32).view(np.uint32)[0] >> 16
        assert got == int(want, 16), src


def test_bf16_round_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(M.bf16_round(x), want)


def test_rmsnorm_matches_torch():
    x = np.random.default_rng(1).standard_normal((5, 96)) * 4
    g = np.random.default_rng(2).standard_normal(96)
    want = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(M.rmsnorm(x, g, 1e-6), want, rtol=1e-13, atol=1e-13)
    # unit gains: output mean square is ms / (ms + eps)
    y = M.rmsnorm(x, np.ones(96), 1e-6)
    ms = (x * x).mean(-1)
    np.testing.assert_allclose((y * y).mean(-1), ms / (ms + 1e-6), rtol=1e-12)


def test_rope_closed_form_hd4():
    theta = 1e4
    e = np.eye(4)[:, None, :]  # four unit vectors as [T=4, H=1, hd=4]
    out = M.rope(e, np.ones(4), theta)[:, 0, :]
    f1 = theta ** -0.5
    # pairs are (0, 2) and (1, 3); pair 0 turns by 1 rad, pair 1 by theta^-1/2 rad
    np.testing.assert_allclose(out[0], [np.cos(1), 0, np.sin(1), 0], atol=1e-15)
    np.testing.assert_allclose(out[1], [0, np.cos(f1), 0, np.sin(f1)], atol=1e-15)
    np.testing.assert_allclose(out[2], [-np.sin(1), 0, np.cos(1), 0], atol=1e-15)
    np.testing.assert_allclose(out[3], [0, -np.sin(f1), 0, np.cos(f1)], atol=1e-15)


def test_rope_invariants():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 2, 64))
    k = rng.standard_normal((1, 2, 64))
    assert np.allclose(M.rope(q, np.array([0]), 1e6), q)  # position 0 is the identity
    for p in (1, 17, 1500):
        r = M.rope(q, np.array([p]), 1e6)
        np.testing.assert_allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-12)
    # the score depends only on the position difference
    d1 = np.sum(M.rope(q, np.array([10]), 1e4) * M.rope(k, np.array([3]), 1e4))
    d2 = np.sum(M.rope(q, np.array([107]), 1e4) * M.rope(k, np.array([100]), 1e4))
    assert abs(d1 - d2) < 1e-10


def test_attention_matches_torch_sdpa_gqa():
    rng = np.random.default_rng(4)
    t, hq, hkv, hd = 9, 6, 2, 16
    q, k, v = (rng.standard_normal((t, h, hd)) for h in (hq, hkv, hkv))
    got = M.attend(q, k, v, np.arange(t), hq // hkv)
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2)[None]
    want = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 2, 8))
    k = rng.standard_normal((1, 1, 8))
    v = rng.standard_normal((1, 1, 8))
    out = M.attend(q, k, v, np.array([0]), 2)
    np.testing.assert_allclose(out[0, 0], v[0, 0]) and np.testing.assert_allclose(out[0, 1], v[0, 0])
    # zero query: equal scores, output is the mean of the visible values
    vs = rng.standard_normal((5, 1, 8))
    out = M.attend(np.zeros((1, 1, 8)), rng.standard_normal((5, 1, 8)), vs, np.array([4]), 1)
    np.testing.assert_allclose(out[0, 0], vs[:, 0].mean(0), rtol=1e-12)
    # GQA equals MHA over repeated KV heads
    q = rng.standard_normal((4, 4, 8))
    k = rng.standard_normal((4, 2, 8))
    v = rng.standard_normal((4, 2, 8))
    gqa = M.attend(q, k, v, np.arange(4), 2)
    mha = M.attend(q, np.repeat(k, 2, axis=1), np.repeat(v, 2, axis=1), np.arange(4), 1)
    np.testing.assert_allclose(gqa, mha, rtol=1e-14)


def test_silu_matches_torch():
    z = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(M.silu(z), F.silu(torch.from_numpy(z)).numpy(), rtol=1e-14, atol=1e-300)


SMALL = W.ModelShape(2, 64, 4, 2, 16, 96, 200, 1e-6, 1e4)


@pytest.fixture(scope="module")
def small_weights():
    return W.model_weights(SMALL, seed=11)


def _torch_forward(shape, wts, tokens, mode):
    """Independent forward: torch library ops, complex-number RoPE."""
    dt = torch.float64

    def rnd(a):
        t = torch.as_tensor(np.asarray(a, dtype=np.float32))
        return (t.to(torch.bfloat16) if mode == "bf16" else t).to(dt)

    def act(t):
        return t.float().to(torch.bfloat16).to(dt) if mode == "bf16" else t

    T = len(tokens)
    hd = shape.head_dim
    inv = torch.tensor(shape.rope_theta, dtype=dt) ** (-torch.arange(0, hd, 2, dtype=dt) / hd)
    rot = torch.polar(torch.ones(T, hd // 2, dtype=dt), torch.arange(T, dtype=dt)[:, None] * inv[None])

    def rope_c(x):  # x [H, T, hd]: element i and i+hd/2 form one complex number
        c = torch.complex(x[..., : hd // 2], x[..., hd // 2 :]) * rot
        return torch.cat([c.real, c.imag], dim=-1)

    x = rnd(wts["embed"])[torch.as_tensor(tokens)]
    for l in range(shape.n_layers):
        lw = wts["layers"][l]
        a = act(F.rms_norm(x, (shape.d_model,), eps=shape.rms_eps))
        q = F.linear(a, rnd(lw["wq"])).view(T, shape.n_heads, hd).transpose(0, 1)
        k = F.linear(a, rnd(lw["wk"])).view(T, shape.n_kv_heads, hd).transpose(0, 1)
        v = F.linear(a, rnd(lw["wv"])).view(T, shape.n_kv_heads, hd).transpose(0, 1)
        q, k, v = act(rope_c(q)), act(rope_c(k)), act(v)
        o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=True, enable_gqa=True)[0]
        x = x + F.linear(act(o.transpose(0, 1).reshape(T, -1)), rnd(lw["wo"]))
        b = act(F.rms_norm(x, (shape.d_model,), eps=shape.rms_eps))
        h = act(F.silu(F.linear(b, rnd(lw["wgate"]))) * F.linear(b, rnd(lw["wup"])))
        x = x + F.linear(h, rnd(lw["wdown"]))
    f = act(F.rms_norm(x, (shape.d_model,), eps=shape.rms_eps))
    return F.linear(f, rnd(wts["lm_head"])).numpy()


@pytest.mark.parametrize("mode", ["fp32", "bf16"])
def test_full_forward_matches_independent_torch(small_weights, mode):
    model = M.OracleModel(SMALL, small_weights, mode=mode)
    toks = W.prompts(1, 13, SMALL.vocab, seed=5)[0]
    got = model.forward_full(toks)
    want = _torch_forward(SMALL, small_weights, toks, mode)
    # float64 on both sides; bf16 mode can differ only where an intermediate
    # lands within float64 rounding of a bf16 tie
    tol = 1e-10 if mode == "fp32" else 1e-6
    np.testing.assert_allclose(got, want, atol=tol, rtol=0)


@pytest.mark.parametrize("mode", ["fp32", "bf16"])
def test_cached_decode_equals_full_recompute(small_weights, mode):
    model = M.OracleModel(SMALL, small_weights, mode=mode)
    seq = W.prompts(1, 20, SMALL.vocab, seed=6)[0]
    full = model.forward_full(seq)
    cache, last = model.prefill(seq[:12])
    np.testing.assert_allclose(last, full[11], atol=1e-12, rtol=0)
    for t in range(12, 20):
        lg = model.decode(cache, int(seq[t]))
        np.testing.assert_allclose(lg, full[t], atol=1e-12, rtol=0)


def test_bf16_mode_rounding_points(small_weights):
    model = M.OracleModel(SMALL, small_weights, mode="bf16")
    for arr in (model.embed, model.lm_head, model.layers[0]["wq"], model.layers[1]["wdown"]):
        assert np.array_equal(M.bf16_round(arr), arr)
    cache, _ = model.prefill(W.prompts(1, 7, SMALL.vocab, seed=7)[0])
    for k, v in cache:
        assert np.array_equal(M.bf16_round(k), k) and np.array_equal(M.bf16_round(v), v)
