"""Pins for oracle/quant.py: properties that hold for any correct group quantiser, and worked groups."""
import numpy as np
import pytest

import workload as W
from oracle import OracleModel
from oracle.quant import GROUP, dequantize_int4, quantize_int4


def test_sixteen_level_group_is_reconstructed_exactly():
    # a group that already lies on 16 evenly spaced levels (exact in fp32) comes back unchanged
    levels = (np.arange(16, dtype=np.float32) - 7) * np.float32(0.015625)  # -0.109375 .. 0.125, step 2^-6
    w = np.tile(levels, GROUP // 16)[None, :]
    q, s, z = quantize_int4(w)
    assert s[0, 0] == np.float32(0.015625) and z[0, 0] == 7
    assert np.array_equal(q[0], np.tile(np.arange(16), GROUP // 16))
    assert np.array_equal(dequantize_int4(q, s, z), w)


@pytest.mark.parametrize("c", [0.0375, -0.0375, 0.0])
def test_constant_group_is_exact(c):
    w = np.full((2, GROUP), c, dtype=np.float32)
    q, s, z = quantize_int4(w)
    assert np.all(s == (abs(np.float32(c)) if c else 1.0))
    assert np.array_equal(dequantize_int4(q, s, z), w)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_bound_monotonicity_and_levels(seed):
    w = W.weight_matrix(seed, 7, 24, 4 * GROUP)
    q, s, z = quantize_int4(w)
    assert q.dtype == np.uint8 and q.max() <= 15 and z.max() <= 15
    d = dequantize_int4(q, s, z)
    sg = np.repeat(s, GROUP, axis=1)
    # |w - w'| <= s (one step: round-to-nearest plus the rounded zero point at the clamped ends)
    assert np.all(np.abs(d.astype(np.float64) - w) <= sg.astype(np.float64) * (1 + 1e-6))
    # interior values (no clamping) are within half a step
    inner = (q > 0) & (q < 15)
    assert np.all(np.abs(d - w)[inner] <= 0.5 * sg[inner] * (1 + 1e-6))
    for r in range(w.shape[0]):
        for g in range(w.shape[1] // GROUP):
            sl = slice(g * GROUP, (g + 1) * GROUP)
            order = np.argsort(w[r, sl], kind="stable")
            assert np.all(np.diff(q[r, sl][order].astype(int)) >= 0)  # codes are monotone in the weight
            assert len(np.unique(d[r, sl])) <= 16
            # the extremes map to the ends of the code range (up to the rounded zero point)
            assert q[r, sl].min() <= 1 and q[r, sl].max() >= 14


def test_int4_model_uses_exact_dequantised_layers_only():
    shape = W.ModelShape(1, 128, 2, 1, 64, 256, 512)
    wts = W.model_weights(shape)
    m = OracleModel(shape, wts, mode="int4")
    b = OracleModel(shape, wts, mode="bf16")
    assert np.array_equal(m.embed, b.embed) and np.array_equal(m.lm_head, b.lm_head)
    wq = wts["layers"][0]["wq"]
    assert np.array_equal(m.layers[0]["wq"], b.layers[0]["wq"]) is False
    q, s, z = quantize_int4(wq)
    got = m.layers[0]["wq"]
    # every weight is a whole number of its group's steps: w' / s = q - z exactly (the product is not rounded)
    steps = got / np.repeat(s, GROUP, axis=1).astype(np.float64)
    assert np.array_equal(steps, np.round(steps)) and np.abs(steps).max() <= 15
    assert np.array_equal(steps, q.astype(np.float64) - np.repeat(z, GROUP, axis=1))
    # rounded once to fp32 it is the exported form; rounding to bf16 would change some weights
    assert np.array_equal(got.astype(np.float32), dequantize_int4(q, s, z))
    from oracle.model import bf16_round
    assert not np.array_equal(got, bf16_round(got))
