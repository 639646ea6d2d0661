"""Weight-only int4 quantisation of the layer projections (the generation proxy's AWQ-style format).

TEST INFRASTRUCTURE ONLY (see the package header).

The paper's second campaign generates with an AWQ-quantised 72B model (sections 5 and 6.6); it
fixes no format.  Reading (listed in the design notes): the AWQ storage format, 4-bit codes in groups
of 128 consecutive input features of one output row, each group with its own scale and zero point,
quantised by rounding to nearest.  AWQ's activation-aware per-channel scale search needs calibration
activations of a trained model and has no meaning for synthetic weights, so it is not applied; the
stored format and the arithmetic of a GEMM over it are the same.

Per group of one row (fp32 arithmetic throughout, round-half-even):
    lo, hi = min, max of the group's fp32 weights
    s = (hi - lo) / 15                   (a constant group: s = |hi|, or 1 when it is 0; then w' = w)
    z = clamp(rint(-lo / s), 0, 15)
    q = clamp(rint(w / s) + z, 0, 15)    (the 4-bit code)
    w' = (q - z) * s                     (the dequantised weight)

Reading of the dequantised weight: the model multiplies with w' = (q - z) * s exactly, never rounded to
bf16 (a group-quantised GEMM applies s to each group's integer dot product; the product of a 4-bit
integer and an fp32 scale is exact in float64).  ``dequantize_int4`` returns it rounded once to fp32,
the form a device exports.

Parity: pinned in tests/test_oracle_quant.py by the reconstruction bound |w - w'| <= s, monotonicity of
the codes, at most 16 distinct values per group, exact reconstruction of 16-level groups, and the
degenerate constant group.
"""
from __future__ import annotations

import numpy as np

GROUP = 128
F32 = np.float32


def quantize_int4(w):
    """Codes (uint8, [rows, cols]), scales (fp32, [rows, cols / 128]) and zeros (uint8, same) of a matrix."""
    w = np.asarray(w, dtype=F32)
    rows, cols = w.shape
    if cols % GROUP:
        raise ValueError("the input dimension must be a multiple of 128")
    g = w.reshape(rows, cols // GROUP, GROUP)
    lo = g.min(axis=2)
    hi = g.max(axis=2)
    s = ((hi - lo) / F32(15)).astype(F32)
    s = np.where(s == 0, np.where(hi == 0, F32(1), np.abs(hi)), s).astype(F32)
    z = np.clip(np.rint(-lo / s), 0, 15).astype(F32)
    q = np.clip(np.rint(g / s[:, :, None]) + z[:, :, None], 0, 15).astype(np.uint8)
    return q.reshape(rows, cols), s, z.astype(np.uint8)


def dequantize_int4(q, s, z):
    """fp32 dequantised weights (q - z) * s (the product rounded once to fp32)."""
    q = np.asarray(q, dtype=F32)
    rows, cols = q.shape
    g = q.reshape(rows, cols // GROUP, GROUP)
    out = (g - np.asarray(z, dtype=F32)[:, :, None]) * np.asarray(s, dtype=F32)[:, :, None]
    return out.astype(F32).reshape(rows, cols)


def dequantize_int4_exact(q, s, z):
    """float64 dequantised weights (q - z) * s, exact."""
    q = np.asarray(q, dtype=np.float64)
    rows, cols = q.shape
    g = q.reshape(rows, cols // GROUP, GROUP)
    out = (g - np.asarray(z, dtype=np.float64)[:, :, None]) * np.asarray(s, dtype=np.float64)[:, :, None]
    return out.reshape(rows, cols)
