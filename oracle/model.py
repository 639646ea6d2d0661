"""Oracle transformer: plain float64 forward passes of a dense decoder.

TEST INFRASTRUCTURE ONLY (see the package header).

The paper's rollout phase (section 3, "Background") runs a dense decoder-only
transformer (the Qwen2.5 family, section 5) to generate completions; it fixes
no architectural detail beyond that, so the model below is the standard one,
with these readings where the paper is silent:

* RMSNorm: x / sqrt(mean(x^2) + eps) * gain, mean taken in float64; gains 1.
* Rotary embedding, rotate-half pairing (i, i + hd/2), inverse frequency
  theta^(-2i/hd), angle pos * inv_freq evaluated in float64.
* Causal attention with grouped KV heads: query head h reads KV head
  h // (n_heads / n_kv_heads); scale 1/sqrt(hd); max-subtracted softmax.
* SwiGLU MLP: down(silu(gate x) * up x), silu(z) = z / (1 + exp(-z)).
* No biases, untied LM head, logits from the final position(s).

Three numeric modes:

* ``"fp32"``: weights as generated (fp32 values), everything else float64.
* ``"bf16"``: the bf16 precision contract.  Values are rounded to bf16
  (round-to-nearest-even of their fp32 value) at exactly these points: every
  weight; every GEMM left operand (the two RMSNorm outputs, the attention
  output before Wo, silu(g)*u before Wdown, the final-norm output before the
  LM head); q after RoPE; k and v as stored in the cache.  The residual
  stream, accumulations, scores, softmax and logits are not rounded.
* ``"int4"``: the bf16 contract with the layer projections (q, k, v, o, gate,
  up, down) stored as int4 codes in groups of 128 (``oracle.quant``); they
  multiply with their exact dequantised values (q - z) * s.  Embedding and LM
  head as in bf16.

Parity: ``forward_full`` (no cache, full O(T^2) recompute) and the cached
``prefill``/``decode`` path are two independent routes to the same logits and
are checked against each other; the components are pinned against
``torch.nn.functional`` library routines (rms_norm, scaled_dot_product_attention,
silu) and closed forms (RoPE rotation identities, single-key attention) in
``tests/test_oracle_model.py``.  The whole-model logits of a random-init model
have no published value: beyond those pins they are "parity unpinned".
"""
from __future__ import annotations

import numpy as np

import workload

F64 = np.float64


def bf16_round(x) -> np.ndarray:
    """Round to bf16 (nearest, ties to even) of the fp32 value; returned as float64.

    NaN/Inf do not occur on this path and are not special-cased.
    """
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    b = f.view(np.uint32).astype(np.uint64)
    b = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
    return b.astype(np.uint32).view(np.float32).astype(F64)


def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain over the last axis, in float64."""
    x = np.asarray(x, dtype=F64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=F64)


def rope_angles(positions: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """angle[p, i] = pos_p * theta^(-2i/hd) for i < hd/2, float64."""
    i = np.arange(head_dim // 2, dtype=F64)
    inv_freq = np.power(F64(theta), -(2.0 * i) / head_dim)
    return np.asarray(positions, dtype=F64)[:, None] * inv_freq[None, :]


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding.

    x: [T, H, hd]; positions: [T].  Pair (i, i + hd/2) is rotated by angle[p, i]:
    out_i = x_i cos - x_{i+hd/2} sin;  out_{i+hd/2} = x_{i+hd/2} cos + x_i sin.
    """
    x = np.asarray(x, dtype=F64)
    hd = x.shape[-1]
    ang = rope_angles(positions, hd, theta)
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., : hd // 2], x[..., hd // 2 :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray, n_rep: int) -> np.ndarray:
    """Causal grouped-query attention for one sequence.

    q: [Tq, Hq, hd] at absolute positions q_pos; k, v: [Tk, Hkv, hd] at
    positions 0..Tk-1.  Query at position p sees keys 0..p.  Returns [Tq, Hq, hd].
    """
    tq, hq, hd = q.shape
    tk = k.shape[0]
    out = np.empty((tq, hq, hd), dtype=F64)
    scale = 1.0 / np.sqrt(F64(hd))
    key_pos = np.arange(tk)
    for h in range(hq):
        kvh = h // n_rep
        s = (q[:, h, :] @ k[:, kvh, :].T) * scale  # [Tq, Tk]
        s = np.where(key_pos[None, :] <= np.asarray(q_pos)[:, None], s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, kvh, :]
    return out


class OracleModel:
    """Float64 reference decoder over weights from the seeded generator."""

    def __init__(self, shape: workload.ModelShape, weights: dict | None = None, mode: str = "fp32",
                 seed: int = 0, std: float = 0.02):
        if mode not in ("fp32", "bf16", "int4"):
            raise ValueError("mode must be 'fp32', 'bf16' or 'int4'")
        self.shape = shape
        self.mode = mode
        if weights is None:
            weights = workload.model_weights(shape, seed=seed, std=std)
        cast = bf16_round if mode in ("bf16", "int4") else (lambda a: np.asarray(a, dtype=F64))
        if mode == "int4":
            from .quant import dequantize_int4_exact, quantize_int4

            cast_layer = lambda a: dequantize_int4_exact(*quantize_int4(a))
        else:
            cast_layer = cast
        self.embed = cast(weights["embed"])
        self.lm_head = cast(weights["lm_head"])
        self.final_norm = np.asarray(weights["final_norm"], dtype=F64)
        self.layers = []
        for l in range(shape.n_layers):
            lw = weights["layers"][l]
            self.layers.append({k: (np.asarray(v, F64) if k.endswith("norm") else cast_layer(v)) for k, v in lw.items()})

    # rounding at the contract's points (identity in fp32 mode)
    def _r(self, x: np.ndarray) -> np.ndarray:
        return bf16_round(x) if self.mode != "fp32" else x

    @property
    def n_rep(self) -> int:
        return self.shape.n_heads // self.shape.n_kv_heads

    # ------------------------------------------------------------------
    def _qkv(self, lw: dict, x: np.ndarray, positions: np.ndarray):
        s = self.shape
        a = self._r(rmsnorm(x, lw["attn_norm"], s.rms_eps))
        t = x.shape[0]
        q = (a @ lw["wq"].T).reshape(t, s.n_heads, s.head_dim)
        k = (a @ lw["wk"].T).reshape(t, s.n_kv_heads, s.head_dim)
        v = (a @ lw["wv"].T).reshape(t, s.n_kv_heads, s.head_dim)
        q = self._r(rope(q, positions, s.rope_theta))
        k = self._r(rope(k, positions, s.rope_theta))
        v = self._r(v)
        return q, k, v

    def _post_attn(self, lw: dict, x: np.ndarray, o: np.ndarray) -> np.ndarray:
        s = self.shape
        o = self._r(o.reshape(o.shape[0], s.q_dim))
        x = x + o @ lw["wo"].T
        b = self._r(rmsnorm(x, lw["mlp_norm"], s.rms_eps))
        hmid = self._r(silu(b @ lw["wgate"].T) * (b @ lw["wup"].T))
        return x + hmid @ lw["wdown"].T

    def logits_from_hidden(self, x: np.ndarray) -> np.ndarray:
        """Final RMSNorm then the LM head: [T, d] -> [T, V] float64."""
        f = self._r(rmsnorm(x, self.final_norm, self.shape.rms_eps))
        return f @ self.lm_head.T

    # ------------------------------------------------------------------
    def forward_full(self, tokens) -> np.ndarray:
        """Brute force: logits at every position of one sequence, no cache. [T, V]."""
        tokens = np.asarray(tokens).reshape(-1)
        pos = np.arange(tokens.size)
        x = self.embed[tokens].astype(F64)
        for lw in self.layers:
            q, k, v = self._qkv(lw, x, pos)
            o = attend(q, k, v, pos, self.n_rep)
            x = self._post_attn(lw, x, o)
        return self.logits_from_hidden(x)

    # ------------------------------------------------------------------
    def prefill(self, prompt) -> tuple[list, np.ndarray]:
        """Run one prompt; return (per-layer (K, V) cache, logits of the last position [V])."""
        prompt = np.asarray(prompt).reshape(-1)
        pos = np.arange(prompt.size)
        x = self.embed[prompt].astype(F64)
        cache = []
        for lw in self.layers:
            q, k, v = self._qkv(lw, x, pos)
            cache.append((k, v))
            o = attend(q, k, v, pos, self.n_rep)
            x = self._post_attn(lw, x, o)
        return cache, self.logits_from_hidden(x[-1:])[0]

    def decode(self, cache: list, token: int) -> np.ndarray:
        """Append one token at position len(cache) to one sequence's cache; return its logits [V].

        The cache (a list of per-layer (K, V) arrays) is extended in place.
        """
        pos = cache[0][0].shape[0]
        x = self.embed[np.array([token])].astype(F64)
        for l, lw in enumerate(self.layers):
            q, k, v = self._qkv(lw, x, np.array([pos]))
            kc = np.concatenate([cache[l][0], k], axis=0)
            vc = np.concatenate([cache[l][1], v], axis=0)
            cache[l] = (kc, vc)
            o = attend(q, kc, vc, np.array([pos]), self.n_rep)
            x = self._post_attn(lw, x, o)
        return self.logits_from_hidden(x)[0]
