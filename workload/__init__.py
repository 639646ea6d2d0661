"""Seeded synthetic workload for GRPO rollout generation.

This module produces the *inputs* of the rollout path and nothing else:
model weights, prompt token ids, the per-draw uniforms the sampler consumes
and the per-completion rewards fed to the advantage normaliser.  It holds none
of the method's arithmetic (no normalisation, no attention, no sampling, no
advantage formula); the oracle under ``oracle/`` and the GPU library each do
that work in code of their own.  The GPU library synthesises the weights on the
device with its own implementation of the same counter-based generator, from
the same published definition, so the two can be compared bit for bit.

Generator (counter-based, stateless):
    SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
    generators", OOPSLA 2014): the golden-gamma increment
    0x9E3779B97F4A7C15 and the variant-13 finaliser
        z ^= z >> 30; z *= 0xBF58476D1CE4E5B9
        z ^= z >> 27; z *= 0x94D049BB133111EB
        z ^= z >> 31
    all mod 2**64.  Element i of stream ``stream`` under seed ``seed`` is
        h(seed, stream, i) = mix(mix(seed ^ (stream * gamma)) + (i + 1) * gamma)
    so that h(0, 0, 0) is SplitMix64's first output for seed 0.

Weights ("random-init N(0, 0.02)"): v = h(weight_seed, tensor_id, i) with
i = row * in + col of the logical [out, in] matrix; the sum s of the four
16-bit limbs of v is an Irwin-Hall(4) variate; the weight is
fp32(((s - 131070) / 65536) * sqrt(3) * std) evaluated in IEEE double, left to
right, then rounded to nearest-even fp32.  Mean 0, standard deviation ``std``,
support +-3.46 std.  Norm gains are exactly 1.0 and are not hashed.

Tensor ids (``tensor_id``): embedding 0; layer l uses 1 + 9 l + j with
j = 0 attention-norm gain, 1 Wq, 2 Wk, 3 Wv, 4 Wo, 5 MLP-norm gain, 6 Wgate,
7 Wup, 8 Wdown; final-norm gain 1 + 9 L; LM head 2 + 9 L.

Prompts:  tok[p, t] = ((h(prompt_seed, 0x100000, p * P + t) >> 32) * V) >> 32.
Uniforms: u[s, t]   = (h(uniform_seed, 0x200000, s * N + t) >> 40) * 2**-24.
Rewards:  r[s]      = (h(reward_seed, 0x300000, s) >> 40) * 2**-24.
Default seeds: weights 0, prompts 1, uniforms 2, rewards 3.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
M1 = 0xBF58476D1CE4E5B9
M2 = 0x94D049BB133111EB
MASK64 = (1 << 64) - 1

STREAM_PROMPTS = 0x100000
STREAM_UNIFORMS = 0x200000
STREAM_REWARDS = 0x300000

SQRT3 = 1.7320508075688772

_CHUNK = 1 << 22


# ----------------------------------------------------------------------------
# generator
# ----------------------------------------------------------------------------
def mix64_int(z: int) -> int:
    """SplitMix64 finaliser on a Python int (mod 2**64)."""
    z &= MASK64
    z ^= z >> 30
    z = (z * M1) & MASK64
    z ^= z >> 27
    z = (z * M2) & MASK64
    z ^= z >> 31
    return z


def stream_key(seed: int, stream: int) -> int:
    """mix(seed ^ (stream * gamma)): the per-stream base of h()."""
    return mix64_int((seed ^ ((stream * GAMMA) & MASK64)) & MASK64)


def hash_int(seed: int, stream: int, i: int) -> int:
    """h(seed, stream, i) as a Python int: one element, pure integer arithmetic."""
    return mix64_int((stream_key(seed, stream) + (i + 1) * GAMMA) & MASK64)


def _mix64_np(z: np.ndarray) -> np.ndarray:
    # uint64 numpy arithmetic wraps mod 2**64, which is what the finaliser needs
    z ^= z >> np.uint64(30)
    z *= np.uint64(M1)
    z ^= z >> np.uint64(27)
    z *= np.uint64(M2)
    z ^= z >> np.uint64(31)
    return z


def hash_range(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """h(seed, stream, i) for i in [start, start + count) as uint64."""
    key = np.uint64(stream_key(seed, stream))
    idx = np.arange(start + 1, start + 1 + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = idx * np.uint64(GAMMA)
        z += key
        return _mix64_np(z)


def hash_indices(seed: int, stream: int, indices: np.ndarray) -> np.ndarray:
    """h(seed, stream, i) for an arbitrary array of indices (uint64 result)."""
    key = np.uint64(stream_key(seed, stream))
    idx = np.asarray(indices, dtype=np.uint64) + np.uint64(1)
    with np.errstate(over="ignore"):
        z = idx * np.uint64(GAMMA)
        z += key
        return _mix64_np(z)


def _weight_from_hash(v: np.ndarray, std: float) -> np.ndarray:
    m16 = np.uint64(0xFFFF)
    s = (v & m16) + ((v >> np.uint64(16)) & m16) + ((v >> np.uint64(32)) & m16) + (v >> np.uint64(48))
    x = s.astype(np.int64) - 131070
    w = ((x.astype(np.float64) / 65536.0) * SQRT3) * std
    return w.astype(np.float32)


# ----------------------------------------------------------------------------
# model shape and tensor ids
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelShape:
    """Shape of a dense decoder-only transformer (no biases, untied LM head)."""

    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 1e6

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


TINY = ModelShape(2, 128, 4, 4, 32, 512, 1024, 1e-6, 1e4)
SHAPE_7B = ModelShape(28, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1e6)
SHAPE_14B = ModelShape(48, 5120, 40, 8, 128, 13824, 152064, 1e-6, 1e6)
SHAPE_72B = ModelShape(80, 8192, 64, 8, 128, 29568, 152064, 1e-6, 1e6)

# per-layer slot of each tensor within the 9 ids of a layer
ATTN_NORM, WQ, WK, WV, WO, MLP_NORM, WGATE, WUP, WDOWN = range(9)
LAYER_SLOTS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wgate", "wup", "wdown")


def tensor_id_embed() -> int:
    return 0


def tensor_id_layer(layer: int, slot: int) -> int:
    return 1 + 9 * layer + slot


def tensor_id_final_norm(shape: ModelShape) -> int:
    return 1 + 9 * shape.n_layers


def tensor_id_lm_head(shape: ModelShape) -> int:
    return 2 + 9 * shape.n_layers


def logical_shape(shape: ModelShape, slot: str) -> tuple[int, int]:
    """[out, in] of a weight matrix (or [rows, d] of the embedding / LM head)."""
    d, qd, kvd, f, v = shape.d_model, shape.q_dim, shape.kv_dim, shape.d_ff, shape.vocab
    return {
        "embed": (v, d),
        "lm_head": (v, d),
        "wq": (qd, d),
        "wk": (kvd, d),
        "wv": (kvd, d),
        "wo": (d, qd),
        "wgate": (f, d),
        "wup": (f, d),
        "wdown": (d, f),
    }[slot]


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------
def weight_values(seed: int, tensor_id: int, start: int, count: int, std: float = 0.02) -> np.ndarray:
    """Flat fp32 weights of elements [start, start + count) of one tensor."""
    out = np.empty(count, dtype=np.float32)

    def fill(c0: int) -> None:
        n = min(_CHUNK, count - c0)
        out[c0 : c0 + n] = _weight_from_hash(hash_range(seed, tensor_id, start + c0, n), std)

    starts = range(0, count, _CHUNK)
    if count <= 2 * _CHUNK:
        for c0 in starts:
            fill(c0)
    else:  # numpy releases the GIL inside these ufuncs; chunks are independent
        with ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(fill, starts))
    return out


def weight_matrix(seed: int, tensor_id: int, rows: int, cols: int, std: float = 0.02) -> np.ndarray:
    """Full logical [rows, cols] fp32 matrix of one tensor."""
    return weight_values(seed, tensor_id, 0, rows * cols, std).reshape(rows, cols)


def weight_rows(seed: int, tensor_id: int, row_ids, cols: int, std: float = 0.02) -> np.ndarray:
    """Selected rows of a logical [*, cols] matrix (e.g. embedding rows for given tokens)."""
    row_ids = np.asarray(row_ids, dtype=np.int64).reshape(-1)
    out = np.empty((row_ids.size, cols), dtype=np.float32)
    for j, r in enumerate(row_ids):
        out[j] = weight_values(seed, tensor_id, int(r) * cols, cols, std)
    return out


def weight_elements(seed: int, tensor_id: int, flat_indices, std: float = 0.02) -> np.ndarray:
    """Arbitrary elements (flat index row * cols + col) of one tensor."""
    return _weight_from_hash(hash_indices(seed, tensor_id, flat_indices), std)


def model_weights(shape: ModelShape, seed: int = 0, std: float = 0.02, layers=None) -> dict:
    """Every weight of the model as fp32 arrays in logical [out, in] layout.

    ``layers`` restricts generation to a subset of layer indices (the others
    are omitted from the dict); the embedding and LM head are always produced.
    Norm gains are exactly one.
    """
    layers = range(shape.n_layers) if layers is None else layers
    w = {
        "embed": weight_matrix(seed, tensor_id_embed(), *logical_shape(shape, "embed"), std=std),
        "final_norm": np.ones(shape.d_model, dtype=np.float32),
        "lm_head": weight_matrix(seed, tensor_id_lm_head(shape), *logical_shape(shape, "lm_head"), std=std),
        "layers": {},
    }
    for l in layers:
        lw = {"attn_norm": np.ones(shape.d_model, np.float32), "mlp_norm": np.ones(shape.d_model, np.float32)}
        for slot in (WQ, WK, WV, WO, WGATE, WUP, WDOWN):
            name = LAYER_SLOTS[slot]
            lw[name] = weight_matrix(seed, tensor_id_layer(l, slot), *logical_shape(shape, name), std=std)
        w["layers"][l] = lw
    return w


# ----------------------------------------------------------------------------
# prompts, uniforms, rewards
# ----------------------------------------------------------------------------
def prompts(n_prompts: int, prompt_len: int, vocab: int, seed: int = 1) -> np.ndarray:
    """Uniform token ids, int32 [n_prompts, prompt_len] (multiply-shift range reduction)."""
    v = hash_range(seed, STREAM_PROMPTS, 0, n_prompts * prompt_len)
    tok = ((v >> np.uint64(32)) * np.uint64(vocab)) >> np.uint64(32)
    return tok.astype(np.int32).reshape(n_prompts, prompt_len)


def uniforms(n_seqs: int, n_new: int, seed: int = 2, first_seq: int = 0) -> np.ndarray:
    """Sampler uniforms u[s, t] in [0, 1) on a 2**-24 grid, fp32 [n_seqs, n_new].

    ``first_seq`` offsets the global completion index (several waves).
    """
    v = hash_range(seed, STREAM_UNIFORMS, first_seq * n_new, n_seqs * n_new)
    return ((v >> np.uint64(40)).astype(np.float64) * 2.0**-24).astype(np.float32).reshape(n_seqs, n_new)


def rewards(n: int, seed: int = 3, first: int = 0) -> np.ndarray:
    """Per-completion rewards uniform on [0, 1) (2**-24 grid), fp32 [n]."""
    v = hash_range(seed, STREAM_REWARDS, first, n)
    return ((v >> np.uint64(40)).astype(np.float64) * 2.0**-24).astype(np.float32)
