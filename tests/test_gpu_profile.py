"""The projection-timing entry point ``rollout_profile_projections``: it replays one decode step's projection
GEMMs as a HIP graph and must leave the wave's state alone, so that the next decode step returns the same
logits, bit for bit, as on a context that was never measured.  Its launch count and per-launch bytes and
flops follow from the shapes: four projections per layer (QKV, O, gate/up with SwiGLU, down) and the LM head,
each reading its weights, activations and writing its output once."""
import numpy as np
import pytest

import paper_2608_11226_amd as R
import workload as W
from gpu_helpers import log, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SMALL_BF16 = (2, 256, 8, 2, 64, 512, 2048, 1e6)
INT4_SMALL = (2, 256, 8, 2, 64, 512, 2048, 1e6)


def _bf16_accounting(shape, M):
    L, d, nh, nkv, hd, ff, V, _ = shape
    nqkv, qd = (nh + 2 * nkv) * hd, nh * hd
    b = 0.0
    f = 0.0
    for N, K, out_bytes in ((nqkv, d, M * nqkv * 4), (d, qd, M * d * 4), (2 * ff, d, M * ff * 2), (d, ff, M * d * 4)):
        b += L * (N * K * 2 + M * K * 2 + out_bytes)
        f += L * 2.0 * M * N * K
    b += V * d * 2 + M * d * 2 + M * V * 4
    f += 2.0 * M * V * d
    return 4 * L + 1, b, f


def _prefilled(cfg, G, n_prompts, P, seed):
    eng = R.Engine(cfg, group_size=G)
    prompts = to_dev(W.prompts(n_prompts, P, cfg.vocab, seed=seed), torch)
    logits = torch.empty((n_prompts * G, cfg.vocab), dtype=torch.float32, device="cuda:0")
    R.rollout_prefill(eng.ctx, prompts, n_prompts, P, G, logits)
    return eng, logits


def test_projection_replay_leaves_the_wave_untouched_and_counts_the_launches():
    n_prompts, G, P = 3, 4, 40
    S = n_prompts * G
    log(f"projection replay: small GQA bf16, {S} rows")
    cfg = R.model_config(SMALL_BF16, R.DTYPE_BF16, P, 8, S)
    toks = to_dev(np.arange(S, dtype=np.int32) * 37 % cfg.vocab, torch)
    ref, logits_ref = _prefilled(cfg, G, n_prompts, P, seed=61)
    R.rollout_decode_step(ref.ctx, toks, logits_ref)
    ref.synchronize()
    eng, logits = _prefilled(cfg, G, n_prompts, P, seed=61)
    scratch = torch.empty_like(logits)
    pp = R.rollout_profile_projections(eng.ctx, 3, scratch)
    R.rollout_decode_step(eng.ctx, toks, logits)
    eng.synchronize()
    assert torch.equal(logits.view(torch.int32), logits_ref.view(torch.int32)), "the replay changed the wave's state"
    launches, b, f = _bf16_accounting(SMALL_BF16, S)
    assert pp.launches == launches
    assert pp.avg_us > 0
    assert pp.bytes_per_launch == pytest.approx(b / launches, rel=1e-12)
    assert pp.flops_per_launch == pytest.approx(f / launches, rel=1e-12)
    assert bool(torch.isfinite(scratch).all())
    with pytest.raises(R.RolloutError) as e:
        R.rollout_profile_projections(eng.ctx, 0, scratch)
    assert e.value.code == R.EINVAL
    ref.close()
    eng.close()


def test_projection_replay_refuses_int4_batches_that_dequantise_first():
    n_prompts, G, P = 9, 8, 16
    log("projection replay: int4 with 72 rows is refused")
    cfg = R.model_config(INT4_SMALL, R.DTYPE_INT4, P, 8, n_prompts * G)
    eng, logits = _prefilled(cfg, G, n_prompts, P, seed=62)
    with pytest.raises(R.RolloutError) as e:
        R.rollout_profile_projections(eng.ctx, 1, logits)
    assert e.value.code == R.EINVAL
    eng.close()


def test_projection_replay_needs_a_wave():
    cfg = R.model_config(SMALL_BF16, R.DTYPE_BF16, 16, 8, 4)
    eng = R.Engine(cfg, group_size=2)
    logits = torch.empty((4, cfg.vocab), dtype=torch.float32, device="cuda:0")
    with pytest.raises(R.RolloutError) as e:
        R.rollout_profile_projections(eng.ctx, 1, logits)
    assert e.value.code == R.ESTATE
    eng.close()
