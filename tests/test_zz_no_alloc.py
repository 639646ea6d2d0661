"""rollout_sample_noalloc, the allocation-free draw: the same tokens as rollout_sample, the entry point it is a
variant of, on the same logits and uniforms -- bit for bit (both decide in exact integers) -- on two calls in
a row, the second with fewer rows; rows beyond one batch of the fixed scratch; vocabularies that no context
can have (not a multiple of 16) and the largest one the scratch holds, against the oracle; and argument
validation that happens before any device work."""
import numpy as np
import pytest

import paper_2608_11226_amd as R
import workload as W

torch = pytest.importorskip("torch")


def _draw_both(V, S, T, top_p, seed):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((S, V)) * 2.0).astype(np.float32)
    z[: min(S, 4)] = np.round(z[: min(S, 4)], 1)  # ties in value
    u = W.uniforms(S, 1, seed=seed + 1)[:, 0]
    dev = "cuda:0"
    zl = torch.from_numpy(z).to(dev)
    ud = torch.from_numpy(u).to(dev)
    cfg = R.model_config("tiny", R.DTYPE_FP32, 16, 8, 4)
    cfg.vocab = V  # rollout_sample takes the row width from its context
    eng = R.Engine(cfg)
    want = torch.full((S,), -1, dtype=torch.int32, device=dev)
    R.rollout_sample(eng.ctx, zl, S, T, top_p, ud, want)
    eng.synchronize()
    got = torch.full((S,), -1, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream(device=dev)
    R.rollout_sample_noalloc(zl, S, V, T, top_p, ud, got, stream.cuda_stream)
    stream.synchronize()
    eng.close()
    return got.cpu().numpy(), want.cpu().numpy()


@pytest.mark.gpu
@pytest.mark.parametrize("V,T,top_p", [(152064, 0.9, 0.95), (152064, 1.0, 1.0), (152064, 0.0, 1.0), (2048, 0.7, 0.5)])
def test_noalloc_draw_equals_rollout_sample_twice_the_second_smaller(V, T, top_p):
    print(f"noalloc sampler V={V} T={T} top_p={top_p}: 64 rows then 16", flush=True)
    for S, seed in ((64, 3), (16, 7)):
        got, want = _draw_both(V, S, T, top_p, seed)
        assert np.all((want >= 0) & (want < V))
        assert np.array_equal(got, want), np.nonzero(got != want)


@pytest.mark.gpu
def test_noalloc_draw_in_several_batches_of_the_fixed_scratch():
    # 152064 logits per row (38 chunks): exp values; per chunk four words, its 256 digit suffix sums and
    # counts; four 256-bin digit histograms per row -- the 64 MiB scratch holds 91 rows, so 200 rows take
    # three batches
    V, S = 152064, 200
    per_row = 4 * V + 38 * (24 + 256 * 12) + 4 * 256 * 8
    assert (R.NOALLOC_SCRATCH_BYTES - 4096) // per_row < S
    print(f"noalloc sampler V={V}: {S} rows in batches", flush=True)
    got, want = _draw_both(V, S, 0.9, 0.95, 11)
    assert np.array_equal(got, want), np.nonzero(got != want)


@pytest.mark.gpu
@pytest.mark.parametrize("V", [3, 4099])
@pytest.mark.parametrize("T,top_p", [(0.0, 1.0), (1.0, 1.0), (0.9, 0.95), (0.7, 0.5)])
def test_noalloc_draw_matches_the_oracle_at_vocabularies_no_context_has(V, T, top_p):
    # the row width is an argument here, so any vocabulary of at least 2 ids reaches the chunked kernels:
    # 4099 = one 4096-id chunk and one of 3 ids (rows not 16-byte aligned), 3 = one short chunk
    from oracle import sample_row

    S = 48
    rng = np.random.default_rng(V + 5)
    z = (rng.standard_normal((S, V)) * 2.0).astype(np.float32)
    z[:4] = np.round(z[:4], 1)  # ties in value
    u = W.uniforms(S, 1, seed=V)[:, 0]
    print(f"noalloc sampler V={V} T={T} top_p={top_p}: {S} rows against the oracle", flush=True)
    dev = "cuda:0"
    got = torch.full((S,), -1, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream(device=dev)
    R.rollout_sample_noalloc(torch.from_numpy(z).to(dev), S, V, T, top_p, torch.from_numpy(u).to(dev), got,
                             stream.cuda_stream)
    stream.synchronize()
    got = got.cpu().numpy()
    assert np.all((got >= 0) & (got < V))
    checked = 0
    for s in range(S):
        tok, margin = sample_row(z[s], T, top_p, float(u[s]))
        if margin < 1e-6:  # a draw within rounding of flipping (see the sampler parity test)
            continue
        assert got[s] == tok, f"row {s}: gpu {got[s]} oracle {tok} margin {margin}"
        checked += 1
    assert checked >= S - 8


@pytest.mark.gpu
@pytest.mark.parametrize("T,top_p", [(0.9, 0.95), (1.0, 1.0)])
def test_noalloc_draw_at_the_largest_vocabulary_the_scratch_holds(T, top_p):
    # 16,724,608 ids: 64 chunks of 64 batches each, one row per batch of the fixed scratch.  A thousand ids per
    # row stand far above the rest, so the kept set and the draw land among them with CDF buckets of about
    # 1e-3 of the mass (the oracle's margins are then far from the 1e-6 guard), while every pass still covers
    # the whole row.
    from oracle import sample_row

    V, S = 16_724_608, 2
    rng = np.random.default_rng(17)
    z = rng.standard_normal((S, V), dtype=np.float32)
    for s in range(S):
        ids = rng.choice(V, 1000, replace=False)
        z[s, ids] = 14.0 + rng.standard_normal(1000).astype(np.float32)
    u = W.uniforms(S, 1, seed=19)[:, 0]
    print(f"noalloc sampler at the largest vocabulary V={V} T={T} top_p={top_p}: {S} rows", flush=True)
    dev = "cuda:0"
    got = torch.full((S,), -1, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream(device=dev)
    R.rollout_sample_noalloc(torch.from_numpy(z).to(dev), S, V, T, top_p, torch.from_numpy(u).to(dev), got,
                             stream.cuda_stream)
    stream.synchronize()
    got = got.cpu().numpy()
    assert np.all((got >= 0) & (got < V))
    checked = 0
    for s in range(S):
        tok, margin = sample_row(z[s], T, top_p, float(u[s]))
        if margin < 1e-6:
            continue
        assert got[s] == tok, f"row {s}: gpu {got[s]} oracle {tok} margin {margin}"
        checked += 1
    assert checked >= 1


def test_noalloc_validates_before_any_device_work():
    # fake (never dereferenced) addresses: every error below is raised before the device is touched
    fake = 1 << 20
    # the largest row the 64 MiB scratch holds: 16,724,608 exp values, 64 chunks (four words, 256 suffix sums
    # and 256 counts each), four 256-bin histograms and 4 KiB of alignment slack; one logit more is rejected
    with pytest.raises(R.RolloutError, match="ENOMEM"):
        R.rollout_sample_noalloc(fake, 1, 16_724_609, 1.0, 1.0, fake, fake)
    assert "16724609 logits" in R.rollout_last_error()
    with pytest.raises(R.RolloutError, match="ENOMEM"):
        R.rollout_sample_noalloc(fake, 1, 1 << 24, 1.0, 1.0, fake, fake)
    for args in ((0, 1, 1024, 1.0, 1.0, fake, fake), (fake, 0, 1024, 1.0, 1.0, fake, fake),
                 (fake, 1, 1, 1.0, 1.0, fake, fake), (fake, 1, 1024, -1.0, 1.0, fake, fake),
                 (fake, 1, 1024, 1.0, 0.0, fake, fake), (fake, 1, 1024, 1.0, 1.5, fake, fake)):
        with pytest.raises(R.RolloutError, match="EINVAL"):
            R.rollout_sample_noalloc(*args)
    assert "top_p" in R.rollout_last_error()
