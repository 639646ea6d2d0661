"""The path the benchmark times: bf16 ``rollout_generate``, which captures one decode step plus its draw as a
HIP graph per wave and replays it for every later token, against the eager chain of the same operations
through the C ABI (``rollout_prefill`` -> ``rollout_sample`` -> (N - 1) x (``rollout_decode_step`` ->
``rollout_sample``)) on the same device, inputs and uniforms.

Both sides launch the same kernels at the same row counts (the graph replays exactly the launches of one
eager step, with the token column and the positions advanced on the device), every split-K sum is taken in
split order and the sampler's decision is exact integer arithmetic, so the tokens must be identical, bit for
bit -- not merely close.  A second ``rollout_generate`` on the same context must repeat the first exactly
(no dependence on scheduling, XCD placement or leftover state).

Cases: a small GQA model across the decode-attention path switches and several waves, and one layer at the
full width and vocabulary of the 7B, 14B and 72B shapes in their benchmark launch configurations (64 rows on
the ring GEMMs; 256 rows on the split tile GEMM with the shared-prefix attention; 64 rows with eight query
heads per KV head)."""
import numpy as np
import pytest

import paper_2608_11226_amd as R
import workload as W
from gpu_helpers import log, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SMALL_BF16 = (2, 256, 8, 2, 64, 512, 2048, 1e6)
ATTN_KNOBS = [("1", None), ("2", "8"), ("2", "4"), ("0", "4")]


def _set_knobs(monkeypatch, shared, waves):
    if shared is None:
        monkeypatch.delenv("ROLLOUT_SHARED_PREFIX", raising=False)
    else:
        monkeypatch.setenv("ROLLOUT_SHARED_PREFIX", shared)
    if waves is None:
        monkeypatch.delenv("ROLLOUT_ATTN_WAVES", raising=False)
    else:
        monkeypatch.setenv("ROLLOUT_ATTN_WAVES", waves)


def _eager(eng, prompts, G, seqs, N, T, top_p, u):
    """The rollout as separate C-ABI calls, wave by wave (waves of whole groups, as rollout_generate makes)."""
    n_prompts, P = prompts.shape
    V = eng.cfg.vocab
    dev = "cuda:0"
    per_wave = min(seqs, eng.cfg.max_seqs_in_flight) // G
    out = np.full((n_prompts * G, N), -1, dtype=np.int32)
    for p0 in range(0, n_prompts, per_wave):
        np_ = min(per_wave, n_prompts - p0)
        S = np_ * G
        s0 = p0 * G
        logits = torch.empty((S, V), dtype=torch.float32, device=dev)
        toks = torch.empty((N, S), dtype=torch.int32, device=dev)
        uw = to_dev(np.ascontiguousarray(u[s0:s0 + S].T), torch)  # [N, S]: one contiguous column per step
        R.rollout_prefill(eng.ctx, to_dev(prompts[p0:p0 + np_], torch), np_, P, G, logits)
        R.rollout_sample(eng.ctx, logits, S, T, top_p, uw[0], toks[0])
        for t in range(1, N):
            R.rollout_decode_step(eng.ctx, toks[t - 1], logits)
            R.rollout_sample(eng.ctx, logits, S, T, top_p, uw[t], toks[t])
        eng.synchronize()
        out[s0:s0 + S] = toks.cpu().numpy().T
    return out


def _graph(eng, prompts, G, seqs, N, T, top_p, u):
    n_prompts, P = prompts.shape
    out = torch.full((n_prompts * G, N), -1, dtype=torch.int32, device="cuda:0")
    R.rollout_generate(eng.ctx, to_dev(prompts, torch), n_prompts, P, G, seqs, N, T, top_p, to_dev(u, torch), out)
    eng.synchronize()
    return out.cpu().numpy()


def _compare(graph, eager, V):
    assert np.all((graph >= 0) & (graph < V))
    diff = np.argwhere(graph != eager)
    assert diff.size == 0, f"{len(diff)} tokens differ, first at (sequence, step) {tuple(diff[0])}: " \
                           f"graph {graph[tuple(diff[0])]} eager {eager[tuple(diff[0])]}"


@pytest.mark.parametrize("shared,waves", ATTN_KNOBS)
@pytest.mark.parametrize("seqs", [12, 4])
def test_small_bf16_generate_equals_the_eager_chain(seqs, shared, waves, monkeypatch):
    _set_knobs(monkeypatch, shared, waves)
    n_prompts, G, P, N, T, top_p = 3, 4, 40, 12, 0.9, 0.95
    log(f"bf16 small GQA generate vs eager chain: {n_prompts} prompts x {P}, G={G}, {seqs} in flight, N={N}, "
        f"shared={shared} waves={waves}")
    cfg = R.model_config(SMALL_BF16, R.DTYPE_BF16, P, N, n_prompts * G)  # a KV pool for one wave of them all
    eng = R.Engine(cfg, group_size=G)
    prompts = W.prompts(n_prompts, P, cfg.vocab, seed=41)
    u = W.uniforms(n_prompts * G, N, seed=42)
    graph = _graph(eng, prompts, G, seqs, N, T, top_p, u)
    eager = _eager(eng, prompts, G, seqs, N, T, top_p, u)
    _compare(graph, eager, cfg.vocab)
    again = _graph(eng, prompts, G, seqs, N, T, top_p, u)
    assert np.array_equal(graph, again), "a second rollout_generate differs from the first"
    eng.close()


# name: (shape, prompts, prompt length, G, sequences in flight, new tokens, temperature, top-p)
LAUNCH = {
    "7b": ("7b", 8, 256, 8, 64, 16, 0.9, 0.95),
    "14b": ("14b", 16, 512, 16, 256, 8, 1.0, 1.0),
    "72b": ("72b", 8, 512, 8, 64, 8, 1.0, 1.0),
}


@pytest.mark.parametrize("case", sorted(LAUNCH))
def test_generate_in_the_benchmark_launch_configuration_equals_the_eager_chain(case, monkeypatch):
    _set_knobs(monkeypatch, None, None)
    shape, n_prompts, P, G, S, N, T, top_p = LAUNCH[case]
    log(f"bf16 generate vs eager chain, {case} width, one layer: {n_prompts} prompts x {P}, G={G}, {S} in flight, "
        f"N={N}, T={T}, top-p {top_p}")
    cfg = R.model_config(shape, R.DTYPE_BF16, P, N, S, n_layers=1)
    eng = R.Engine(cfg, group_size=G)
    assert eng.cfg.max_seqs_in_flight >= S
    prompts = W.prompts(n_prompts, P, cfg.vocab, seed=43)
    u = W.uniforms(n_prompts * G, N, seed=44)
    graph = _graph(eng, prompts, G, S, N, T, top_p, u)
    log("  graph rollout done")
    eager = _eager(eng, prompts, G, S, N, T, top_p, u)
    log("  eager chain done")
    _compare(graph, eager, cfg.vocab)
    again = _graph(eng, prompts, G, S, N, T, top_p, u)
    assert np.array_equal(graph, again), "a second rollout_generate differs from the first"
    # the draws are not degenerate: the group's members diverge after their shared prompt
    assert len(np.unique(graph[:G, 1:])) > G
    eng.close()


@pytest.mark.parametrize("case", ["7b", "72b"])
def test_weights_bit_exact_on_sampled_indices_at_full_size(case):
    # every matrix of two layers, the embedding and the LM head of a full-width model, on 4096 sampled
    # elements each, against the seeded generator rounded to bf16
    from oracle import bf16_round

    cfg = R.model_config(case, R.DTYPE_BF16, 16, 8, 8, n_layers=2)
    log(f"sampled weights bit-exact, {case} width, two layers")
    eng = R.Engine(cfg)
    sh = W.ModelShape(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff, cfg.vocab,
                      cfg.rms_eps, cfg.rope_theta)
    ids = [(W.tensor_id_embed(), "embed"), (W.tensor_id_lm_head(sh), "lm_head")]
    for l in range(sh.n_layers):
        for slot in (W.WQ, W.WK, W.WV, W.WO, W.WGATE, W.WUP, W.WDOWN):
            ids.append((W.tensor_id_layer(l, slot), W.LAYER_SLOTS[slot]))
    rng = np.random.default_rng(5)
    for tid, name in ids:
        rows, cols = W.logical_shape(sh, name)
        n = rows * cols
        idx = np.unique(np.concatenate([rng.integers(0, n, size=4096), [0, cols - 1, n - cols, n - 1]]))
        out = torch.empty(n, dtype=torch.float32, device="cuda:0")
        R.rollout_export_weight(eng.ctx, tid, out)
        eng.synchronize()
        got = out[torch.from_numpy(idx).to("cuda:0")].cpu().numpy()
        del out
        want = bf16_round(W.weight_elements(0, tid, idx)).astype(np.float32)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), f"tensor {tid} ({name})"
    eng.close()
