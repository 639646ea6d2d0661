"""Full-size parity: one transformer layer (two at the 7B width) at the full width and vocabulary of a
benchmark shape, run by the GPU in that benchmark's launch configuration, against the oracle on sampled outputs.

* 7B-class (d 3584, GQA 28/4 x 128, FFN 18944, vocabulary 152064): 8 prompts x 256 tokens, G = 8, 64
  sequences -- prefill at M = 2048 on the tile GEMM, decode at M = 64 on the ring GEMMs and the 4-wave
  decode attention (256 workgroups), the full LM head.
* 14B-class (d 5120, GQA 40/8 x 128, FFN 13824): 16 prompts x 512 tokens, G = 16, 256 sequences -- prefill
  at M = 8192, decode at M = 256 on the tile GEMM (split K; gate/up with SwiGLU in the epilogue), the
  shared-prefix attention (suffix and prefix passes, 4-wave workgroups, two tiles per softmax update).
* 72B-class (d 8192, GQA 64/8 x 128, FFN 29568): 8 prompts x 512 tokens, G = 8, 64 sequences -- prefill
  at M = 4096, decode at M = 64 on the ring GEMMs (gate/up N = 59136), the 4-wave decode attention with
  eight query heads per KV head (512 workgroups, two per CU).

The oracle is fed only what the compared outputs need: the embedding rows of the tokens used and the
LM-head rows of a sample of vocabulary ids (both from the seeded generator, like the device's own
synthesis), and the full layer.  Prefill logits are compared for the sampled prompts (every member of the
group shares them), decode logits (two teacher-forced steps with fixed tokens) for one sequence of each
sampled group.  Tolerance: 3e-2 max-abs (the bf16 contract)."""
import numpy as np
import pytest

import paper_2608_11226_amd as R
import workload as W
from gpu_helpers import log, to_dev
from oracle import OracleModel

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

STEPS = 2
CASES = {
    # name: (shape name, model shape, prompts, prompt length, G, prompts compared on the oracle)
    "7b": ("7b", W.ModelShape(1, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1e6), 8, 256, 8, range(8)),
    # two layers: the residual add + RMSNorm between layers (fp32 residual, bf16 normed operand) at full width
    "7b-2layers": ("7b", W.ModelShape(2, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1e6), 8, 256, 8, (0, 3, 6)),
    "14b": ("14b", W.ModelShape(1, 5120, 40, 8, 128, 13824, 152064, 1e-6, 1e6), 16, 512, 16, (0, 5, 10, 15)),
    "72b": ("72b", W.ModelShape(1, 8192, 64, 8, 128, 29568, 152064, 1e-6, 1e6), 8, 512, 8, (0, 4, 7)),
}


def _oracle(shape, token_ids, vocab_ids):
    ids = np.unique(token_ids)
    remap = {int(t): j for j, t in enumerate(ids)}
    d = shape.d_model
    w = {"embed": W.weight_rows(0, W.tensor_id_embed(), ids, d),
         "lm_head": W.weight_rows(0, W.tensor_id_lm_head(shape), vocab_ids, d),
         "final_norm": np.ones(d, dtype=np.float32)}
    w["layers"] = {}
    for layer in range(shape.n_layers):
        lw = {"attn_norm": np.ones(d, np.float32), "mlp_norm": np.ones(d, np.float32)}
        for slot, name in enumerate(W.LAYER_SLOTS):
            if name.endswith("norm"):
                continue
            lw[name] = W.weight_matrix(0, W.tensor_id_layer(layer, slot), *W.logical_shape(shape, name))
            log(f"  oracle weight layer {layer} {name} {lw[name].shape} generated")
        w["layers"][layer] = lw
    log("  oracle weights generated")
    model = OracleModel(shape, w, mode="bf16")
    to_local = np.vectorize(lambda t: remap[int(t)])
    return model, to_local


@pytest.mark.parametrize("case", sorted(CASES))
def test_full_width_layer_in_the_benchmark_launch_configuration(case, monkeypatch):
    monkeypatch.delenv("ROLLOUT_SHARED_PREFIX", raising=False)
    monkeypatch.delenv("ROLLOUT_ATTN_WAVES", raising=False)
    name, shape, n_prompts, P, G, compared = CASES[case]
    S = n_prompts * G
    log(f"full-size parity, {case}: {shape.n_layers} layer(s) at full width, {n_prompts} prompts x {P}, G={G}, "
        f"{S} sequences, prefill + {STEPS} decode steps")
    rng = np.random.default_rng(11)
    prompts = W.prompts(n_prompts, P, shape.vocab, seed=71)
    feed = W.prompts(STEPS, S, shape.vocab, seed=72)  # teacher-forced decode tokens [step, sequence]
    vocab_ids = np.sort(rng.choice(shape.vocab, size=4096, replace=False))
    dev = "cuda:0"
    cfg = R.model_config(name, R.DTYPE_BF16, P, 8, S, n_layers=shape.n_layers)
    eng = R.Engine(cfg, group_size=G)
    cols = torch.from_numpy(vocab_ids).to(dev)
    logits = torch.empty((S, shape.vocab), dtype=torch.float32, device=dev)
    R.rollout_prefill(eng.ctx, to_dev(prompts, torch), n_prompts, P, G, logits)
    eng.synchronize()
    got = [logits[:, cols].cpu().numpy()]
    for t in range(STEPS):
        R.rollout_decode_step(eng.ctx, to_dev(feed[t].astype(np.int32), torch), logits)
        eng.synchronize()
        got.append(logits[:, cols].cpu().numpy())
    eng.close()
    log("  gpu done")

    seqs = {p: p * G + (p % G) for p in compared}  # one sequence per compared group, a different member each
    used = np.concatenate([prompts[list(compared)].reshape(-1)] + [feed[:, s] for s in seqs.values()])
    model, to_local = _oracle(shape, used, vocab_ids)
    worst = 0.0
    for p in compared:
        cache, lg = model.prefill(to_local(prompts[p]))
        errs = [max(float(np.max(np.abs(got[0][p * G + g] - lg))) for g in range(G))]  # the group shares it
        s = seqs[p]
        for t in range(STEPS):
            lg = model.decode(cache, int(to_local(feed[t, s])))
            errs.append(float(np.max(np.abs(got[t + 1][s] - lg))))
        worst = max(worst, max(errs))
        log(f"  prompt {p}: max abs logit error prefill {errs[0]:.4g}, decode {[round(e, 5) for e in errs[1:]]}")
    assert worst <= 3e-2
