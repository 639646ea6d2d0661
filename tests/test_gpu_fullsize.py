"""Full-size parity: one transformer layer of the 7B-class shape (d 3584, GQA 28/4 x 128, FFN 18944,
vocabulary 152064) run by the GPU in the launch configuration of the 7B rollout benchmark (8 prompts x 256
tokens, G = 8, 64 sequences: prefill at M = 2048 on the tile GEMM, decode at M = 64 on the ring GEMMs and
decode attention, the full LM head), against the oracle on sampled outputs.

The oracle is fed only what these outputs need: the embedding rows of the tokens used and the LM-head rows
of a sample of vocabulary ids (both from the seeded generator, like the device's own synthesis), and the
full layer.  Prefill logits are compared for every prompt, decode logits (two teacher-forced steps with
fixed tokens) for one sequence of every group.  Tolerance: 3e-2 max-abs (the bf16 contract)."""
import numpy as np
import pytest

import paper_2608_11226_amd as R
import workload as W
from gpu_helpers import log, to_dev
from oracle import OracleModel

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SHAPE = W.ModelShape(1, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1e6)
N_PROMPTS, P, G, STEPS = 8, 256, 8, 2
S = N_PROMPTS * G


def _oracle(prompts, feed, vocab_ids):
    ids = np.unique(np.concatenate([prompts.reshape(-1), feed.reshape(-1)]))
    remap = {int(t): j for j, t in enumerate(ids)}
    d = SHAPE.d_model
    w = {"embed": W.weight_rows(0, W.tensor_id_embed(), ids, d),
         "lm_head": W.weight_rows(0, W.tensor_id_lm_head(SHAPE), vocab_ids, d),
         "final_norm": np.ones(d, dtype=np.float32)}
    lw = {"attn_norm": np.ones(d, np.float32), "mlp_norm": np.ones(d, np.float32)}
    for slot, name in enumerate(W.LAYER_SLOTS):
        if name.endswith("norm"):
            continue
        lw[name] = W.weight_matrix(0, W.tensor_id_layer(0, slot), *W.logical_shape(SHAPE, name))
    w["layers"] = {0: lw}
    log("  oracle weights generated")
    model = OracleModel(SHAPE, w, mode="bf16")
    to_local = np.vectorize(lambda t: remap[int(t)])
    return model, to_local


def test_7b_width_layer_in_the_benchmark_launch_configuration():
    log("full-size parity: one 7B-width layer, 8 prompts x 256, G=8, 64 sequences, prefill + 2 decode steps")
    rng = np.random.default_rng(11)
    prompts = W.prompts(N_PROMPTS, P, SHAPE.vocab, seed=71)
    feed = W.prompts(STEPS, S, SHAPE.vocab, seed=72)  # teacher-forced decode tokens [step, sequence]
    vocab_ids = np.sort(rng.choice(SHAPE.vocab, size=4096, replace=False))
    dev = "cuda:0"
    cfg = R.model_config("7b", R.DTYPE_BF16, P, 8, S, n_layers=1)
    eng = R.Engine(cfg, group_size=G)
    logits = torch.empty((S, SHAPE.vocab), dtype=torch.float32, device=dev)
    R.rollout_prefill(eng.ctx, to_dev(prompts, torch), N_PROMPTS, P, G, logits)
    eng.synchronize()
    got = [logits[:, torch.from_numpy(vocab_ids).to(dev)].cpu().numpy()]
    for t in range(STEPS):
        R.rollout_decode_step(eng.ctx, to_dev(feed[t].astype(np.int32), torch), logits)
        eng.synchronize()
        got.append(logits[:, torch.from_numpy(vocab_ids).to(dev)].cpu().numpy())
    eng.close()
    log("  gpu done")

    model, to_local = _oracle(prompts, feed, vocab_ids)
    worst = 0.0
    for p in range(N_PROMPTS):
        cache, lg = model.prefill(to_local(prompts[p]))
        errs = [max(float(np.max(np.abs(got[0][p * G + g] - lg))) for g in range(G))]  # the group shares it
        s = p * G + (p % G)  # one sequence per group, a different member each time
        for t in range(STEPS):
            lg = model.decode(cache, int(to_local(feed[t, s])))
            errs.append(float(np.max(np.abs(got[t + 1][s] - lg))))
        worst = max(worst, max(errs))
        log(f"  prompt {p}: max abs logit error prefill {errs[0]:.4g}, decode {[round(e, 5) for e in errs[1:]]}")
    assert worst <= 3e-2
