"""GPU parity of stop-token completions under continuous batching (rollout_generate_eos) and of the
length-target reward, through the C ABI, against oracle/batching.py."""
import numpy as np
import pytest

import paper_2608_11226_amd as R
import workload as W
from gpu_helpers import guarded_token_compare, log, shape_of, to_dev
from oracle import OracleModel, rollout
from oracle.batching import continuous_schedule, length_target_reward, rollout_eos, sequence_schedule

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SMALL_BF16 = (2, 256, 8, 2, 64, 512, 2048, 1e6)


def _run_eos(eng, prompts, G, slots, N, T, top_p, u, stop, refill, whole_groups=1):
    n_prompts, P = prompts.shape
    S = n_prompts * G
    dev = "cuda:0"
    tokens = torch.full((S, N), -7, dtype=torch.int32, device=dev)
    lengths = torch.full((S,), -7, dtype=torch.int32, device=dev)
    admit = torch.full((S,), -7, dtype=torch.int32, device=dev)
    stop_t = to_dev(np.asarray(stop, dtype=np.int32), torch) if len(stop) else torch.zeros(1, dtype=torch.int32,
                                                                                            device=dev)
    steps = R.rollout_generate_eos(eng.ctx, to_dev(prompts, torch), n_prompts, P, G, slots, N, T, top_p,
                                   to_dev(u, torch), stop_t, len(stop), refill, whole_groups, tokens, lengths, admit)
    eng.synchronize()
    return tokens.cpu().numpy(), lengths.cpu().numpy(), admit.cpu().numpy(), steps


def _expected_schedule(L, G, slots, refill, whole_groups):
    if whole_groups:
        sch = continuous_schedule(L, G, slots // G, refill)
        return np.repeat(sch["admit"], G), sch["steps"]
    sch = sequence_schedule(L, slots, refill)
    return sch["admit"], sch["steps"]


def _check_structure(tokens, lengths, stop, N, V):
    stop = set(int(s) for s in stop)
    for s in range(tokens.shape[0]):
        L = int(lengths[s])
        assert 1 <= L <= N
        assert np.all(tokens[s, L:] == -1), f"completion {s} not padded after its end"
        body = tokens[s, :L]
        assert np.all((body >= 0) & (body < V))
        hits = [t for t in range(L) if int(body[t]) in stop]
        # ends at its first stop token, or runs to max_new_tokens without one
        assert (hits and hits[0] == L - 1) or (not hits and L == N), f"completion {s}: stop rule"


@pytest.mark.parametrize("whole_groups", [1, 0])
@pytest.mark.parametrize("T,top_p,refill", [(1.0, 1.0, 1), (0.8, 0.9, 3), (0.0, 1.0, 2)])
def test_tiny_fp32_eos_matches_oracle(T, top_p, refill, whole_groups):
    G, n_prompts, P, N, slots = 4, 5, 12, 16, 8
    log(f"tiny fp32 eos: {n_prompts} prompts x G={G}, {slots} slots, refill every {refill} "
        f"({'whole groups' if whole_groups else 'single completions'}), T={T} top_p={top_p}")
    cfg = R.model_config("tiny", R.DTYPE_FP32, P, N, 2 * slots)  # room for the prompt records of single refill
    eng = R.Engine(cfg, group_size=G)
    model = OracleModel(shape_of(cfg), mode="fp32")
    prompts = W.prompts(n_prompts, P, cfg.vocab, seed=51)
    u = W.uniforms(n_prompts * G, N, seed=52)
    plain = rollout(model, prompts, G, N, T, top_p, u, keep_logits=False)["tokens"]
    # stop tokens taken from the draws themselves so that the completions end at different lengths
    stop = sorted({int(plain[0, 2]), int(plain[5, 6]), int(plain[9, 0]), int(plain[14, 11])})
    ref = rollout_eos(model, prompts, G, N, T, top_p, u, stop)
    tok, L, admit, steps = _run_eos(eng, prompts, G, slots, N, T, top_p, u, stop, refill, whole_groups)
    _check_structure(tok, L, stop, N, cfg.vocab)
    compared, skipped = guarded_token_compare(tok, np.where(ref["tokens"] < 0, -1, ref["tokens"]), ref["margins"])
    log(f"  lengths {L.tolist()}; compared {compared} tokens, skipped {skipped} after near-ties")
    exact = [s for s in range(n_prompts * G) if np.all(ref["margins"][s, :ref["lengths"][s]] >= 1e-5)]
    for s in exact:
        assert L[s] == ref["lengths"][s], f"completion {s}: length {L[s]} oracle {ref['lengths'][s]}"
    assert compared >= 60 and len(exact) >= n_prompts * G // 2
    # the schedule follows the refill rule for the lengths the device produced
    want_admit, want_steps = _expected_schedule(L, G, slots, refill, whole_groups)
    assert list(admit) == list(want_admit) and steps == want_steps, (admit, want_admit, steps, want_steps)
    assert len(set(admit.tolist())) > 1, "no refill happened"
    eng.close()


@pytest.mark.parametrize("whole_groups,P", [(1, 16), (0, 16), (0, 20)])
def test_tiny_fp32_eos_without_stop_set_equals_generate(whole_groups, P):
    G, n_prompts, N = 2, 4, 12
    log(f"tiny fp32 eos with an empty stop set against rollout_generate, whole_groups={whole_groups} P={P}")
    cfg = R.model_config("tiny", R.DTYPE_FP32, P, N, 32)  # a KV pool with room for 8 slots and 9 prompt records
    eng = R.Engine(cfg, group_size=G)
    prompts = W.prompts(n_prompts, P, cfg.vocab, seed=21)
    u = W.uniforms(n_prompts * G, N, seed=22)
    tok, L, admit, steps = _run_eos(eng, prompts, G, 8, N, 0.8, 0.9, u, [], 4, whole_groups)
    assert np.all(L == N) and list(admit) == [0] * (n_prompts * G) and steps == 12
    out = torch.full((n_prompts * G, N), -1, dtype=torch.int32, device="cuda:0")
    R.rollout_generate(eng.ctx, to_dev(prompts, torch), n_prompts, P, G, 8, N, 0.8, 0.9, to_dev(u, torch), out)
    eng.synchronize()
    assert np.array_equal(out.cpu().numpy(), tok)
    eng.close()


@pytest.mark.parametrize("refill,slots,whole_groups,P,shared", [
    (1, 8, 1, 40, "1"), (4, 16, 1, 40, "1"), (2, 4, 1, 40, "1"), (2, 8, 1, 40, "2"), (3, 16, 1, 32, "2"),
    (1, 8, 0, 40, "1"), (3, 12, 0, 32, "1"), (2, 5, 0, 40, "2")])
def test_bf16_eos_schedule_and_stop_rule(refill, slots, whole_groups, P, shared, monkeypatch):
    # shared = "2" forces the shared-prefix attention wherever whole groups make it possible
    monkeypatch.setenv("ROLLOUT_SHARED_PREFIX", shared)
    G, n_prompts, N = 4, 7, 24
    log(f"bf16 small GQA eos: {n_prompts} prompts x G={G}, {slots} slots, refill every {refill}, "
        f"whole_groups={whole_groups}, P={P}, shared prefix {shared}")
    cfg = R.model_config(SMALL_BF16, R.DTYPE_BF16, P, N, 2 * slots + G)
    eng = R.Engine(cfg, group_size=G)
    prompts = W.prompts(n_prompts, P, cfg.vocab, seed=61)
    u = W.uniforms(n_prompts * G, N, seed=62)
    stop = list(range(0, cfg.vocab, 16))  # 1 in 16 ids: random-init completions end after ~16 tokens
    tok, L, admit, steps = _run_eos(eng, prompts, G, slots, N, 1.0, 1.0, u, stop, refill, whole_groups)
    _check_structure(tok, L, stop, N, cfg.vocab)
    log(f"  lengths mean {L.mean():.1f} min {L.min()} max {L.max()}; {steps} decode steps")
    eff_slots = min(slots, n_prompts * G) if not whole_groups else min(slots // G, n_prompts) * G
    want_admit, want_steps = _expected_schedule(L, G, eff_slots, refill, whole_groups)
    assert list(admit) == list(want_admit) and steps == want_steps
    assert L.min() < N and len(set(L.tolist())) > 3
    # token 0 of every completion is drawn from its prompt's prefill logits with u[s, 0]: the admission
    # prefills one prompt at a time (M = P rows), so the same prefill through rollout_prefill + rollout_sample
    # runs the same kernels at the same M and must draw the same token, exactly
    logits = torch.empty((G, cfg.vocab), dtype=torch.float32, device="cuda:0")
    first = torch.empty(G, dtype=torch.int32, device="cuda:0")
    want0 = np.empty(n_prompts * G, dtype=np.int32)
    for p in range(n_prompts):
        R.rollout_prefill(eng.ctx, to_dev(prompts[p:p + 1], torch), 1, P, G, logits)
        R.rollout_sample(eng.ctx, logits, G, 1.0, 1.0, to_dev(np.ascontiguousarray(u[p * G:(p + 1) * G, 0]), torch),
                         first)
        eng.synchronize()
        want0[p * G:(p + 1) * G] = first.cpu().numpy()
    log(f"  token 0 equal to the one-prompt prefill's draw: {int(np.sum(want0 == tok[:, 0]))}/{n_prompts * G}")
    assert np.array_equal(want0, tok[:, 0])
    eng.close()


def test_single_refill_rejects_groups_wider_than_the_context():
    # a group's token-0 prefill and draw fill G rows of buffers sized for the context's sequence rows
    cfg = R.model_config("tiny", R.DTYPE_FP32, 8, 4, 4)
    eng = R.Engine(cfg, group_size=1)
    assert eng.cfg.max_seqs_in_flight == 4
    dev = "cuda:0"
    G = 8
    prompts = W.prompts(1, 8, cfg.vocab)
    u = W.uniforms(G, 4)
    tokens = torch.empty((G, 4), dtype=torch.int32, device=dev)
    lengths = torch.empty(G, dtype=torch.int32, device=dev)
    stop = torch.zeros(1, dtype=torch.int32, device=dev)
    with pytest.raises(R.RolloutError, match="ENOMEM"):
        R.rollout_generate_eos(eng.ctx, to_dev(prompts, torch), 1, 8, G, 4, 4, 1.0, 1.0, to_dev(u, torch), stop, 0, 1,
                               0, tokens, lengths)
    eng.synchronize()  # nothing was enqueued; the context stays usable
    eng.close()


def test_single_refill_matches_whole_group_refill_tokens():
    # the same completions, whichever slots and steps serve them
    G, n_prompts, P, N = 2, 6, 20, 14
    cfg = R.model_config("tiny", R.DTYPE_FP32, P, N, 16)
    eng = R.Engine(cfg, group_size=G)
    prompts = W.prompts(n_prompts, P, cfg.vocab, seed=81)
    u = W.uniforms(n_prompts * G, N, seed=82)
    stop = list(range(0, cfg.vocab, 9))
    a = _run_eos(eng, prompts, G, 4, N, 1.0, 1.0, u, stop, 2, 1)
    b = _run_eos(eng, prompts, G, 5, N, 1.0, 1.0, u, stop, 3, 0)
    log(f"  decode steps: whole groups {a[3]}, single completions {b[3]}")
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    eng.close()


def test_length_rewards_and_token_total():
    rng = np.random.default_rng(3)
    L = rng.integers(1, 400, size=300).astype(np.int32)
    rew = torch.empty(300, dtype=torch.float32, device="cuda:0")
    tot = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    R.rollout_length_rewards(to_dev(L, torch), 300, 128, rew, tot)
    torch.cuda.synchronize()
    want = length_target_reward(L, 128).astype(np.float32)
    assert np.array_equal(rew.cpu().numpy(), want)
    assert int(tot.item()) == int(L.sum())


def test_bad_stop_id_is_reported():
    cfg = R.model_config("tiny", R.DTYPE_FP32, 8, 4, 4)
    eng = R.Engine(cfg, group_size=2)
    prompts = W.prompts(2, 8, cfg.vocab)
    u = W.uniforms(4, 4)
    dev = "cuda:0"
    tokens = torch.empty((4, 4), dtype=torch.int32, device=dev)
    lengths = torch.empty(4, dtype=torch.int32, device=dev)
    stop = torch.tensor([3, cfg.vocab + 9], dtype=torch.int32, device=dev)
    R.rollout_generate_eos(eng.ctx, to_dev(prompts, torch), 2, 8, 2, 4, 4, 1.0, 1.0, to_dev(u, torch), stop, 2, 1, 1,
                           tokens, lengths)
    with pytest.raises(R.RolloutError, match="outside"):
        eng.synchronize()
    eng.close()


def test_whole_group_refill_with_groups_wider_than_a_workgroup():
    # G = 260 slots per range: the admission kernel covers them all
    G, n_prompts, P, N = 260, 3, 16, 6
    cfg = R.model_config("tiny", R.DTYPE_FP32, P, N, G)
    eng = R.Engine(cfg, group_size=G)
    prompts = W.prompts(n_prompts, P, cfg.vocab, seed=91)
    u = W.uniforms(n_prompts * G, N, seed=92)
    stop = list(range(0, cfg.vocab, 4))
    tok, L, admit, steps = _run_eos(eng, prompts, G, G, N, 1.0, 1.0, u, stop, 1, 1)
    _check_structure(tok, L, stop, N, cfg.vocab)
    want_admit, want_steps = _expected_schedule(L, G, G, 1, 1)
    assert list(admit) == list(want_admit) and steps == want_steps
    assert sorted(set(admit.tolist())) == sorted(set(want_admit.tolist())) and len(set(admit.tolist())) == 3
    eng.close()
