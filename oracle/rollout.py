"""Oracle rollout: G sampled completions per prompt, then group advantages.

TEST INFRASTRUCTURE ONLY (see the package header).

The rollout phase of a GRPO step (section 3, "Background"): for each of B
prompts, G completions.  Readings where the paper is silent:

* Sequence order is group-major, s = p * G + g, so each group is contiguous
  (section 4.3 keeps the generation batch a multiple of G).
* Each prompt is run once and its cache and last-position logits are shared
  by the G completions; this equals running the G copies separately because
  the forward pass is deterministic.
* Token 0 of every completion is drawn from the prompt's logits with
  u[s, 0]; token t >= 1 comes from a decode step that feeds token t - 1 at
  position P + t - 1 and draws with u[s, t].  Exactly N tokens, no EOS.
"""
from __future__ import annotations

import copy

import numpy as np

from .grpo import grpo_advantages
from .sampler import sample_batch


def rollout(model, prompts: np.ndarray, group_size: int, max_new_tokens: int, temperature: float,
            top_p: float, uniforms: np.ndarray, keep_logits: bool = True, rewards=None,
            adv_eps: float = 0.0, adv_ddof: int = 1) -> dict:
    """Run the cached rollout.

    prompts int [B, P]; uniforms fp32 [B*G, N].  Returns a dict with
    ``tokens`` int32 [S, N], ``margins`` float64 [S, N], ``logits`` float64
    [N, S, V] (when keep_logits), and, when rewards are given,
    ``advantages`` and ``zero_var_groups``.
    """
    prompts = np.asarray(prompts)
    n_prompts = prompts.shape[0]
    s_total = n_prompts * group_size
    n = max_new_tokens
    tokens = np.zeros((s_total, n), dtype=np.int32)
    margins = np.zeros((s_total, n), dtype=np.float64)
    logits_all = [] if keep_logits else None

    caches = []
    logits = np.empty((s_total, model.shape.vocab), dtype=np.float64)
    for p in range(n_prompts):
        cache, lg = model.prefill(prompts[p])
        for g in range(group_size):
            caches.append(copy.deepcopy(cache) if g else cache)
            logits[p * group_size + g] = lg
    for t in range(n):
        if keep_logits:
            logits_all.append(logits.copy())
        tokens[:, t], margins[:, t] = sample_batch(logits, temperature, top_p, uniforms[:, t])
        if t + 1 < n:
            for s in range(s_total):
                logits[s] = model.decode(caches[s], int(tokens[s, t]))
    out = {"tokens": tokens, "margins": margins}
    if keep_logits:
        out["logits"] = np.stack(logits_all)
    if rewards is not None:
        out["advantages"], out["zero_var_groups"] = grpo_advantages(rewards, group_size, adv_eps, adv_ddof)
    return out
