"""Oracle for stop-token-terminated completions under continuous batching.

TEST INFRASTRUCTURE ONLY (see the package header).

The paper's controller counts T_k, the non-padding tokens a generation batch
produced (section 4.5, the objective of eq. 4), and its runs score completions
with a reward for closeness to a 128-token length target (section 5).  Both
presuppose completions of different lengths, which end when the model emits a
stop token.  The paper fixes neither the stop rule, nor how a batch of
variable-length completions is scheduled, nor the reward formula.  Readings
taken here (listed in the design notes as well):

* Stop rule.  A completion draws exactly as in ``rollout`` (token t with
  uniform u[s, t]) and ends after drawing a token of the stop set, which is
  kept as its last token, or after ``max_new_tokens`` tokens.  Its length L
  counts the stop token; positions t >= L hold the pad value -1.
* Continuous batching.  ``seqs_in_flight`` slots are refilled as completions
  end; the host inspects them every ``refill_interval`` decode steps (the
  boundaries are the multiples of R).  Two granularities:
  - whole groups: slot ranges of G hold one group each (section 4.3 keeps the
    batch a multiple of G); a range whose G completions have all ended takes
    the next prompt's group, which is prefilled and draws its token 0 there;
  - single completions: a slot whose completion has ended takes the next
    completion in order s = p * G + g (a group's prompt is prefilled when its
    first completion is admitted, and every member draws token 0 from those
    logits); freed slots are filled in slot order.
  The rollout ends at the first boundary where everything has been admitted
  and has ended.  Per completion the tokens do not depend on the schedule:
  only its prompt, its own uniforms and the model enter them.
* Length-target reward.  r = 1 - min(1, |L - L*| / L*) for target L*: 1 at
  the target, falling linearly to 0 at distance L*.

Parity: ``rollout_eos`` is pinned against the plain rollout truncated at the
first stop token (an independent code path) and against the empty and full
stop sets; ``continuous_schedule`` against a step-by-step simulation of the
slots and hand-worked schedules (``tests/golden/batching_schedule.txt``);
``sequence_schedule`` against ``simulate_sequence_slots`` (a step simulation that
also tracks each group's prompt record) and a hand-worked case;
``length_target_reward`` against its closed-form points.  All in
``tests/test_oracle_batching.py``.
"""
from __future__ import annotations

import copy

import numpy as np

from .sampler import sample_row

PAD = -1


def rollout_eos(model, prompts: np.ndarray, group_size: int, max_new_tokens: int, temperature: float,
                top_p: float, uniforms: np.ndarray, stop_ids) -> dict:
    """Completions that end at the first drawn stop token (or after max_new_tokens).

    prompts int [B, P]; uniforms fp32 [B*G, N] indexed by completion s = p*G + g and token t.
    Returns ``tokens`` int32 [S, N] (PAD after the end), ``lengths`` int32 [S] and ``margins``
    float64 [S, N] (inf after the end).
    """
    prompts = np.asarray(prompts)
    stop = set(int(t) for t in np.asarray(stop_ids).reshape(-1))
    n_prompts = prompts.shape[0]
    n = max_new_tokens
    s_total = n_prompts * group_size
    tokens = np.full((s_total, n), PAD, dtype=np.int32)
    lengths = np.zeros(s_total, dtype=np.int32)
    margins = np.full((s_total, n), np.inf, dtype=np.float64)
    for p in range(n_prompts):
        cache0, logits0 = model.prefill(prompts[p])
        for g in range(group_size):
            s = p * group_size + g
            cache = copy.deepcopy(cache0)
            logits = logits0
            t = 0
            while True:
                tok, margin = sample_row(logits, temperature, top_p, float(uniforms[s, t]))
                tokens[s, t] = tok
                margins[s, t] = margin
                t += 1
                if tok in stop or t == n:
                    break
                logits = model.decode(cache, tok)
            lengths[s] = t
    return {"tokens": tokens, "lengths": lengths, "margins": margins}


def sequence_schedule(lengths, slots: int, refill_interval: int) -> dict:
    """Single-completion refill: admission and release boundary of every completion, and the steps in all.

    Same rule as ``continuous_schedule`` with ranges of one completion: a completion admitted at b ends
    at step b + L - 1 and its slot is seen free at b + R * max(1, ceil((L - 1) / R)).
    """
    lengths = np.asarray(lengths).reshape(-1)
    return continuous_schedule(lengths, 1, slots, refill_interval)


def continuous_schedule(lengths, group_size: int, slot_groups: int, refill_interval: int) -> dict:
    """Admission boundary of every group and the decode steps the rollout takes.

    lengths int [n_groups * G]; ``slot_groups`` slot ranges of G; boundaries are the multiples of
    ``refill_interval`` decode steps.  A group admitted at boundary b draws token 0 there and token
    t at decode step b + t, so it ends at step f = b + max(L) - 1; its slot range is seen free at the
    first checked boundary after b that is >= f, i.e. b + R * max(1, ceil((f - b) / R)).
    Returns ``admit`` int [n_groups], ``free`` int [n_groups] (the boundary each group is seen
    ended) and ``steps`` (decode steps in all).
    """
    lengths = np.asarray(lengths).reshape(-1, group_size)
    n_groups = lengths.shape[0]
    R = int(refill_interval)
    admit = np.full(n_groups, -1, dtype=np.int64)
    free = np.full(n_groups, -1, dtype=np.int64)
    # event list of slot ranges: (boundary at which the range is seen free, range index)
    nxt = 0
    ready = []
    for k in range(min(slot_groups, n_groups)):
        ready.append((0, k))
    while ready:
        ready.sort()
        b, k = ready.pop(0)
        if nxt >= n_groups:
            continue
        grp = nxt
        nxt += 1
        admit[grp] = b
        span = int(lengths[grp].max()) - 1  # decode steps until its last draw
        seen = b + R * max(1, -(-span // R))
        free[grp] = seen
        ready.append((seen, k))
    steps = int(free.max()) if n_groups else 0
    return {"admit": admit, "free": free, "steps": steps}


def simulate_slots(lengths, group_size: int, slot_groups: int, refill_interval: int) -> dict:
    """Step-by-step simulation of the same slot machine (a second, independent route to the schedule).

    Every slot holds (completion, tokens drawn so far); each decode step every live slot draws one
    token; at every multiple of ``refill_interval`` the host scans the slot ranges in order and refills
    each whose completions have all ended.
    """
    lengths = np.asarray(lengths).reshape(-1)
    n_groups = lengths.size // group_size
    R = int(refill_interval)
    slots = [None] * slot_groups  # (group, drawn[G]) or None
    admit = np.full(n_groups, -1, dtype=np.int64)
    free = np.full(n_groups, -1, dtype=np.int64)
    nxt = 0

    def admit_into(k, step):
        nonlocal nxt
        g0 = nxt
        nxt += 1
        admit[g0] = step
        slots[k] = (g0, [1] * group_size)  # token 0 comes from the prefill logits

    for k in range(slot_groups):
        if nxt < n_groups:
            admit_into(k, 0)
    step = 0
    while any(sl is not None for sl in slots):
        for _ in range(R):
            step += 1
            for sl in slots:
                if sl is None:
                    continue
                grp, drawn = sl
                for j in range(group_size):
                    if drawn[j] < lengths[grp * group_size + j]:
                        drawn[j] += 1
        for k in range(slot_groups):
            sl = slots[k]
            if sl is None:
                continue
            grp, drawn = sl
            if all(drawn[j] >= lengths[grp * group_size + j] for j in range(group_size)):
                free[grp] = step
                slots[k] = None
                if nxt < n_groups:
                    admit_into(k, step)
    return {"admit": admit, "free": free, "steps": step}


def simulate_sequence_slots(lengths, group_size: int, slots: int, refill_interval: int) -> dict:
    """Step-by-step simulation of single-completion refill, tracking groups and their prompt records.

    Besides the schedule it reports the most prompt records (a group's shared prompt cache, alive from
    its first admission until its last completion ends) held at once, which sizes the KV pool.
    """
    lengths = np.asarray(lengths).reshape(-1)
    n = lengths.size
    R = int(refill_interval)
    slot = [-1] * slots
    drawn = [0] * slots
    admit = np.full(n, -1, dtype=np.int64)
    free = np.full(n, -1, dtype=np.int64)
    ended = {}
    live_groups = set()
    most = 0
    nxt = 0

    def admit_into(r, step):
        nonlocal nxt, most
        s = nxt
        nxt += 1
        admit[s] = step
        slot[r] = s
        drawn[r] = 1
        live_groups.add(s // group_size)
        most = max(most, len(live_groups))

    for r in range(slots):
        if nxt < n:
            admit_into(r, 0)
    step = 0
    while any(x >= 0 for x in slot):
        for _ in range(R):
            step += 1
            for r in range(slots):
                if slot[r] >= 0 and drawn[r] < lengths[slot[r]]:
                    drawn[r] += 1
        for r in range(slots):
            s = slot[r]
            if s < 0 or drawn[r] < lengths[s]:
                continue
            free[s] = step
            slot[r] = -1
            p = s // group_size
            ended[p] = ended.get(p, 0) + 1
            if ended[p] == group_size:
                live_groups.discard(p)
            if nxt < n:
                admit_into(r, step)
    return {"admit": admit, "free": free, "steps": step, "most_records": most}


def length_target_reward(lengths, target: int = 128) -> np.ndarray:
    """r = 1 - min(1, |L - target| / target), float64."""
    L = np.asarray(lengths, dtype=np.float64)
    return 1.0 - np.minimum(1.0, np.abs(L - target) / float(target))
