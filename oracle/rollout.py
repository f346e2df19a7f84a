"""Multi-wave speculative rollout with exact-q commits, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

SAKI, Sec. 3.5 and the engine-resident q backend (App. I): every wave, for
each unfinished sequence,
  1. the student drafts k tokens autoregressively from its committed prefix,
     z_j ~ p(. | prefix, z_<j);
  2. the teacher and the bridge are evaluated on the k draft prefixes and the
     block is verified with first-rejection semantics (oracle/verify.py);
  3. the accepted drafts, and the correction if one was drawn, are committed;
     every later draft state is discarded, and the next wave starts from the
     new committed prefix;
  4. the per-position metadata the objective needs (token, corrected flag,
     lambda*, KL, TV, log p and log pi of the token, teacher mode) is packed
     in token order.
App. F (Prop. spec_exact) shows the committed trajectory has the law
prod_t q_t(y_t | x, y_<t) of sequential exact-q sampling.

The "model" is any object with
    initial(prompt_ids) -> states       (one state per sequence)
    advance(states, tokens) -> states   (state after appending a token)
    logits(states) -> (s, t)            (student / teacher logits [n, V])
so that the logits at a prefix are a function of its state alone.

Readings fixed here (the paper gives the schedule, not these details):
  * draft z_j of sequence b in wave w is drawn by the two-level race of
    oracle/coupling.py on the proposal streams of global row
    g = w * B * k + b * k + j, the row that also keys the verification of that
    position; so a draft equals the proposal the coupling would make at g;
  * all B sequences keep their rows in every wave (finished ones are drafted
    and verified but commit nothing), so the keys do not depend on which
    sequences are still running;
  * a sequence finishes when it reaches max_len tokens (the wave's commit is
    cut there) or commits eos_id (verification already ends a block at an
    accepted EOS; a correction equal to eos_id ends it too);
  * a wave that commits nothing for an unfinished sequence (a non-finite
    logit or an out-of-vocabulary draft at the block's first position) stops
    that sequence with status 2.
"""
import numpy as np

from . import philox
from .bridge import log_softmax
from .coupling import CHUNK, exponential_race
from .verify import verify_blocks

DONE_RUNNING = 0
DONE_FINISHED = 1
DONE_STOPPED = 2


def draft_tokens(s, seed, row_offset, row_step, chunk=CHUNK):
    """z_r ~ softmax(s_r) by the two-level race keyed by g = row_offset + r * row_step.

    Rows with a non-finite logit give -1.  Returns (tokens, chunk gaps, entry gaps).
    """
    s = np.atleast_2d(np.asarray(s, np.float64))
    n = s.shape[0]
    z = np.full(n, -1, np.int64)
    gaps = np.full((n, 2), np.inf)
    for r in range(n):
        if not np.isfinite(s[r]).all():
            continue
        g = row_offset + r * row_step
        z[r], _, gaps[r, 0], gaps[r, 1] = exponential_race(
            log_softmax(s[r]), seed, g, philox.STREAM_PROP_CHUNK, philox.STREAM_PROP_ELEM, chunk)
    return z, gaps[:, 0], gaps[:, 1]


def committed_state(model, H, b, m, last):
    """State after m committed tokens of sequence b, the last being `last`.

    H[j][b] is the state after the first j drafts.  Accepted drafts are the
    draft path itself; a correction replaces the draft at its position, so the
    state is rebuilt from the prefix before it and every later draft state is
    dropped (rollback).
    """
    return model.advance(np.array([H[m - 1][b]]), np.array([last]))[0]


def rollout(model, prompts, k, max_len, eps, seed, eos_id=-1, chunk=CHUNK, max_waves=None):
    """Runs waves until every sequence is finished.

    Returns a dict with
      tokens [B, max_len] (-1 past the end), corrected, lam, kl, tv, logp,
      logt, teacher_argmax (same shape, token-aligned), length [B], done [B],
      waves (number of waves run), and min_margin [B]: the smallest decision
      margin seen in the committed part of each sequence (the accept margin
      |u - alpha| and the relative key gaps of the draft and correction
      races), which says how close a sequence came to a different path.
    """
    prompts = np.asarray(prompts)
    B = prompts.shape[0]
    state = model.initial(prompts)
    tokens = np.full((B, max_len), -1, np.int64)
    corrected = np.zeros((B, max_len), np.int64)
    teacher_argmax = np.full((B, max_len), -1, np.int64)
    meta = {key: np.full((B, max_len), np.nan) for key in ("lam", "kl", "tv", "logp", "logt")}
    length = np.zeros(B, np.int64)
    done = np.zeros(B, np.int64)
    min_margin = np.full(B, np.inf)
    if max_len <= 0:
        done[:] = DONE_FINISHED
    wave = 0
    limit = max_waves if max_waves is not None else max_len + 1
    while (done == DONE_RUNNING).any() and wave < limit:
        g0 = wave * B * k
        # 1. drafting from the committed prefixes
        H = [state]
        S = []
        Z = []
        draft_gap = []
        for j in range(k):
            s_j, _ = model.logits(H[j])
            z_j, gc, ge = draft_tokens(s_j, seed, g0 + j, k, chunk)
            S.append(s_j)
            Z.append(z_j)
            draft_gap.append(np.minimum(gc, ge))
            H.append(model.advance(H[j], np.where(z_j >= 0, z_j, 0)))
        # 2. teacher on the draft prefixes, block-major rows b * k + j
        states_bk = np.stack(H[:k], axis=1).reshape(-1)
        s_bk, t_bk = model.logits(states_bk)
        drafts = np.stack(Z, axis=1).reshape(-1)
        v = verify_blocks(s_bk, t_bk, k, drafts, eps, seed, row_offset=g0, eos_id=eos_id,
                          chunk=chunk)
        logpi = np.stack([log_softmax(t_bk[r]) if np.isfinite(t_bk[r]).all()
                          else np.full(t_bk.shape[1], np.nan) for r in range(B * k)])
        dgap = np.stack(draft_gap, axis=1).reshape(-1)
        # 3-4. commit up to the first rejection, token-aligned metadata
        new_state = state.copy()
        for b in range(B):
            if done[b] != DONE_RUNNING:
                continue
            n = int(v["accepted_len"][b])
            c = int(v["correction"][b])
            commit = [int(drafts[b * k + j]) for j in range(n)] + ([c] if c >= 0 else [])
            commit = commit[:max_len - length[b]]
            if not commit:
                done[b] = DONE_STOPPED
                continue
            for j, y in enumerate(commit):
                r = b * k + j
                pos = length[b] + j
                tokens[b, pos] = y
                corrected[b, pos] = 1 if j == n else 0
                meta["lam"][b, pos] = v["lam"][r]
                meta["kl"][b, pos] = v["kl"][r]
                meta["tv"][b, pos] = v["tv"][r]
                meta["logp"][b, pos] = v["logp"][r, y]
                meta["logt"][b, pos] = logpi[r, y]
                teacher_argmax[b, pos] = int(np.argmax(t_bk[r]))
                m = min(v["margin"][r], dgap[r])
                if j == n:
                    m = min(m, v["gaps"][b, 0], v["gaps"][b, 1])
                min_margin[b] = min(min_margin[b], m)
            m = len(commit)
            new_state[b] = committed_state(model, H, b, m, commit[-1])
            length[b] += m
            if length[b] >= max_len or (eos_id >= 0 and commit[-1] == eos_id):
                done[b] = DONE_FINISHED
        state = new_state
        wave += 1
    out = dict(tokens=tokens, corrected=corrected, teacher_argmax=teacher_argmax, length=length,
               done=done, waves=wave, min_margin=min_margin)
    out.update(meta)
    return out


def sequential_law(model, prompt, V, L, eps):
    """Exact law of y_1..y_L under sequential q sampling (Prop. spec_exact).

    Enumerates every prefix of length < L; returns an array [V] * L of
    prod_t q_t(y_t | y_<t), with q_t the bridge at lambda* of that prefix.
    """
    from .bridge import bridge_rows
    law = np.zeros((V,) * L)
    state0 = model.initial(np.array([prompt]))

    def walk(state, prefix, prob):
        if len(prefix) == L:
            law[tuple(prefix)] = prob
            return
        s, t = model.logits(state)
        q = np.exp(bridge_rows(s, t, eps)["logq"][0])
        for y in range(V):
            walk(model.advance(state, np.array([y])), prefix + [y], prob * q[y])

    walk(state0, [], 1.0)
    return law


__all__ = ["committed_state", "draft_tokens", "rollout", "sequential_law", "DONE_RUNNING", "DONE_FINISHED",
           "DONE_STOPPED"]
