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


def commit_wave(traj, k, eos_id, accepted_len, correction, per_pos):
    """First-rejection commit of one wave into token-aligned trajectories.

    traj: dict of numpy arrays tokens, corrected, teacher_argmax, lam, kl, tv,
    logp, logt ([B, max_len]), length and done ([B]), updated in place.
    per_pos: dict of [B * k] arrays token (the committed token of each
    verified position: the draft where accepted, the correction where
    rejected), lam, kl, tv, logp, logt, teacher_argmax.
    For each running sequence b the n = accepted_len[b] accepted drafts and,
    if n < k and correction[b] >= 0, the correction are appended, cut at
    max_len; later positions of the block are dropped.  Returns the number m
    committed per sequence (0 for sequences not running).
    """
    B = traj["length"].shape[0]
    max_len = traj["tokens"].shape[1]
    n_commit = np.zeros(B, np.int64)
    for b in range(B):
        if traj["done"][b] != DONE_RUNNING:
            continue
        length = int(traj["length"][b])
        if length < 0 or length > max_len:
            traj["done"][b] = DONE_STOPPED
            continue
        n = min(max(int(accepted_len[b]), 0), k)
        want = n + (1 if n < k and correction[b] >= 0 else 0)
        m = min(want, max_len - length)
        for j in range(m):
            r = b * k + j
            pos = length + j
            traj["tokens"][b, pos] = per_pos["token"][r]
            traj["corrected"][b, pos] = 1 if j == n else 0
            for key in ("lam", "kl", "tv", "logp", "logt", "teacher_argmax"):
                traj[key][b, pos] = per_pos[key][r]
        traj["length"][b] = length + m
        n_commit[b] = m
        if m == 0:
            traj["done"][b] = DONE_STOPPED
        elif length + m >= max_len or (eos_id >= 0 and per_pos["token"][b * k + m - 1] == eos_id):
            traj["done"][b] = DONE_FINISHED
    return n_commit


def new_trajectories(B, max_len):
    traj = dict(tokens=np.full((B, max_len), -1, np.int64),
                corrected=np.zeros((B, max_len), np.int64),
                teacher_argmax=np.full((B, max_len), -1, np.int64),
                length=np.zeros(B, np.int64), done=np.zeros(B, np.int64),
                margin=np.full((B, max_len), np.nan))
    for key in ("lam", "kl", "tv", "logp", "logt"):
        traj[key] = np.full((B, max_len), np.nan)
    if max_len <= 0:
        traj["done"][:] = DONE_FINISHED
    return traj


def rollout(model, prompts, k, max_len, eps, seed, eos_id=-1, chunk=CHUNK, max_waves=None):
    """Runs waves until every sequence is finished.

    Returns the trajectories of commit_wave (tokens, corrected,
    teacher_argmax, lam, kl, tv, logp, logt [B, max_len], -1 / NaN past the
    end; length, done [B]), plus waves (the number of waves run) and margin
    [B, max_len]: the smallest decision margin behind each committed token
    (the accept margin |u - alpha| and the relative key gap of the draft race
    at that position, and at a correction the key gaps of the residual race),
    which says how close the sequence came to a different path there.
    """
    prompts = np.asarray(prompts)
    B = prompts.shape[0]
    state = model.initial(prompts)
    traj = new_trajectories(B, max_len)
    wave = 0
    limit = max_waves if max_waves is not None else max_len + 1
    while (traj["done"] == DONE_RUNNING).any() and wave < limit:
        g0 = wave * B * k
        # 1. drafting from the committed prefixes
        H = [state]
        Z = []
        draft_gap = []
        for j in range(k):
            s_j, _ = model.logits(H[j])
            z_j, gc, ge = draft_tokens(s_j, seed, g0 + j, k, chunk)
            Z.append(z_j)
            draft_gap.append(np.minimum(gc, ge))
            H.append(model.advance(H[j], np.where(z_j >= 0, z_j, 0)))
        # 2. teacher on the draft prefixes, block-major rows b * k + j
        states_bk = np.stack(H[:k], axis=1).reshape(-1)
        s_bk, t_bk = model.logits(states_bk)
        drafts = np.stack(Z, axis=1).reshape(-1)
        v = verify_blocks(s_bk, t_bk, k, drafts, eps, seed, row_offset=g0, eos_id=eos_id,
                          chunk=chunk)
        # per-position token and metadata of the verified positions
        R = B * k
        token = drafts.copy()
        margin = np.minimum(v["margin"], np.stack(draft_gap, axis=1).reshape(-1))
        for b in range(B):
            if v["correction"][b] >= 0:
                r = b * k + v["accepted_len"][b]
                token[r] = v["correction"][b]
                margin[r] = min(margin[r], v["gaps"][b, 0], v["gaps"][b, 1])
        idx = np.clip(token, 0, t_bk.shape[1] - 1)
        logpi = np.stack([log_softmax(t_bk[r]) if np.isfinite(t_bk[r]).all()
                          else np.full(t_bk.shape[1], np.nan) for r in range(R)])
        per_pos = dict(token=token, lam=v["lam"], kl=v["kl"], tv=v["tv"],
                       logp=v["logp"][np.arange(R), idx], logt=logpi[np.arange(R), idx],
                       teacher_argmax=np.argmax(t_bk, axis=1), margin=margin)
        # 3-4. commit up to the first rejection, token-aligned metadata
        length0 = traj["length"].copy()
        n_commit = commit_wave(traj, k, eos_id, v["accepted_len"], v["correction"], per_pos)
        new_state = state.copy()
        for b in range(B):
            m = int(n_commit[b])
            if m > 0:
                traj["margin"][b, length0[b]:length0[b] + m] = margin[b * k:b * k + m]
                new_state[b] = committed_state(model, H, b, m, int(token[b * k + m - 1]))
        state = new_state
        wave += 1
    traj["waves"] = wave
    return traj


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


__all__ = ["commit_wave", "committed_state", "draft_tokens", "new_trajectories", "rollout", "sequential_law", "DONE_RUNNING", "DONE_FINISHED",
           "DONE_STOPPED"]
