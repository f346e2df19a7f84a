"""Speculative block verification with first-rejection semantics, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

SAKI, Sec. 3.5 and App. I: the student drafts up to k tokens; for every
block position the bridge q_j and the acceptance alpha_j(z_j) =
exp(min(0, log q_j(z_j) - log p_j(z_j))) are formed; the longest
consecutively accepted prefix is committed (a running product of the
acceptance indicators); at the first rejection j a correction is drawn from
[q_j - p_j]_+ and committed, and every later position is discarded.  App. F
proves this has the law of sequential exact-q sampling.

Rows are block-major: row b*k + j is position j of block b, with global row
index g = row_offset + b*k + j, which keys that position's uniforms.

Readings where the paper is silent (it tests "EOS in discarded suffixes"
without defining it):
  * when all k drafts are accepted there is no correction (-1) and no bonus
    token;
  * with eos_id >= 0, an accepted draft equal to eos_id at position j < n
    ends the block there: n = j + 1 and no correction is drawn;
  * a position with non-finite logits (status 1) or a draft outside the
    vocabulary (status 2) ends the block before it: n = j, no correction.
"""
import numpy as np

from . import philox
from .bridge import bridge_rows
from .coupling import residual_draw, CHUNK


def verify_blocks(s, t, k, draft, eps, seed, row_offset=0, eos_id=-1, chunk=CHUNK):
    """Returns dict: accepted_len [B], correction [B], and per-position arrays
    lam, kl, tv, accept_prob, u, margin, accepted (0/1), evaluated (0/1).
    Positions are examined in order and the bridge is formed only at the
    positions a block reaches (up to its first rejection): the per-position
    values of positions after that are NaN."""
    s = np.atleast_2d(np.asarray(s, np.float64))
    t = np.atleast_2d(np.asarray(t, np.float64))
    n_rows, V = s.shape
    assert n_rows % k == 0
    B = n_rows // k
    draft = np.asarray(draft, np.int64)
    finite = np.isfinite(s).all(axis=1) & np.isfinite(t).all(axis=1)
    ok_draft = (draft >= 0) & (draft < V)
    good = finite & ok_draft
    lam = np.full(n_rows, np.nan)
    kl = np.full(n_rows, np.nan)
    tv = np.full(n_rows, np.nan)
    alpha = np.full(n_rows, np.nan)
    u = np.full(n_rows, np.nan)
    logp = np.full((n_rows, V), np.nan)
    logq = np.full((n_rows, V), np.nan)
    accepted = np.zeros(n_rows, np.int64)
    evaluated = np.zeros(n_rows, np.int64)
    acc_len = np.empty(B, np.int64)
    corr = np.full(B, -1, np.int64)
    gaps = np.full((B, 2), np.inf)
    for blk in range(B):
        n = k
        draw = False
        for j in range(k):
            r = blk * k + j
            if not good[r]:
                n = j
                break
            evaluated[r] = 1
            b = bridge_rows(s[r:r + 1], t[r:r + 1], eps)
            lam[r], kl[r], tv[r] = b["lam"][0], b["kl"][0], b["tv"][0]
            logp[r], logq[r] = b["logp"][0], b["logq"][0]
            z = draft[r]
            alpha[r] = np.exp(min(0.0, logq[r, z] - logp[r, z]))
            u[r] = philox.uniform(seed, philox.STREAM_ACCEPT, row_offset + r, 0)
            if u[r] < alpha[r]:
                accepted[r] = 1
                if eos_id >= 0 and draft[r] == eos_id:
                    n = j + 1
                    break
            else:
                n = j
                draw = True
                break
        acc_len[blk] = n
        if draw:
            r = blk * k + n
            c, gp = residual_draw(logp[r], logq[r], seed, row_offset + r, chunk)
            corr[blk] = c
            gaps[blk] = gp
    return dict(accepted_len=acc_len, correction=corr, lam=lam, kl=kl, tv=tv,
                accept_prob=alpha, u=u, margin=np.abs(u - alpha), accepted=accepted,
                evaluated=evaluated, good=good, gaps=gaps, logp=logp, logq=logq)
