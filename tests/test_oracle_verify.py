"""Pins for the oracle's speculative block verification (Sec. 3.5, App. F, App. I)."""
import itertools

import numpy as np
import pytest
import scipy.stats

from oracle import bridge, coupling, philox, verify


def test_no_rejection_when_student_equals_teacher():
    rng = np.random.default_rng(0)
    s = rng.normal(0, 2, (4 * 8, 100))
    draft = rng.integers(0, 100, 32)
    out = verify.verify_blocks(s, s.copy(), 8, draft, 0.2, seed=5)
    assert out["accepted_len"].tolist() == [8] * 4
    assert out["correction"].tolist() == [-1] * 4


def test_first_rejection_and_per_row_agreement_with_coupling_accept():
    rng = np.random.default_rng(1)
    k, B, V = 6, 40, 64
    s = rng.normal(0, 2, (B * k, V))
    t = rng.normal(0, 2, (B * k, V))
    draft = rng.integers(0, V, B * k)
    out = verify.verify_blocks(s, t, k, draft, 0.3, seed=11, row_offset=100)
    b = bridge.bridge_rows(s, t, 0.3)
    assert (out["accepted_len"] < k).any() and (out["accepted_len"] > 0).any()
    for blk in range(B):
        n = out["accepted_len"][blk]
        for j in range(k):
            r = blk * k + j
            # Eq. accept via the App. I log form, and u from the ACCEPT stream
            a = np.exp(min(0.0, b["logq"][r, draft[r]] - b["logp"][r, draft[r]]))
            u = philox.uniform(11, philox.STREAM_ACCEPT, 100 + r, 0)
            if j < n:
                assert u < a
            elif j == n:
                assert u >= a
                c = out["correction"][blk]
                assert b["logq"][r, c] > b["logp"][r, c]  # residual support
            if j > n:
                assert out["evaluated"][r] == 0
        if n == k:
            assert out["correction"][blk] == -1


def test_eos_in_accepted_prefix_ends_block():
    rng = np.random.default_rng(2)
    k, V = 4, 20
    s = rng.normal(0, 1, (k, V))
    draft = np.array([3, 7, 5, 1])
    out = verify.verify_blocks(s, s.copy(), k, draft, 0.1, seed=1, eos_id=7)
    assert out["accepted_len"].tolist() == [2] and out["correction"].tolist() == [-1]
    # EOS only in the discarded suffix changes nothing
    t = s.copy()
    out2 = verify.verify_blocks(s, t, k, np.array([3, 5, 5, 7]), 0.1, seed=1, eos_id=7)
    out3 = verify.verify_blocks(s, t, k, np.array([3, 5, 5, 7]), 0.1, seed=1, eos_id=-1)
    assert out2["accepted_len"].tolist() == [4] and out3["accepted_len"].tolist() == [4]


def test_bad_draft_and_non_finite_end_block():
    s = np.zeros((6, 10))
    t = np.ones((6, 10))
    t[4, 2] = np.inf
    out = verify.verify_blocks(s, t, 3, np.array([1, 99, 2, 0, 0, 0]), 0.1, seed=0)
    assert out["accepted_len"].tolist() == [1, 1]
    assert out["correction"].tolist() == [-1, -1]


def _toy_logits(prefix, V, which):
    """Deterministic logits of a tiny synthetic autoregressive 'model'."""
    h = 1469598103934665603
    for tok in (which,) + tuple(prefix):
        h = ((h ^ (tok + 1)) * 1099511628211) % (1 << 64)
    rng = np.random.default_rng(h)
    return rng.normal(0, 1.2, V)


def test_block_verify_has_sequential_exact_q_law():
    """App. F: drafting k tokens from the student, verifying them in one block,
    committing through the first rejection plus its correction, and restarting
    from the true prefix gives the law prod_t q_t(y_t | y_<t)."""
    V, L, k, eps = 3, 3, 2, 0.15
    # exact law by enumeration
    prob = {}
    for seq in itertools.product(range(V), repeat=L):
        pr = 1.0
        for i in range(L):
            s = _toy_logits(seq[:i], V, 0)
            t = _toy_logits(seq[:i], V, 1)
            b = bridge.bridge_rows(s[None], t[None], eps)
            pr *= np.exp(b["logq"][0][seq[i]])
        prob[seq] = pr
    assert abs(sum(prob.values()) - 1) < 1e-12
    n = 8000
    rng = np.random.default_rng(123)
    counts = {seq: 0 for seq in prob}
    g = 0
    for trial in range(n):
        y = []
        while len(y) < L:
            kk = min(k, L - len(y))
            drafts, rows_s, rows_t = [], [], []
            pre = list(y)
            for j in range(kk):
                s = _toy_logits(tuple(pre), V, 0)
                t = _toy_logits(tuple(pre), V, 1)
                p = np.exp(bridge.log_softmax(s[None])[0])
                z = int(rng.choice(V, p=p))
                drafts.append(z)
                rows_s.append(s)
                rows_t.append(t)
                pre.append(z)
            out = verify.verify_blocks(np.array(rows_s), np.array(rows_t), kk, np.array(drafts),
                                       eps, seed=77, row_offset=g)
            g += kk
            m = int(out["accepted_len"][0])
            y.extend(drafts[:m])
            if m < kk:
                y.append(int(out["correction"][0]))
        counts[tuple(y[:L])] += 1
    seqs = sorted(prob)
    obs = np.array([counts[q] for q in seqs], float)
    exp = np.array([prob[q] for q in seqs]) * n
    stat = ((obs - exp) ** 2 / exp).sum()
    assert scipy.stats.chi2.sf(stat, len(seqs) - 1) > 1e-5
