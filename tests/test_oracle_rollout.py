"""Pins of the multi-wave rollout oracle (oracle/rollout.py).

The central pin is Prop. spec_exact (App. F): trajectories from speculative
waves with first-rejection commit and rollback have the law
prod_t q_t(y_t | y_<t) of sequential exact-q sampling.  The law is enumerated
on a tiny synthetic model (V = 3, L = 3) and compared with the empirical law of
4,000 rollouts by a chi-square test; the same test tells q from p, and a
rollout with a planted rollback mistake fails it.
"""
import numpy as np
import pytest
from scipy.stats import chisquare

from oracle import bridge, coupling, rollout
from paper_2609_36601_amd.workloads import SyntheticAR, SyntheticARTorch

V_LAW, L_LAW, EPS_LAW, N_LAW = 3, 3, 0.2, 4000


def _pvalue(obs, law, n):
    """Chi-square p-value with the cells of expected count < 5 pooled."""
    e = law * n
    keep = e >= 5
    o2, e2 = obs[keep], e[keep]
    if (~keep).any():
        if e[~keep].sum() > 0:
            o2 = np.append(o2, obs[~keep].sum())
            e2 = np.append(e2, e[~keep].sum())
        elif obs[~keep].sum() > 0:
            return 0.0  # outcomes the law gives probability 0
    return chisquare(o2, e2 * (o2.sum() / e2.sum())).pvalue


def _empirical(k, seed):
    m = SyntheticAR(V_LAW, seed=0)
    out = rollout.rollout(m, np.zeros(N_LAW, np.int64), k, L_LAW, EPS_LAW, seed=seed)
    assert (out["length"] == L_LAW).all()
    idx = out["tokens"] @ (V_LAW ** np.arange(L_LAW - 1, -1, -1))
    return np.bincount(idx, minlength=V_LAW ** L_LAW), out


@pytest.fixture(scope="module")
def laws():
    m = SyntheticAR(V_LAW, seed=0)
    q = rollout.sequential_law(m, 0, V_LAW, L_LAW, EPS_LAW).reshape(-1)
    p = rollout.sequential_law(m, 0, V_LAW, L_LAW, 0.0).reshape(-1)
    return q, p


def test_sequential_law_is_a_distribution(laws):
    q, p = laws
    assert abs(q.sum() - 1.0) < 1e-12 and abs(p.sum() - 1.0) < 1e-12
    # the bridge moves the law: the test below can tell q from p
    assert 0.5 * np.abs(q - p).sum() > 0.2


def test_rollout_has_sequential_q_law(laws):
    """Prop. spec_exact, k = 2 drafts per wave."""
    q, p = laws
    obs, out = _empirical(2, seed=11)
    assert out["corrected"].mean() > 0.1  # rejections and rollbacks do happen
    assert _pvalue(obs, q, N_LAW) > 1e-3
    assert _pvalue(obs, p, N_LAW) < 1e-9


def test_planted_rollback_mistake_fails_law(laws, monkeypatch):
    """Continuing from the rejected draft's state instead of the correction's
    keeps the committed tokens right but the next wave's context wrong."""
    q, _ = laws
    monkeypatch.setattr(rollout, "committed_state", lambda model, H, b, m, last: H[m][b])
    obs, _ = _empirical(2, seed=11)
    assert _pvalue(obs, q, N_LAW) < 1e-9


def test_one_draft_per_wave_is_sequential_coupling():
    """With k = 1 every wave is one coupling step at row g = wave * B + b."""
    V, B, L, eps, seed = 40, 6, 5, 0.05, 3
    m = SyntheticAR(V, seed=7)
    out = rollout.rollout(m, np.arange(B), 1, L, eps, seed)
    state = m.initial(np.arange(B))
    for w in range(L):
        s, t = m.logits(state)
        ref = coupling.couple_rows(s, t, eps, seed, row_offset=w * B)
        np.testing.assert_array_equal(out["tokens"][:, w], ref["token"])
        np.testing.assert_array_equal(out["corrected"][:, w], ref["corrected"])
        np.testing.assert_allclose(out["tv"][:, w], ref["tv"], rtol=0, atol=0)
        state = m.advance(state, ref["token"])


def test_metadata_is_token_aligned():
    """Each committed position's metadata equals the bridge at its prefix,
    recomputed by replaying the committed tokens through the model."""
    V, B, L, k, eps, seed = 50, 5, 9, 3, 0.1, 21
    m = SyntheticAR(V, seed=4)
    out = rollout.rollout(m, np.arange(B), k, L, eps, seed)
    assert (out["length"] == L).all()
    for b in range(B):
        state = m.initial(np.array([b]))
        for pos in range(L):
            s, t = m.logits(state)
            br = bridge.bridge_rows(s, t, eps)
            y = out["tokens"][b, pos]
            assert out["lam"][b, pos] == br["lam"][0]
            assert out["tv"][b, pos] == br["tv"][0]
            assert out["kl"][b, pos] == br["kl"][0]
            assert out["logp"][b, pos] == br["logp"][0, y]
            assert out["logt"][b, pos] == br["logpi"][0, y]
            assert out["teacher_argmax"][b, pos] == np.argmax(t[0])
            state = m.advance(state, np.array([y]))


def test_eos_and_max_len():
    V, B, L, k, eps, seed, eos = 6, 40, 7, 3, 0.05, 5, 2
    m = SyntheticAR(V, seed=1)
    out = rollout.rollout(m, np.arange(B), k, L, eps, seed, eos_id=eos)
    assert (out["done"] == rollout.DONE_FINISHED).all()
    ended = 0
    for b in range(B):
        n = out["length"][b]
        toks = out["tokens"][b]
        assert 1 <= n <= L
        assert (toks[n:] == -1).all() and (toks[:n] >= 0).all()
        assert (toks[:n - 1] != eos).all()  # nothing is committed after an EOS
        if n < L:
            assert toks[n - 1] == eos
            ended += 1
        assert np.isnan(out["tv"][b, n:]).all()
    assert ended > 0  # some sequence did stop on EOS
    # without EOS every sequence runs to max_len
    out2 = rollout.rollout(m, np.arange(B), k, L, eps, seed)
    assert (out2["length"] == L).all()
    # identical prefixes up to each sequence's EOS
    for b in range(B):
        n = out["length"][b]
        np.testing.assert_array_equal(out["tokens"][b, :n], out2["tokens"][b, :n])


def test_rollout_waves_commit_at_least_one_token():
    V, B, L, k, eps, seed = 30, 4, 12, 4, 0.05, 9
    m = SyntheticAR(V, seed=2)
    out = rollout.rollout(m, np.arange(B), k, L, eps, seed)
    assert out["waves"] <= L
    assert (out["length"] == L).all()


def test_torch_model_matches_numpy_model():
    torch = pytest.importorskip("torch")
    for seed in (0, 5, 2 ** 63 + 17):
        m = SyntheticAR(33, seed)
        mt = SyntheticARTorch(33, seed)
        h = m.initial(np.arange(7))
        ht = mt.initial(torch.arange(7))
        assert (h.view(np.int64) == ht.numpy()).all()
        tok = (np.arange(7) * 5) % 33
        h2 = m.advance(h, tok)
        h2t = mt.advance(ht, torch.as_tensor(tok))
        assert (h2.view(np.int64) == h2t.numpy()).all()
        s, t = m.logits(h2)
        so = torch.empty(7, 33)
        to = torch.empty(7, 33, dtype=torch.bfloat16)
        mt.logits_into(h2t, so, to)
        assert (so.numpy() == s).all() and (to.float().numpy() == t).all()
