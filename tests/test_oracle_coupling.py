"""Pins for the oracle's maximal coupling (Sec. 3.3, Prop. 1, App. D, App. E).

Laws are checked by Monte Carlo over many global rows (each row has its own
Philox stream) with chi-square / binomial bounds at about the 1e-5 level,
and identities by exact enumeration on tiny vocabularies.
"""
import numpy as np
import pytest
import scipy.special
import scipy.stats

from oracle import bridge, coupling, philox


def _chi2_ok(counts, probs, alpha=1e-5):
    counts = np.asarray(counts, float)
    probs = np.asarray(probs, float)
    keep = probs > 0
    assert counts[~keep].sum() == 0, "mass outside the support"
    if keep.sum() == 1:
        return True
    exp = probs[keep] * counts.sum()
    stat = ((counts[keep] - exp) ** 2 / exp).sum()
    return scipy.stats.chi2.sf(stat, keep.sum() - 1) > alpha


def _binom_ok(k, n, p, alpha=1e-5):
    lo = scipy.stats.binom.ppf(alpha / 2, n, p)
    hi = scipy.stats.binom.isf(alpha / 2, n, p)
    return lo <= k <= hi


@pytest.mark.parametrize("chunk", [4, 3])
def test_two_level_race_law(chunk):
    # hierarchical race with small chunks: the winner has law w / sum(w)
    w = np.array([0.05, 0.3, 0.0, 0.1, 0.02, 0.2, 0.08, 0.0, 0.15, 0.1])
    with np.errstate(divide="ignore"):
        log_w = np.log(w)
    n = 20000
    counts = np.zeros(len(w))
    for g in range(n):
        v, _, _, _ = coupling.exponential_race(log_w, 7, g, 0, 1, chunk=chunk)
        counts[v] += 1
    assert _chi2_ok(counts, w / w.sum())


def test_race_chunk_level_law_at_full_chunk_size():
    # V = 3000 (3 chunks of 1024 plus a ragged one): the winning chunk has law W_c
    rng = np.random.default_rng(1)
    s = rng.normal(0, 2, 3000)
    logp = bridge.log_softmax(s[None])[0]
    n_chunks = 3
    Wc = np.array([np.exp(logp[c * 1024:(c + 1) * 1024]).sum() for c in range(n_chunks)])
    counts = np.zeros(n_chunks)
    for g in range(12000):
        _, c, _, _ = coupling.exponential_race(logp, 3, g, 0, 1)
        counts[c] += 1
    assert _chi2_ok(counts, Wc)


def _tiny_rows(seed=0, V=6, corr=0.2, scale=1.5):
    rng = np.random.default_rng(seed)
    s = rng.normal(0, scale, V)
    t = corr * s + np.sqrt(1 - corr ** 2) * rng.normal(0, scale, V)
    return s, t


def test_accept_probability_enumeration_equals_one_minus_tv():
    # Prop. 1: sum_z p(z) min(1, q(z)/p(z)) = 1 - TV(p, q)
    for seed in range(5):
        s, t = _tiny_rows(seed)
        b = bridge.bridge_rows(s[None], t[None], 0.1)
        p, q = np.exp(b["logp"][0]), np.exp(b["logq"][0])
        alpha = np.exp(np.minimum(0.0, b["logq"][0] - b["logp"][0]))
        assert np.sum(p * alpha) == pytest.approx(1.0 - b["tv"][0], abs=1e-14)
        assert np.sum(np.minimum(p, q)) == pytest.approx(1.0 - b["tv"][0], abs=1e-14)


@pytest.fixture(scope="module")
def mc_run():
    s, t = _tiny_rows(3, V=6, corr=0.0, scale=0.8)
    n = 40000
    out = coupling.couple_rows(np.tile(s, (n, 1)), np.tile(t, (n, 1)), 0.1, seed=2024)
    b = bridge.bridge_rows(s[None], t[None], 0.1)
    return s, t, out, np.exp(b["logp"][0]), np.exp(b["logq"][0]), b["tv"][0]


def test_correction_rate_equals_tv(mc_run):
    _, _, out, p, q, tv = mc_run
    n = len(out["corrected"])
    assert 0.05 < tv < 0.5
    assert _binom_ok(int(out["corrected"].sum()), n, tv)


def test_output_marginal_is_q(mc_run):
    # Prop. 1: the coupled output has marginal q
    _, _, out, p, q, _ = mc_run
    assert _chi2_ok(np.bincount(out["token"], minlength=len(q)), q)


def test_proposal_marginal_is_p(mc_run):
    _, _, out, p, q, _ = mc_run
    assert _chi2_ok(np.bincount(out["proposal"], minlength=len(p)), p)


def test_conditional_laws_on_correction(mc_run):
    # App. D: Pr(Z = v | C = 1) = [p - q]_+ / TV and Pr(Y = v | C = 1) = [q - p]_+ / TV
    _, _, out, p, q, tv = mc_run
    c = out["corrected"] == 1
    assert _chi2_ok(np.bincount(out["proposal"][c], minlength=len(p)), np.maximum(p - q, 0) / tv)
    assert _chi2_ok(np.bincount(out["token"][c], minlength=len(p)), np.maximum(q - p, 0) / tv)
    # residual support: only tokens with log(pi/p) above the App. E threshold
    assert np.all(q[out["token"][c]] > p[out["token"][c]])


def test_accepted_token_is_proposal_and_pinsker(mc_run):
    _, _, out, p, q, tv = mc_run
    a = out["corrected"] == 0
    assert np.array_equal(out["token"][a], out["proposal"][a])
    assert tv <= np.sqrt(out["kl"][0] / 2) <= np.sqrt(0.1 / 2) + 1e-12


def test_eps_zero_never_corrects():
    rng = np.random.default_rng(5)
    s = rng.normal(0, 3, (64, 50))
    t = rng.normal(0, 3, (64, 50))
    out = coupling.couple_rows(s, t, 0.0, seed=1)
    assert np.all(out["lam"] == 0) and np.all(out["corrected"] == 0)
    # q = p up to the float64 rounding of the normaliser Z(0) = sum p
    assert np.all(out["accept_prob"] >= 1.0 - 1e-15) and np.all(out["tv"] < 1e-15)
    assert np.array_equal(out["token"], out["proposal"])


def test_teacher_argmax_lowest_index_on_ties():
    s = np.zeros((2, 8))
    t = np.array([[0, 3, 1, 3, 2, 3, 0, 0], [5, 5, 5, 5, 5, 5, 5, 5]], float)
    out = coupling.couple_rows(s, t, 0.1, seed=0)
    assert out["teacher_argmax"].tolist() == [1, 0]


def test_determinism_and_row_offset_invariance():
    rng = np.random.default_rng(8)
    s = rng.normal(0, 2, (20, 2500))
    t = 0.5 * s + rng.normal(0, 2, (20, 2500))
    full = coupling.couple_rows(s, t, 0.3, seed=77)
    again = coupling.couple_rows(s, t, 0.3, seed=77)
    part = coupling.couple_rows(s[7:15], t[7:15], 0.3, seed=77, row_offset=7)
    for key in ("proposal", "token", "corrected", "lam", "tv"):
        assert np.array_equal(full[key], again[key])
        assert np.array_equal(full[key][7:15], part[key])
    other = coupling.couple_rows(s, t, 0.3, seed=78)
    assert not np.array_equal(full["proposal"], other["proposal"])


def test_non_finite_rows_flagged():
    s = np.zeros((3, 10))
    t = np.ones((3, 10))
    s[1, 4] = np.inf
    t[2, 0] = np.nan
    out = coupling.couple_rows(s, t, 0.1, seed=0)
    assert out["row_status"].tolist() == [0, 1, 1]
    assert np.isnan(out["lam"][1]) and out["token"][2] == -1
