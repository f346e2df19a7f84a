"""Pins for the oracle's bridge: log-softmax, KL(q_lam||p), lam*, TV.

Each check is independent of the oracle's own arithmetic: a library routine,
a 50-digit mpmath evaluation of the definition, a constrained optimiser, a
root finder, closed forms and the paper's identities.
"""
import mpmath
import numpy as np
import pytest
import scipy.optimize
import scipy.special
from hypothesis import given, settings, strategies as st

from oracle import bridge

mpmath.mp.dps = 50


def _rows(seed, n, V, scale=2.0, corr=0.6):
    rng = np.random.default_rng(seed)
    s = rng.normal(0, scale, (n, V))
    t = corr * s + np.sqrt(1 - corr ** 2) * rng.normal(0, scale, (n, V))
    return s, t


def _mp_kl(s, t, lam):
    """KL(q_lam || p) from the definition, in 50-digit arithmetic."""
    s = [mpmath.mpf(float(x)) for x in s]
    t = [mpmath.mpf(float(x)) for x in t]
    lam = mpmath.mpf(float(lam))
    zs = mpmath.fsum(mpmath.exp(x) for x in s)
    zt = mpmath.fsum(mpmath.exp(x) for x in t)
    p = [mpmath.exp(x) / zs for x in s]
    pi = [mpmath.exp(x) / zt for x in t]
    w = [pv ** (1 - lam) * tv ** lam for pv, tv in zip(p, pi)]
    Z = mpmath.fsum(w)
    q = [x / Z for x in w]
    return mpmath.fsum(qv * mpmath.log(qv / pv) for qv, pv in zip(q, p)), q, p


def test_log_softmax_matches_scipy():
    s, _ = _rows(0, 7, 300, scale=5.0)
    assert np.allclose(bridge.log_softmax(s), scipy.special.log_softmax(s, axis=-1),
                       rtol=0, atol=1e-13)


@pytest.mark.parametrize("seed", range(6))
def test_kl_matches_mpmath_definition(seed):
    s, t = _rows(seed, 1, 6)
    for lam in [0.0, 1e-3, 0.17, 0.5, 0.93, 1.0]:
        want, _, _ = _mp_kl(s[0], t[0], lam)
        got = bridge.kl_bridge(bridge.log_softmax(s), bridge.log_softmax(t), [lam])[0]
        # float64: A(lam) = log Z is formed from O(1) logs, ~1e-16 absolute
        assert abs(got - float(want)) <= 1e-12 * abs(float(want)) + 5e-16


def test_kl_at_one_is_teacher_student_kl_library():
    s, t = _rows(3, 4, 50)
    p = scipy.special.softmax(s, axis=-1)
    pi = scipy.special.softmax(t, axis=-1)
    want = scipy.special.rel_entr(pi, p).sum(axis=-1)
    got = bridge.kl_bridge(bridge.log_softmax(s), bridge.log_softmax(t), np.ones(4))
    assert np.allclose(got, want, rtol=1e-12)


def test_small_lambda_closed_form():
    # KL(q_lam||p) = lam^2 Var_p(ell)/2 + O(lam^3) with ell = log pi - log p
    s, t = _rows(4, 3, 40)
    p = scipy.special.softmax(s, axis=-1)
    ell = scipy.special.log_softmax(t, axis=-1) - scipy.special.log_softmax(s, axis=-1)
    var = (p * ell ** 2).sum(-1) - (p * ell).sum(-1) ** 2
    lam = 1e-4
    got = bridge.kl_bridge(bridge.log_softmax(s), bridge.log_softmax(t), np.full(3, lam))
    assert np.allclose(got, lam ** 2 * var / 2, rtol=2e-3)


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("eps", [0.01, 0.1, 0.4])
def test_lambda_star_root_and_brentq(seed, eps):
    s, t = _rows(seed + 10, 1, 6)
    kl1 = float(_mp_kl(s[0], t[0], 1.0)[0])
    lam = bridge.lambda_star(s, t, eps)[0]
    if kl1 <= eps:
        assert lam == 1.0
        return
    root = scipy.optimize.brentq(lambda x: float(_mp_kl(s[0], t[0], x)[0]) - eps, 0.0, 1.0,
                                 xtol=1e-15, rtol=1e-15)
    assert abs(lam - root) <= 1e-12 * root
    assert abs(float(_mp_kl(s[0], t[0], lam)[0]) - eps) <= 1e-12 * eps


@pytest.mark.parametrize("seed", range(4))
def test_trb_optimality_against_slsqp(seed):
    # App. A: q_lam* solves min KL(q||pi) s.t. KL(q||p) <= eps, sum q = 1
    s, t = _rows(seed + 40, 1, 5, scale=1.5, corr=0.2)
    p = scipy.special.softmax(s[0])
    pi = scipy.special.softmax(t[0])
    eps = 0.05
    lam = bridge.lambda_star(s, t, eps)[0]
    assert 0 < lam < 1
    q_star = np.exp(bridge.bridge_log_q(bridge.log_softmax(s), bridge.log_softmax(t), [lam])[0][0])

    def kl(a, b):
        return float(np.sum(a * (np.log(a) - np.log(b))))

    res = scipy.optimize.minimize(
        lambda q: kl(q, pi), x0=p.copy(), method="SLSQP",
        bounds=[(1e-12, 1.0)] * 5,
        constraints=[{"type": "eq", "fun": lambda q: q.sum() - 1.0},
                     {"type": "ineq", "fun": lambda q: eps - kl(q, p)}],
        options={"ftol": 1e-14, "maxiter": 500})
    assert res.success
    assert np.allclose(res.x, q_star, atol=2e-5)
    assert kl(q_star, pi) <= res.fun + 1e-9


def test_endpoints_and_special_rows():
    s, t = _rows(7, 3, 30)
    kl1 = bridge.kl_teacher_student(bridge.log_softmax(s), bridge.log_softmax(t))
    # eps = 0 admits only q = p (App. G)
    assert np.all(bridge.lambda_star(s, t, 0.0) == 0.0)
    # teacher endpoint when KL(pi||p) <= eps, including equality
    assert np.all(bridge.lambda_star(s, t, float(kl1.max()) + 1e-9) == 1.0)
    lam_eq = bridge.lambda_star(s[:1], t[:1], float(kl1[0]))
    assert lam_eq[0] == 1.0
    # p = pi (t = s + constant): KL = 0 for every lam, lam* = 1 even at eps = 0
    sq = np.round(s * 256) / 256  # so that s + 3 is exact
    assert bridge.lambda_star(sq, sq + 3.0, 0.0).tolist() == [1.0] * 3
    b = bridge.bridge_rows(sq, sq + 3.0, 0.0)
    assert np.all(b["tv"] < 1e-15)


@settings(max_examples=30, deadline=None)
@given(st.integers(0, 10_000), st.integers(2, 40))
def test_kl_monotone_in_lambda(seed, V):
    s, t = _rows(seed, 1, V, scale=3.0, corr=0.0)
    lams = np.linspace(0, 1, 41)
    lp, lt = bridge.log_softmax(s), bridge.log_softmax(t)
    kls = np.array([bridge.kl_bridge(lp, lt, [x])[0] for x in lams])
    assert np.all(np.diff(kls) >= -1e-14)
    assert kls[0] == pytest.approx(0.0, abs=1e-15)


@pytest.mark.parametrize("eps", [0.02, 0.2, 0.5])
def test_tv_identities_and_pinsker(eps):
    s, t = _rows(11, 16, 200, scale=3.0, corr=0.5)
    b = bridge.bridge_rows(s, t, eps)
    p, q = np.exp(b["logp"]), np.exp(b["logq"])
    assert np.allclose(q.sum(-1), 1.0, atol=1e-13)
    assert np.allclose(b["tv"], np.maximum(p - q, 0).sum(-1), atol=1e-13)
    assert np.allclose(b["tv"], 0.5 * np.abs(p - q).sum(-1), atol=1e-13)
    assert np.allclose(b["tv"], 1.0 - np.minimum(p, q).sum(-1), atol=1e-13)
    # Cor. 1: TV <= sqrt(KL/2) <= sqrt(eps/2)
    assert np.all(b["tv"] <= np.sqrt(b["kl"] / 2) + 1e-12)
    assert np.all(b["kl"] <= eps * (1 + 1e-12))


def test_residual_support_threshold():
    # App. E: q_lam(v) > p(v)  <=>  log(pi(v)/p(v)) > log Z_lam / lam
    s, t = _rows(12, 8, 300, scale=3.0, corr=0.4)
    b = bridge.bridge_rows(s, t, 0.2)
    ell = b["logpi"] - b["logp"]
    thresh = (b["A"] / b["lam"])[:, None]
    above = np.exp(b["logq"]) > np.exp(b["logp"])
    margin = np.abs(ell - thresh) > 1e-9
    assert np.array_equal(above[margin], (ell > thresh)[margin])
