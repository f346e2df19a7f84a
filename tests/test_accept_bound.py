"""The mathematics behind the lambda-free accept bound of speculative
verification (Sec. 3.5, Eq. accept), checked on the CPU against the oracle's
exact lambda* and q.

With x = log pi - log p and A(lam) = log sum_v p_v exp(lam x_v) (the log
normaliser of the bridge, Eq. bridge), g(lam) = lam x_z - A(lam) =
log q_lam(z) - log p(z) is concave with g(0) = 0.  On a bracket [la, lb] of
lambda* it lies above the smaller of its end values, and a draft whose
uniform lies below exp of that is accepted whatever lambda* is.  Above the
middle node lm (KL(lm) < eps) the bracket can end below 1, where convexity
alone forces KL > eps:
    lh = lm (KL(pi||p) - eps) / (lm A'(1) - A(lm) - eps),
and on [lm, lh] g lies above lam x_z minus the chord of A from lm to 1.
"""
import numpy as np
import pytest

from oracle import bridge


def _mid_lambda(eps):
    return min(0.5, max(0.05, 0.5 * np.sqrt(eps)))


def _A_and_slope(logp, x, lam):
    """A(lam) and A'(lam) = E_q[x] for one row, float64."""
    a = logp + lam * x
    A = bridge.logsumexp(a)
    q = np.exp(a - A)
    return A, float((q * x).sum())


def _rows(seed, n, V):
    rng = np.random.default_rng(seed)
    s = rng.normal(0.0, 3.0, (n, V))
    rho = rng.uniform(0.2, 0.99, (n, 1))
    t = rho * s + np.sqrt(1.0 - rho ** 2) * rng.normal(0.0, 3.0, (n, V))
    return s, t


@pytest.mark.parametrize("eps", [0.05, 0.2, 0.5])
def test_bracket_end_bounds_lambda_star_and_the_bound_holds(eps):
    s, t = _rows(11, 48, 512)
    logp, logpi = bridge.log_softmax(s), bridge.log_softmax(t)
    lam_star = bridge.lambda_star(s, t, eps)
    lm = _mid_lambda(eps)
    rng = np.random.default_rng(5)
    tightened = 0
    for r in range(s.shape[0]):
        x = logpi[r] - logp[r]
        Am, Dm = _A_and_slope(logp[r], x, lm)
        A1, D1 = _A_and_slope(logp[r], x, 1.0)
        klm, kl1 = lm * Dm - Am, D1 - A1
        assert abs(A1) < 1e-12  # sum_v pi_v = 1
        if not (klm < eps < kl1):
            continue
        den = lm * D1 - Am - eps
        if den <= 0.0:
            continue  # the lower bound on KL never reaches eps: the bracket stays [lm, 1]
        lh = lm * (kl1 - eps) / den
        assert lh > lm
        if lh >= 1.0:
            continue  # nor below 1: g(1) stays
        # the bracket end: KL(lh) > eps, so lambda* < lh
        assert bridge.kl_bridge(logp[r], logpi[r], [lh])[0] > eps - 1e-12
        assert lam_star[r] <= lh + 1e-12
        # the bound at both brackets lies below g(lambda*) for every draft
        logq, _ = bridge.bridge_log_q(logp[r], logpi[r], [lam_star[r]])
        g_star = logq[0] - logp[r]
        g_lm = lm * x - Am
        chord_lh = Am + (A1 - Am) * (lh - lm) / (1.0 - lm)
        old = np.minimum(g_lm, x - A1)
        new = np.minimum(g_lm, lh * x - chord_lh)
        z = rng.choice(x.size, 64, replace=False)
        assert np.all(new[z] <= g_star[z] + 1e-10)
        assert np.all(new >= old - 1e-12)  # never looser than the bracket [lm, 1]
        tightened += int(np.any(new > old + 1e-3))
    assert tightened > 0
