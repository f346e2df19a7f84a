"""Trust-region geometric bridge, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Definitions (SAKI, Sec. 3.2, Eq. bridge and Eq. trust_region; App. A):
  p  = softmax(s)       frozen behaviour student at the prefix
  pi = softmax(t)       fixed teacher
  q_lam(v) = p(v)^(1-lam) pi(v)^lam / Z(lam),   Z(lam) = sum_u p^(1-lam) pi^lam
  lam* = the largest lam in [0, 1] with KL(q_lam || p) <= eps.

Writing ell_v = log pi(v) - log p(v), q_lam = softmax(log p + lam*ell) and
A(lam) = log Z(lam) = log sum_v p(v) exp(lam*ell_v), so that
log q_lam(v) - log p(v) = lam*ell_v - A(lam) (App. E writes the same ratio).
KL(lam) is non-decreasing on [0, 1] (its derivative is lam * Var_{q_lam}(ell)),
so the feasible set is an interval [0, lam*] and bisection finds its end.

Readings where the paper is silent:
  * feasibility uses "<=" (Eq. trust_region), so lam* = 1 iff KL(pi||p) <= eps;
  * if t - s is the same for every vocab entry then p = pi, KL(lam) = 0 for
    every lam and lam* = 1 (also at eps = 0);
  * otherwise eps = 0 gives lam* = 0 and q = p (App. G, eps = 0 case).
"""
import numpy as np

BISECTION_STEPS = 64


def log_softmax(x):
    """log softmax over the last axis, max-shifted, float64."""
    x = np.asarray(x, dtype=np.float64)
    m = x.max(axis=-1, keepdims=True)
    y = x - m
    return y - np.log(np.exp(y).sum(axis=-1, keepdims=True))


def logsumexp(x, axis=-1):
    x = np.asarray(x, dtype=np.float64)
    m = x.max(axis=axis, keepdims=True)
    return (m + np.log(np.exp(x - m).sum(axis=axis, keepdims=True))).squeeze(axis)


def bridge_log_q(logp, logpi, lam):
    """log q_lam for rows; lam has one entry per row.  Returns (log q, A(lam))."""
    logp = np.atleast_2d(logp)
    logpi = np.atleast_2d(logpi)
    lam = np.asarray(lam, dtype=np.float64).reshape(-1, 1)
    # log of p^(1-lam) pi^lam, then normalise by Z(lam) (Eq. bridge)
    z = (1.0 - lam) * logp + lam * logpi
    log_z = logsumexp(z, axis=-1)
    return z - log_z[:, None], log_z


def kl_bridge(logp, logpi, lam):
    """KL(q_lam || p) = sum_v q_lam(v) log(q_lam(v) / p(v)) per row (Eq. trust_region).

    log(q/p) is formed as lam*ell - A(lam) (App. E: q/p = (pi/p)^lam / Z), which
    avoids subtracting two O(1) logarithms when lam is small.
    """
    logp = np.atleast_2d(logp)
    logpi = np.atleast_2d(logpi)
    lam = np.asarray(lam, dtype=np.float64).reshape(-1, 1)
    ell = logpi - logp
    log_ratio_unnorm = lam * ell
    A = logsumexp(logp + log_ratio_unnorm, axis=-1)[:, None]
    log_ratio = log_ratio_unnorm - A
    q = np.exp(logp + log_ratio)
    return (q * log_ratio).sum(axis=-1)


def kl_teacher_student(logp, logpi):
    """KL(pi || p), the value of KL(q_lam || p) at the teacher endpoint lam = 1."""
    logp = np.atleast_2d(logp)
    logpi = np.atleast_2d(logpi)
    return (np.exp(logpi) * (logpi - logp)).sum(axis=-1)


def constant_difference(s, t):
    """True for rows where t - s takes one value over the whole vocabulary (p = pi)."""
    d = np.atleast_2d(np.asarray(t, np.float64) - np.asarray(s, np.float64))
    return (d == d[:, :1]).all(axis=-1)


def lambda_star(s, t, eps, steps=BISECTION_STEPS):
    """Largest feasible lam in [0, 1] per row (Eq. trust_region), by bisection.

    Returns lam (float64 per row).  The lower end of the final bracket is
    returned, so KL(q_lam || p) <= eps holds at the returned value.
    """
    s = np.atleast_2d(np.asarray(s, np.float64))
    t = np.atleast_2d(np.asarray(t, np.float64))
    eps = float(eps)
    logp, logpi = log_softmax(s), log_softmax(t)
    n = s.shape[0]
    lam = np.ones(n)
    kl1 = kl_teacher_student(logp, logpi)
    same = constant_difference(s, t)
    # teacher endpoint feasible (App. G) or p = pi: lam* = 1
    interior = (~same) & (kl1 > eps)
    if eps == 0.0:
        # App. G: radius zero admits only q = p
        lam[interior] = 0.0
        return lam
    idx = np.nonzero(interior)[0]
    if idx.size == 0:
        return lam
    lo = np.zeros(idx.size)
    hi = np.ones(idx.size)
    lp, lpi = logp[idx], logpi[idx]
    for _ in range(steps):
        mid = 0.5 * (lo + hi)
        feasible = kl_bridge(lp, lpi, mid) <= eps
        lo = np.where(feasible, mid, lo)
        hi = np.where(feasible, hi, mid)
    lam[idx] = lo
    return lam


def total_variation(logp, logq):
    """TV(p, q) = sum_v [q(v) - p(v)]_+  (Eq. correction_tv and App. D)."""
    p = np.exp(np.atleast_2d(logp))
    q = np.exp(np.atleast_2d(logq))
    return np.maximum(q - p, 0.0).sum(axis=-1)


def bridge_rows(s, t, eps):
    """Everything the bridge fixes per row, as a dict of float64 arrays.

    lam, kl = KL(q_lam*||p), tv, A = log Z(lam*), logp, logpi, logq.
    """
    s = np.atleast_2d(np.asarray(s, np.float64))
    t = np.atleast_2d(np.asarray(t, np.float64))
    logp, logpi = log_softmax(s), log_softmax(t)
    lam = lambda_star(s, t, eps)
    logq, A = bridge_log_q(logp, logpi, lam)
    kl = kl_bridge(logp, logpi, lam)
    tv = total_variation(logp, logq)
    return dict(lam=lam, kl=kl, tv=tv, A=A, logp=logp, logpi=logpi, logq=logq)
