"""Fixed-prefix probe metrics of a student distribution S against a teacher
T at one position, in float64 (Sec. 4 probe analysis; App. "fixed-prefix
probe").

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

  C_1(h)  = S(v*_T(h)),               v*_T the teacher's Top-1 token
  C_k(h)  = sum_{v in S^T_k(h)} S(v), S^T_k the teacher's Top-k set (k = 16 in
                                      the paper); C_k - C_1 is the student's
                                      mass on the teacher-supported alternatives
  KL(T || S) = sum_v T(v) (log T(v) - log S(v))  (the conflict measure whose
                                      quartiles partition the probe positions)
  H(S)    = -sum_v S(v) log S(v)      (student entropy)
The Top-k set takes the k largest teacher logits, ties to the lower index
(the same tie rule as the teacher mode).
"""
import numpy as np

from .bridge import log_softmax


def teacher_topk(t, k):
    """Indices of the k largest entries of t (ties to the lower index), best first."""
    t = np.asarray(t, np.float64)
    order = np.lexsort((np.arange(t.shape[0]), -t))
    return order[:k]


def probe_metrics(s, t, k=16):
    """Per-row C_1, C_k, KL(T || S), H(S) and the Top-k index sets."""
    s = np.atleast_2d(np.asarray(s, np.float64))
    t = np.atleast_2d(np.asarray(t, np.float64))
    n, V = s.shape
    k = min(k, V)
    logS = log_softmax(s)
    logT = log_softmax(t)
    S = np.exp(logS)
    T = np.exp(logT)
    top = np.stack([teacher_topk(t[r], k) for r in range(n)])
    idx = np.arange(n)
    c1 = S[idx, top[:, 0]]
    ck = np.take_along_axis(S, top, axis=1).sum(axis=1)
    kl = np.sum(T * (logT - logS), axis=1)
    h = -np.sum(S * logS, axis=1)
    return dict(c1=c1, ck=ck, kl_ts=kl, entropy=h, topk=top)


__all__ = ["teacher_topk", "probe_metrics"]
