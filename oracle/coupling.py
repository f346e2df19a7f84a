"""Maximal coupling of p and q_lam*, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

SAKI, Sec. 3.3: draw z ~ p; accept with probability min(1, q(z)/p(z))
(Eq. accept); on rejection draw the correction from the normalised positive
residual r(v) = [q(v) - p(v)]_+ / sum_u [q(u) - p(u)]_+ (Eq. residual).
App. I gives the acceptance in log space, exp(min(0, log q(a) - log p(a))).

The paper does not fix how the draws are made.  This project fixes them so
that a fast implementation and this oracle make the same draws:

  * uniforms come from Philox-4x32-10 keyed by (seed, stream, global row),
    see oracle/philox.py;
  * the accept test is "accept iff u < alpha" with u in (0, 1), so
    alpha = 1 always accepts;
  * z ~ p and c ~ r are drawn by a two-level exponential race over vocab
    chunks of CHUNK entries: each chunk c gets E_c = -ln u_c and the chunk
    with the smallest E_c / W_c wins (W_c = the chunk's total weight); then
    each entry v of that chunk with w_v > 0 gets E_v = -ln u_v and the
    smallest E_v / w_v wins.  Ties go to the lowest index.  The minimum of
    independent Exp(w_v) variables is Exp(sum w_v) and its argmin has law
    w_v / sum w_v, so the winner of either level has exactly the law
    w / sum(w), and the two levels compose to the law w / sum(w) over the
    vocabulary.  (The paper itself uses exponential-race keys -log U / d for
    weighted selection, App. C.)  Keys are compared as ln E - ln w, which
    orders them the same way.
"""
import numpy as np

from . import philox
from .bridge import bridge_rows, log_softmax, logsumexp

CHUNK = 1024


def _uniform_block(seed, stream, g, lo, hi):
    return philox.uniforms(seed, stream, g, range(lo, hi))


def exponential_race(log_w, seed, g, chunk_stream, elem_stream, chunk=CHUNK):
    """Two-level exponential race on log weights log_w (one row); -inf = weight 0.

    Returns (winner index, chunk index, relative key gap at the chunk level,
    relative key gap at the element level).  The gaps (second-best key /
    best key - 1) say how close each decision was to a tie.
    """
    log_w = np.asarray(log_w, dtype=np.float64)
    V = log_w.shape[0]
    n_chunks = (V + chunk - 1) // chunk
    log_wc = np.array([logsumexp(log_w[c * chunk:(c + 1) * chunk])
                       if np.isfinite(log_w[c * chunk:(c + 1) * chunk]).any() else -np.inf
                       for c in range(n_chunks)])
    E_c = -np.log(_uniform_block(seed, chunk_stream, g, 0, n_chunks))
    key_c = np.where(np.isfinite(log_wc), np.log(E_c) - log_wc, np.inf)
    c0 = int(np.argmin(key_c))
    lo, hi = c0 * chunk, min(V, (c0 + 1) * chunk)
    E_v = -np.log(_uniform_block(seed, elem_stream, g, lo, hi))
    lw = log_w[lo:hi]
    key_v = np.where(np.isfinite(lw), np.log(E_v) - lw, np.inf)
    j = int(np.argmin(key_v))
    return lo + j, c0, _gap(key_c), _gap(key_v)


def _gap(keys):
    """Distance between the best and second-best race keys, relative to E/w.

    Keys are ln(E/w); exp(k2 - k1) - 1 is the relative gap of E/w.
    """
    k = np.sort(keys[np.isfinite(keys)])
    if k.size < 2:
        return np.inf
    return float(np.expm1(k[1] - k[0]))


def couple_rows(s, t, eps, seed, row_offset=0, chunk=CHUNK):
    """Maximal coupling for every row of (s, t).  Returns a dict of per-row arrays.

    Keys: lam, kl, tv, A, proposal, accept_prob, u, margin, corrected, token,
    teacher_argmax, logp_token, logt_token, logq_token, gaps (prop chunk,
    prop elem, res chunk, res elem), plus the full logp / logpi / logq.
    """
    s = np.atleast_2d(np.asarray(s, np.float64))
    t = np.atleast_2d(np.asarray(t, np.float64))
    n, V = s.shape
    # the bridge assumes positive softmax probabilities (App. E); a row with
    # a non-finite logit gets status 1 and NaN / -1 outputs
    good = np.isfinite(s).all(axis=1) & np.isfinite(t).all(axis=1)
    s = np.where(good[:, None], s, 0.0)
    t = np.where(good[:, None], t, 0.0)
    b = bridge_rows(s, t, eps)
    out = dict(lam=b["lam"], kl=b["kl"], tv=b["tv"], A=b["A"],
               logp=b["logp"], logpi=b["logpi"], logq=b["logq"])
    proposal = np.empty(n, np.int64)
    token = np.empty(n, np.int64)
    corrected = np.zeros(n, np.int64)
    alpha = np.empty(n)
    u_acc = np.empty(n)
    gaps = np.full((n, 4), np.inf)
    for r in range(n):
        g = row_offset + r
        logp, logq = b["logp"][r], b["logq"][r]
        # z ~ p (Sec. 3.3)
        z, _, gc, ge = exponential_race(logp, seed, g, philox.STREAM_PROP_CHUNK,
                                        philox.STREAM_PROP_ELEM, chunk)
        gaps[r, 0], gaps[r, 1] = gc, ge
        proposal[r] = z
        # Eq. accept, in the log form of App. I
        alpha[r] = np.exp(min(0.0, logq[z] - logp[z]))
        u = philox.uniform(seed, philox.STREAM_ACCEPT, g, 0)
        u_acc[r] = u
        if u < alpha[r]:
            token[r] = z
        else:
            corrected[r] = 1
            # Eq. residual: c ~ [q - p]_+ / sum [q - p]_+
            w = np.maximum(np.exp(logq) - np.exp(logp), 0.0)
            with np.errstate(divide="ignore"):
                log_w = np.log(w)
            c, _, gc, ge = exponential_race(log_w, seed, g, philox.STREAM_RES_CHUNK,
                                            philox.STREAM_RES_ELEM, chunk)
            gaps[r, 2], gaps[r, 3] = gc, ge
            token[r] = c
    idx = np.arange(n)
    # teacher mode v* = argmax_v t_v, lowest index on ties (Sec. 3.4)
    vstar = np.argmax(t, axis=-1)
    out.update(
        proposal=proposal, token=token, corrected=corrected, accept_prob=alpha,
        u=u_acc, margin=np.abs(u_acc - alpha), teacher_argmax=vstar,
        logp_token=b["logp"][idx, token], logt_token=b["logpi"][idx, token],
        logq_token=b["logq"][idx, token], gaps=gaps,
        row_status=np.where(good, 0, 1))
    bad = ~good
    for key in ("lam", "kl", "tv", "A", "accept_prob", "margin", "logp_token",
                "logt_token", "logq_token"):
        out[key] = np.where(bad, np.nan, out[key])
    for key in ("proposal", "token", "teacher_argmax"):
        out[key] = np.where(bad, -1, out[key])
    out["corrected"] = np.where(bad, 0, out["corrected"])
    return out


def residual_draw(logp, logq, seed, g, chunk=CHUNK):
    """c ~ [q - p]_+ normalised, for one row (Eq. residual).  Returns (c, gaps)."""
    w = np.maximum(np.exp(logq) - np.exp(logp), 0.0)
    with np.errstate(divide="ignore"):
        log_w = np.log(w)
    c, _, gc, ge = exponential_race(log_w, seed, g, philox.STREAM_RES_CHUNK,
                                    philox.STREAM_RES_ELEM, chunk)
    return c, (gc, ge)


__all__ = ["CHUNK", "exponential_race", "couple_rows", "residual_draw", "log_softmax"]
