"""Supervision variants at correction positions, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Teacher-sampled target (App. C, "teacher-sampled supervision"): at a
correction the supervision target is a draw v~ ~ pi_T instead of the teacher
mode v*, and the row's loss is L_TS = -log pi_theta(v~), whose expected
gradient over v~ is that of KL(pi_T || pi_theta).  The draw uses the same
two-level exponential race as the coupling (oracle/coupling.py) on log pi_T,
with its own Philox streams (TS_CHUNK, TS_ELEM); routing with target v~ is
route_rows with teacher_argmax replaced by the targets.

Placement controls (Sec. 4.1 and App. "Additional Placement-Control
Results"): for trajectory i with valid positions V_i, m_i = sum_{t in V_i}
C_{i,t} positions of V_i are selected, and the selected positions receive the
teacher-mode loss while the other valid positions keep the RKL loss
(route_rows with corrected replaced by the selection).
  Random-TM      : m_i positions of V_i uniformly at random without
                   replacement (count-matched random placement).
  TV-Weighted-TM : m_i positions without replacement with weights
                   d_{i,t} = TV(p_{i,t}, q_{i,t}), by exponential-race keys
                   -log U_{i,t} / d_{i,t} (the m_i smallest win); if fewer than
                   m_i valid positions have d > 0, the remaining ones are
                   filled uniformly from the positions with d = 0.
U_{i,t} is the STREAM_SELECT uniform of the position's global row.  Keys are
compared as ln E - ln d (E = -ln U), which orders them as E / d; ties go to the
lower row.  The smallest m keys of independent Exp(d_t) races are a weighted
sample without replacement (successive draws with law d_t / sum of the rest).
"""
import numpy as np

from . import philox
from .bridge import log_softmax
from .coupling import CHUNK, exponential_race

MODE_RANDOM = 0
MODE_TV_WEIGHTED = 1


def teacher_sample(t, seed, row_offset=0, chunk=CHUNK):
    """v~ ~ softmax(t) for every row by the two-level race.  Returns (targets, gaps)."""
    t = np.atleast_2d(np.asarray(t, np.float64))
    n = t.shape[0]
    logpi = log_softmax(t)
    out = np.empty(n, np.int64)
    gaps = np.full((n, 2), np.inf)
    for r in range(n):
        v, _, gc, ge = exponential_race(logpi[r], seed, row_offset + r, philox.STREAM_TS_CHUNK,
                                        philox.STREAM_TS_ELEM, chunk)
        out[r] = v
        gaps[r] = gc, ge
    return out, gaps


def correction_targets(coupled, t, seed, row_offset=0, sample=False, chunk=CHUNK):
    """Target of the gradient's indicator per row: y at accepted rows; at
    corrections v* (teacher mode) or v~ ~ pi_T (teacher-sampled).  Also returns
    the race gaps of the teacher draws (inf at rows without a draw)."""
    C = np.asarray(coupled["corrected"]) != 0
    target = np.where(C, coupled["teacher_argmax"], coupled["token"]).astype(np.int64)
    gaps = np.full((target.shape[0], 2), np.inf)
    if sample:
        ts, g = teacher_sample(t, seed, row_offset, chunk)
        target = np.where(C, ts, target)
        gaps[C] = g[C]
    bad = np.asarray(coupled["row_status"]) != 0
    target = np.where(bad, -1, target)
    return target, gaps


def select_positions(tv, corrected, valid, traj_offsets, seed, row_offset=0,
                     mode=MODE_TV_WEIGHTED):
    """Selection mask (0/1 per row) of a placement control, one trajectory per
    row range [traj_offsets[i], traj_offsets[i + 1]).  Also returns, per
    trajectory, the relative gap between the last selected key and the first
    one left out within the same tier (inf when there is no such pair): how
    close the selection was to a tie."""
    tv = np.asarray(tv, np.float64)
    C = np.asarray(corrected) != 0
    M = np.ones(tv.shape[0], bool) if valid is None else (np.asarray(valid) != 0)
    off = np.asarray(traj_offsets, np.int64)
    sel = np.zeros(tv.shape[0], np.uint8)
    gaps = np.full(off.shape[0] - 1, np.inf)
    for i in range(off.shape[0] - 1):
        rows = np.arange(off[i], off[i + 1])
        rows = rows[M[rows]]
        m = int(C[rows].sum())
        if m == 0:
            continue
        E = np.array([-np.log(philox.uniform(seed, philox.STREAM_SELECT, row_offset + int(r), 0))
                      for r in rows])
        if mode == MODE_RANDOM:
            tiers = [(rows, np.log(E))]
        else:
            d = tv[rows]
            pos = d > 0
            with np.errstate(divide="ignore"):
                tiers = [(rows[pos], np.log(E[pos]) - np.log(d[pos])), (rows[~pos], np.log(E[~pos]))]
        left = m
        for r_t, k_t in tiers:
            if left == 0:
                break
            order = np.lexsort((r_t, k_t))  # by key, then by row
            take = order[:left]
            sel[r_t[take]] = 1
            if left < order.size:
                gaps[i] = min(gaps[i], float(np.expm1(k_t[order[left]] - k_t[order[left - 1]])))
            left -= take.size
    return sel, gaps


__all__ = ["MODE_RANDOM", "MODE_TV_WEIGHTED", "teacher_sample", "correction_targets",
           "select_positions"]
