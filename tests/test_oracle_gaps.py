"""Pins for the decision gaps the oracle reports next to its race winners
and placement selections.

The parity rules excuse a GPU/oracle mismatch of a race winner only when the
best and second-best keys of that race were within 1e-6 of each other
(relative gap of E / w), and a selection mismatch only when the last key taken
and the first key left out were that close.  These tests fix the gap
functions on hand-computed key sets and on races built to tie exactly, so a
wrong key set, a wrong order or a log-scale gap in place of the relative one
fails here rather than silently widening the excuse.
"""
import math

import numpy as np

from oracle import coupling, philox, supervision


def test_gap_hand_computed_key_sets():
    g = coupling._gap
    # an exact tie at the best key
    assert g(np.array([1.25, 1.25])) == 0.0
    assert g(np.array([3.0, 0.5, 0.5])) == 0.0
    # fewer than two finite keys: no competitor, no tie possible
    assert g(np.array([0.7])) == math.inf
    assert g(np.array([np.inf, 2.0, np.inf])) == math.inf
    assert g(np.array([], dtype=float)) == math.inf
    # the two smallest finite keys, relative gap of E / w = e^(k2 - k1) - 1;
    # infinite keys (zero weights) are not competitors
    keys = np.array([2.0, np.inf, 0.5, 1.2, np.inf])
    assert g(keys) == np.expm1(0.7)
    assert abs(g(keys) - 1.0137527074704766) < 1e-15
    # not the log-scale difference, not the largest key
    assert g(keys) != 0.7 and g(keys) != np.expm1(1.5)
    # invariant under the order of the keys
    rng = np.random.default_rng(0)
    for _ in range(20):
        assert g(rng.permutation(keys)) == g(keys)
    # a shift of every key leaves the gap
    assert abs(g(keys + 10.0) - g(keys)) < 1e-13


def _exps(stream, g, n, seed):
    return -np.log(philox.uniforms(seed, stream, g, range(n)))


def test_race_gap_exact_element_tie():
    """Weights chosen so that entries 1 and 3 of a one-chunk row have equal
    keys E_v / w_v: the element gap is 0 (to rounding), the winner is the
    lower index of the tie, and the chunk gap is inf (one chunk)."""
    seed, g, V = 77, 12, 4
    E = _exps(philox.STREAM_PROP_ELEM, g, V, seed)
    # w_v = E_v / k_v with k_1 = k_3 the smallest key
    k = np.array([5.0, 1.0, 3.0, 1.0])
    log_w = np.log(E) - np.log(k)
    win, c0, gc, ge = coupling.exponential_race(log_w, seed, g, philox.STREAM_PROP_CHUNK,
                                                philox.STREAM_PROP_ELEM, chunk=4)
    assert c0 == 0 and gc == math.inf
    assert ge < 1e-12
    assert win == 1
    # break the tie by 1e-3 of the key: the gap is 1e-3 and entry 3 wins
    k2 = k.copy()
    k2[3] = 1.0 / (1.0 + 1e-3)
    win, _, _, ge = coupling.exponential_race(np.log(E) - np.log(k2), seed, g, philox.STREAM_PROP_CHUNK,
                                              philox.STREAM_PROP_ELEM, chunk=4)
    assert win == 3 and abs(ge - 1e-3) < 1e-12


def test_race_gap_exact_chunk_tie_and_zero_weights():
    """Two chunks of two entries whose chunk keys E_c / W_c tie exactly: the
    chunk gap is 0 and chunk 0 wins.  Inside the winning chunk one entry has
    weight 0 (log w = -inf): it is not a competitor, so the element gap is inf."""
    seed, g = 5, 3
    Ec = _exps(philox.STREAM_RES_CHUNK, g, 2, seed)
    # chunk weights W_c = E_c (keys ln E_c - ln W_c = 0 for both chunks)
    log_w = np.array([np.log(Ec[0]), -np.inf, np.log(Ec[1]) - np.log(2.0), np.log(Ec[1]) - np.log(2.0)])
    win, c0, gc, ge = coupling.exponential_race(log_w, seed, g, philox.STREAM_RES_CHUNK,
                                                philox.STREAM_RES_ELEM, chunk=2)
    assert c0 == 0 and gc < 1e-12
    assert win == 0 and ge == math.inf


def test_couple_rows_reports_the_race_gaps():
    """couple_rows stores (proposal chunk, proposal element, residual chunk,
    residual element) gaps; the residual ones stay inf at accepted rows."""
    rng = np.random.default_rng(4)
    s = rng.normal(0, 2, (40, 9))
    t = rng.normal(0, 2, (40, 9))
    o = coupling.couple_rows(s, t, 0.3, 11, 0, chunk=3)
    gaps = o["gaps"]
    assert gaps.shape == (40, 4)
    acc = o["corrected"] == 0
    assert np.all(np.isinf(gaps[acc, 2:])) and np.all(np.isfinite(gaps[:, :2]))
    assert np.all(gaps >= 0)
    # recompute the proposal gaps of row 0 from its keys
    logp = o["logp"][0]
    z, _, gc, ge = coupling.exponential_race(logp, 11, 0, philox.STREAM_PROP_CHUNK, philox.STREAM_PROP_ELEM, 3)
    assert z == o["proposal"][0] and gc == gaps[0, 0] and ge == gaps[0, 1]


def test_selection_gap_exact_tie_and_tiers():
    """TV-Weighted-TM: weights d chosen so that rows 1 and 2 of one trajectory
    have equal keys E / d and m = 1: the gap is 0 and the lower row is taken.
    A trajectory whose m exceeds its rows with d > 0 fills from the d = 0 tier:
    the gap then comes from that tier's keys."""
    seed, off = 9, 100
    E = np.array([-np.log(philox.uniform(seed, philox.STREAM_SELECT, off + r, 0)) for r in range(8)])
    # trajectory 0 = rows 0..3, one correction; keys E_r / d_r = (4, 1, 1, 2)
    d0 = E[:4] / np.array([4.0, 1.0, 1.0, 2.0])
    # trajectory 1 = rows 4..7, three corrections, one row with d > 0
    d1 = np.array([0.3, 0.0, 0.0, 0.0])
    tv = np.concatenate([d0, d1])
    corrected = np.array([1, 0, 0, 0, 1, 1, 1, 0])
    sel, gaps = supervision.select_positions(tv, corrected, None, [0, 4, 8], seed, off,
                                             supervision.MODE_TV_WEIGHTED)
    assert sel[:4].tolist() == [0, 1, 0, 0]
    assert gaps[0] < 1e-12
    # rows 5..7 have d = 0: two of them are drawn by their keys ln E
    assert sel[4] == 1 and sel[4:].sum() == 3
    k = np.log(E[5:8])
    order = np.argsort(k, kind="stable")
    assert sel[5 + order[2]] == 0 and sel[5 + order[0]] == 1 and sel[5 + order[1]] == 1
    assert abs(gaps[1] - np.expm1(k[order[2]] - k[order[1]])) < 1e-15


def test_selection_gap_random_mode():
    """Random-TM with m = 2 of 5 rows: the gap is between the second and third
    smallest ln E of the trajectory, relative (e^(k3 - k2) - 1)."""
    seed, off = 21, 7
    k = np.array([np.log(-np.log(philox.uniform(seed, philox.STREAM_SELECT, off + r, 0))) for r in range(5)])
    sel, gaps = supervision.select_positions(np.zeros(5), [1, 1, 0, 0, 0], None, [0, 5], seed, off,
                                             supervision.MODE_RANDOM)
    order = np.argsort(k)
    assert set(np.nonzero(sel)[0]) == set(order[:2].tolist())
    assert abs(gaps[0] - np.expm1(k[order[2]] - k[order[1]])) < 1e-15
