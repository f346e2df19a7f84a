"""Pins for the oracle's supervision variants: the teacher-sampled target
(App. C) and the Random-TM / TV-Weighted-TM placement controls (Sec. 4.1,
App. "Additional Placement-Control Results").

Laws are checked by Monte Carlo over many global rows (each row has its own
Philox streams) with chi-square / binomial bounds at about the 1e-5 level;
counts and supports exactly.
"""
import itertools

import numpy as np
import pytest
import scipy.stats

from oracle import bridge, coupling, philox, routing, supervision


def _chi2_ok(counts, probs, alpha=1e-5):
    counts = np.asarray(counts, float)
    probs = np.asarray(probs, float)
    keep = probs > 0
    assert counts[~keep].sum() == 0, "mass outside the support"
    exp = probs[keep] * counts.sum()
    stat = ((counts[keep] - exp) ** 2 / exp).sum()
    return scipy.stats.chi2.sf(stat, keep.sum() - 1) > alpha


def _binom_ok(k, n, p, alpha=1e-5):
    lo = scipy.stats.binom.ppf(alpha / 2, n, p)
    hi = scipy.stats.binom.isf(alpha / 2, n, p)
    return lo <= k <= hi


def test_teacher_sample_law_is_pi():
    # v~ ~ pi_T: the two-level race on log pi with small chunks, one draw per global row
    t = np.array([1.0, -0.5, 2.0, 0.3, -2.0, 1.2, 0.0])
    pi = np.exp(t - t.max()); pi /= pi.sum()
    n = 20000
    draws, _ = supervision.teacher_sample(np.tile(t, (n, 1)), seed=11, chunk=3)
    counts = np.bincount(draws, minlength=len(t))
    assert _chi2_ok(counts, pi)


def test_teacher_sample_uses_its_own_streams():
    # the teacher draw is not the proposal draw of the same row re-used
    rng = np.random.default_rng(0)
    s = rng.normal(size=(400, 50)); t = s.copy()  # p = pi: same law, different streams
    ts, _ = supervision.teacher_sample(t, seed=5)
    ev = coupling.couple_rows(s, t, 0.1, seed=5)
    assert (ts != ev["proposal"]).mean() > 0.5
    ts2, _ = supervision.teacher_sample(t, seed=5)
    assert np.array_equal(ts, ts2)


def test_teacher_sampled_loss_expected_gradient_is_forward_kl():
    # E_{v~ ~ pi}[grad -log p(v~)] = p - pi = grad of KL(pi || p) w.r.t. s (App. C)
    s = np.array([0.5, -1.0, 1.5, 0.0, 0.7])
    t = np.array([1.0, 0.2, -0.5, 1.4, 0.1])
    p = np.exp(s - s.max()); p /= p.sum()
    pi = np.exp(t - t.max()); pi /= pi.sum()
    n = 40000
    v, _ = supervision.teacher_sample(np.tile(t, (n, 1)), seed=3)
    S = np.tile(s, (n, 1))
    C = np.ones(n, np.int64)
    _, _, g = routing.route_rows(S, v, C, v, np.zeros(n))
    mean_g = g.mean(axis=0)
    se = np.sqrt(pi * (1 - pi) / n)
    assert np.all(np.abs(mean_g - (p - pi)) < 6 * se)
    # and the loss is -log p(v~)
    l, _, _ = routing.route_rows(S[:5], v[:5], C[:5], v[:5], np.zeros(5), want_grad=False)
    assert np.allclose(l, -np.log(p[v[:5]]))


def test_correction_targets_route_by_event():
    rng = np.random.default_rng(1)
    s = rng.normal(size=(300, 40)) * 2
    t = 0.5 * s + rng.normal(size=(300, 40))
    t[7] = np.nan
    ev = coupling.couple_rows(s, t, 0.3, seed=9)
    mode, _ = supervision.correction_targets(ev, t, 9, sample=False)
    samp, gaps = supervision.correction_targets(ev, t, 9, sample=True)
    C = ev["corrected"] == 1
    ok = ev["row_status"] == 0
    assert C.sum() > 20
    assert np.array_equal(mode[ok & ~C], ev["token"][ok & ~C])
    assert np.array_equal(samp[ok & ~C], ev["token"][ok & ~C])
    assert np.array_equal(mode[ok & C], ev["teacher_argmax"][ok & C])
    assert mode[7] == -1 and samp[7] == -1
    assert np.all(np.isinf(gaps[~C]))
    # at corrections the sampled target is a draw from pi, not always the mode
    assert (samp[ok & C] != mode[ok & C]).any()


def _traj(lengths):
    return np.concatenate([[0], np.cumsum(lengths)])


def test_selection_counts_and_support():
    rng = np.random.default_rng(2)
    lengths = [7, 1, 12, 5, 9]
    off = _traj(lengths)
    n = off[-1]
    for mode in (supervision.MODE_RANDOM, supervision.MODE_TV_WEIGHTED):
        for seed in range(20):
            C = (rng.random(n) < 0.4).astype(np.uint8)
            M = (rng.random(n) < 0.8).astype(np.uint8)
            tv = np.where(rng.random(n) < 0.3, 0.0, rng.random(n))
            sel, _ = supervision.select_positions(tv, C, M, off, seed, mode=mode)
            assert np.all(sel[M == 0] == 0)
            for i in range(len(lengths)):
                r = slice(off[i], off[i + 1])
                assert sel[r].sum() == (C[r] * M[r]).sum()


def test_random_tm_marginal_is_count_matched_uniform():
    # m of L valid positions uniformly: each position is selected w.p. m / L
    L, m, n_traj = 6, 2, 6000
    off = _traj([L] * n_traj)
    C = np.tile([1, 1, 0, 0, 0, 0], n_traj).astype(np.uint8)
    tv = np.ones(L * n_traj)
    sel, _ = supervision.select_positions(tv, C, None, off, 4, mode=supervision.MODE_RANDOM)
    counts = sel.reshape(n_traj, L).sum(axis=0)
    for k in counts:
        assert _binom_ok(k, n_traj, m / L)
    # the selected pair is uniform over the 15 pairs
    pairs = [tuple(np.flatnonzero(r)) for r in sel.reshape(n_traj, L)]
    keys = list(itertools.combinations(range(L), 2))
    cnt = np.array([sum(1 for q in pairs if q == k) for k in keys])
    assert _chi2_ok(cnt, np.full(len(keys), 1 / len(keys)))


def test_tv_weighted_single_selection_law():
    # m = 1: the selected position has law d_t / sum d (exponential race)
    d = np.array([0.05, 0.3, 0.1, 0.25, 0.0, 0.3])
    L, n_traj = len(d), 12000
    off = _traj([L] * n_traj)
    C = np.tile([0, 0, 1, 0, 0, 0], n_traj).astype(np.uint8)
    sel, _ = supervision.select_positions(np.tile(d, n_traj), C, None, off, 8,
                                          mode=supervision.MODE_TV_WEIGHTED)
    counts = sel.reshape(n_traj, L).sum(axis=0)
    assert _chi2_ok(counts, d / d.sum())


def test_tv_weighted_pair_law_is_successive_sampling():
    # m = 2 without replacement: P{a, b} = d_a/D d_b/(D - d_a) + d_b/D d_a/(D - d_b)
    d = np.array([0.4, 0.1, 0.3, 0.2])
    L, n_traj = len(d), 12000
    off = _traj([L] * n_traj)
    C = np.tile([1, 1, 0, 0], n_traj).astype(np.uint8)
    sel, _ = supervision.select_positions(np.tile(d, n_traj), C, None, off, 21,
                                          mode=supervision.MODE_TV_WEIGHTED)
    keys = list(itertools.combinations(range(L), 2))
    D = d.sum()
    probs = np.array([d[a] / D * d[b] / (D - d[a]) + d[b] / D * d[a] / (D - d[b]) for a, b in keys])
    rows = sel.reshape(n_traj, L)
    cnt = np.array([np.sum(rows[:, a] & rows[:, b]) for a, b in keys])
    assert probs.sum() == pytest.approx(1.0)
    assert _chi2_ok(cnt, probs)


def test_tv_weighted_uniform_fill_when_too_few_positive():
    # 2 positions with d > 0, m = 3: both are taken, the third is uniform over the d = 0 ones
    d = np.array([0.2, 0.0, 0.0, 0.5, 0.0, 0.0])
    L, n_traj = len(d), 8000
    off = _traj([L] * n_traj)
    C = np.tile([1, 1, 1, 0, 0, 0], n_traj).astype(np.uint8)
    sel, _ = supervision.select_positions(np.tile(d, n_traj), C, None, off, 17,
                                          mode=supervision.MODE_TV_WEIGHTED)
    rows = sel.reshape(n_traj, L)
    assert np.all(rows[:, 0] == 1) and np.all(rows[:, 3] == 1)
    fill = rows[:, [1, 2, 4, 5]].sum(axis=0)
    assert fill.sum() == n_traj
    assert _chi2_ok(fill, np.full(4, 0.25))


def test_selection_deterministic_and_row_keyed():
    rng = np.random.default_rng(5)
    off = _traj([10, 10])
    C = (rng.random(20) < 0.5).astype(np.uint8)
    tv = rng.random(20)
    a, _ = supervision.select_positions(tv, C, None, off, 99, row_offset=1000)
    b, _ = supervision.select_positions(tv, C, None, off, 99, row_offset=1000)
    assert np.array_equal(a, b)
    # the second trajectory alone, given its own global rows, selects the same positions
    c, _ = supervision.select_positions(tv[10:], C[10:], None, _traj([10]), 99, row_offset=1010)
    assert np.array_equal(a[10:], c)
