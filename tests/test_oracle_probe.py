"""Pins for the oracle's fixed-prefix probe metrics (C_1, C_k, KL(T||S), H(S))."""
import numpy as np
import scipy.special
import scipy.stats

from oracle import probe


def test_topk_matches_sorting_with_lowest_index_ties():
    t = np.array([1.0, 3.0, 3.0, -1.0, 2.0, 3.0, 2.0])
    assert list(probe.teacher_topk(t, 4)) == [1, 2, 5, 4]
    assert list(probe.teacher_topk(t, 7)) == [1, 2, 5, 4, 6, 0, 3]
    rng = np.random.default_rng(0)
    for _ in range(20):
        x = np.round(rng.normal(size=50) * 2) / 2  # many ties
        k = int(rng.integers(1, 50))
        top = probe.teacher_topk(x, k)
        # brute force: v is in the set iff fewer than k entries beat it (value, then index)
        beats = [(np.sum(x > x[v]) + np.sum((x == x[v]) & (np.arange(50) < v))) for v in range(50)]
        assert set(top) == {v for v in range(50) if beats[v] < k}


def test_metrics_against_library_routines():
    rng = np.random.default_rng(1)
    s = rng.normal(size=(6, 40)) * 2
    t = rng.normal(size=(6, 40)) * 2
    m = probe.probe_metrics(s, t, k=16)
    S = scipy.special.softmax(s, axis=1)
    T = scipy.special.softmax(t, axis=1)
    assert np.allclose(m["kl_ts"], scipy.special.rel_entr(T, S).sum(axis=1), rtol=1e-12)
    assert np.allclose(m["entropy"], scipy.stats.entropy(S, axis=1), rtol=1e-12)
    for r in range(6):
        order = np.argsort(-t[r], kind="stable")
        assert np.isclose(m["c1"][r], S[r, order[0]])
        assert np.isclose(m["ck"][r], S[r, order[:16]].sum())


def test_metric_bounds_and_special_cases():
    rng = np.random.default_rng(2)
    s = rng.normal(size=(5, 30)) * 3
    t = rng.normal(size=(5, 30)) * 3
    m = probe.probe_metrics(s, t, k=16)
    assert np.all(m["c1"] <= m["ck"] + 1e-15) and np.all(m["ck"] <= 1 + 1e-12)
    assert np.all(m["kl_ts"] >= 0) and np.all(m["entropy"] >= 0)
    # k = V: the Top-k set is everything
    assert np.allclose(probe.probe_metrics(s, t, k=30)["ck"], 1.0)
    # S = T (logits equal up to a constant): KL 0, C_1 = T(v*)
    m2 = probe.probe_metrics(t + 4.0, t, k=3)
    assert np.allclose(m2["kl_ts"], 0.0, atol=1e-12)
    T = scipy.special.softmax(t, axis=1)
    assert np.allclose(m2["c1"], T.max(axis=1))
    # uniform student: entropy log V, C_k = k / V
    m3 = probe.probe_metrics(np.zeros((5, 30)), t, k=4)
    assert np.allclose(m3["entropy"], np.log(30))
    assert np.allclose(m3["ck"], 4 / 30)
