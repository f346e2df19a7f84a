"""Pins for the oracle's routed loss and gradient (Sec. 3.4, App. B, App. G, App. H)."""
import numpy as np
import pytest
import scipy.stats
import torch

from oracle import bridge, coupling, routing


def _events(seed, n, V):
    rng = np.random.default_rng(seed)
    s = rng.normal(0, 2, (n, V))
    t = 0.3 * s + rng.normal(0, 2, (n, V))
    return s, t, coupling.couple_rows(s, t, 0.3, seed=seed)


def test_gradient_matches_torch_autograd():
    s, t, ev = _events(1, 24, 37)
    assert 0 < ev["corrected"].sum() < 24
    mask = (np.arange(24) % 5 != 0).astype(np.float64)
    scale = 1.0 / mask.sum()
    _, loss_sum, grad = routing.couple_and_route(ev, s, mask, scale)
    S = torch.tensor(s, dtype=torch.float64, requires_grad=True)
    logp = torch.log_softmax(S, dim=-1)
    logpi = torch.log_softmax(torch.tensor(t, dtype=torch.float64), dim=-1)
    y = torch.tensor(ev["token"])
    vs = torch.tensor(ev["teacher_argmax"])
    C = torch.tensor(ev["corrected"], dtype=torch.float64)
    M = torch.tensor(mask)
    idx = torch.arange(24)
    A = (logpi[idx, y] - logp[idx, y]).detach()  # sg[...] of Eq. k1_advantage_token
    L = (M * ((1 - C) * (-A) * logp[idx, y] + C * (-logp[idx, vs]))).sum() * scale
    L.backward()
    assert float(L) == pytest.approx(loss_sum, rel=1e-13)
    assert np.allclose(S.grad.numpy(), grad, rtol=0, atol=1e-15)


def test_gradient_central_differences():
    s, t, ev = _events(2, 6, 9)
    adv = ev["logt_token"] - ev["logp_token"]  # held fixed (detached)
    _, _, grad = routing.route_rows(s, ev["token"], ev["corrected"], ev["teacher_argmax"], adv)
    h = 1e-6
    for r in range(6):
        for j in range(9):
            sp, sm = s.copy(), s.copy()
            sp[r, j] += h
            sm[r, j] -= h
            lp = routing.route_rows(sp, ev["token"], ev["corrected"], ev["teacher_argmax"], adv,
                                    want_grad=False)[0][r]
            lm = routing.route_rows(sm, ev["token"], ev["corrected"], ev["teacher_argmax"], adv,
                                    want_grad=False)[0][r]
            assert (lp - lm) / (2 * h) == pytest.approx(grad[r, j], abs=1e-7)


def test_gradient_rows_sum_to_zero_and_masking():
    s, t, ev = _events(3, 30, 50)
    mask = np.ones(30)
    mask[::3] = 0
    rl, ls, grad = routing.couple_and_route(ev, s, mask, 0.25)
    assert np.allclose(grad.sum(axis=1), 0, atol=1e-14)
    assert np.all(grad[::3] == 0) and np.all(rl[::3] == 0)
    assert ls == pytest.approx(0.25 * rl.sum(), rel=1e-14)


def test_correction_rows_carry_only_teacher_mode():
    # App. H: at a correction the RKL term is exactly zero and the target is v*
    s, t, ev = _events(4, 40, 30)
    rl, _, _ = routing.couple_and_route(ev, s)
    c = ev["corrected"] == 1
    assert c.any()
    logp = bridge.log_softmax(s)
    assert np.allclose(rl[c], -logp[np.nonzero(c)[0], ev["teacher_argmax"][c]], rtol=1e-14)


def test_eps_zero_reduces_to_plain_rkl():
    # App. G: with eps = 0 every row is accepted and L is the student-rollout RKL mean
    rng = np.random.default_rng(5)
    s = rng.normal(0, 2, (50, 40))
    t = rng.normal(0, 2, (50, 40))
    ev = coupling.couple_rows(s, t, 0.0, seed=9)
    rl, ls, _ = routing.couple_and_route(ev, s, None, 1.0 / 50)
    logp, logpi = bridge.log_softmax(s), bridge.log_softmax(t)
    idx = np.arange(50)
    y = ev["token"]
    k1 = logp[idx, y] - logpi[idx, y]
    assert ls == pytest.approx(np.mean(k1 * logp[idx, y]), rel=1e-13)


def test_expected_overlap_identity():
    # Eq. expected_overlap_k1: E[(1 - C) L_RKL(Z)] = sum_v min(p, q) L_RKL(v)
    rng = np.random.default_rng(6)
    s = rng.normal(0, 1.0, 6)
    t = rng.normal(0, 1.0, 6)
    b = bridge.bridge_rows(s[None], t[None], 0.1)
    p, q = np.exp(b["logp"][0]), np.exp(b["logq"][0])
    L_rkl = -(b["logpi"][0] - b["logp"][0]) * b["logp"][0]
    want = np.sum(np.minimum(p, q) * L_rkl)
    n = 30000
    ev = coupling.couple_rows(np.tile(s, (n, 1)), np.tile(t, (n, 1)), 0.1, seed=31)
    rl, _, _ = routing.couple_and_route(ev, np.tile(s, (n, 1)), want_grad=False)
    vals = (1 - ev["corrected"]) * rl
    se = vals.std() / np.sqrt(n)
    assert abs(vals.mean() - want) < 5 * se
