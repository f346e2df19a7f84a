"""GPU parity: the HIP library (through its C ABI) against the float64 oracle.

Small configurations are compared on every row; the full-size configurations
run in the bench's launch configuration and are compared on sampled rows, and
on properties that hold at any size for every row.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import bridge, coupling, routing, verify
from paper_2609_36601_amd import workloads
from tests import parity

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def np_out(out):
    return {k: v.cpu().numpy() for k, v in out.items() if isinstance(v, torch.Tensor)}


def f64(x):
    return x.float().cpu().numpy().astype(np.float64)


def run_and_compare(saki, s, t, eps, seed, row_offset=0, rows=None, grad=True, valid=None,
                    grad_dtype=torch.float32, target_sample=False):
    say(f"couple n={s.shape[0]} V={s.shape[1]} dtype={s.dtype} eps={eps} offset={row_offset} "
        f"target_sample={target_sample}")
    vm = None if valid is None else torch.as_tensor(valid, dtype=torch.uint8, device=DEV)
    out = saki.couple(s, t, eps, seed, row_offset, route=True,
                      grad_dtype=grad_dtype if grad else None, valid_mask=vm, grad_scale=1.0,
                      correction_target=saki.SAKI_TARGET_SAMPLE if target_sample else saki.SAKI_TARGET_MODE)
    torch.cuda.synchronize()
    o = np_out(out)
    rows = np.arange(s.shape[0]) if rows is None else np.asarray(rows)
    g = f64(out["grad"][torch.as_tensor(rows, device=DEV)]) if grad else None
    R = parity.compare_couple(o, f64(s[torch.as_tensor(rows, device=DEV)]),
                              f64(t[torch.as_tensor(rows, device=DEV)]), eps, seed, row_offset,
                              rows, grad=g, valid=valid, target_sample=target_sample)
    say(R.summary())
    R.check()
    return out, o, R


def test_tiny_all_rows(saki_lib):
    s, t = workloads.rows("tiny", 0, 256, device=DEV)
    run_and_compare(saki_lib, s, t, 0.1, workloads.coupling_seed("tiny"))


@pytest.mark.parametrize("eps", [0.05, 0.2])
def test_mid_sampled_rows(saki_lib, eps):
    s, t = workloads.rows("mid", 0, 4096, device=DEV)
    rng = np.random.default_rng(int(eps * 100))
    rows = np.unique(np.concatenate([[0, 1, 4095], rng.choice(4096, 45, replace=False)]))
    out, o, R = run_and_compare(saki_lib, s, t, eps, workloads.coupling_seed("mid"), rows=rows)
    # properties on every row; rows that break one are compared with the oracle
    bad = np.nonzero((o["row_status"] != 0) | (o["kl"] > eps * (1 + 1e-5) + 1e-9) |
                     (o["tv"] > np.sqrt(o["kl"] / 2) * (1 + 1e-5) + 1e-7))[0]
    if bad.size:
        say(f"rows breaking a property: {bad[:10].tolist()} (of {bad.size})")
        ii = torch.as_tensor(bad[:4], device=DEV)
        R2 = parity.compare_couple(o, f64(s[ii]), f64(t[ii]), eps, workloads.coupling_seed("mid"), 0,
                                   bad[:4])
        say(R2.summary())
        R2.check()
    assert bad.size == 0


def _row_properties(o, eps, grad=None):
    assert np.all(o["row_status"] == 0)
    lam = o["lambda"]
    assert np.all((lam >= 0) & (lam <= 1))
    interior = lam < 1
    assert np.all(np.abs(o["kl"][interior] - eps) <= 2e-5 * eps)
    assert np.all(o["kl"] <= eps * (1 + 2e-5))
    # Cor. 1 (Pinsker) and Prop. 1 (correction rate = TV, on average)
    assert np.all(o["kl"] >= 0)
    assert np.all(o["tv"] <= np.sqrt(o["kl"] / 2) * (1 + 1e-5) + 1e-7)
    n = len(lam)
    rate, mean_tv = o["corrected"].mean(), o["tv"].mean()
    assert abs(rate - mean_tv) < 6 * np.sqrt(mean_tv * (1 - mean_tv) / n) + 1e-3
    acc = o["corrected"] == 0
    assert np.array_equal(o["token"][acc], o["proposal"][acc])


def test_large_full_size_sampled(saki_lib):
    cfg = workloads.CONFIGS["large"]
    n, V = cfg["rows"], cfg["V"]
    say(f"generate large {n}x{V}")
    s = torch.empty(n, V, dtype=torch.bfloat16, device=DEV)
    t = torch.empty_like(s)
    workloads.fill("large", s, t)
    eps = 0.2
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, 1023, 1024, n - 1], rng.choice(n, 6, replace=False)]))
    out, o, R = run_and_compare(saki_lib, s, t, eps, workloads.coupling_seed("large"), rows=rows)
    _row_properties(o, eps)
    g = out["grad"]
    # every gradient row sums to zero (sum_j (p_j - 1[j = hot]) = 0)
    sums = g[:4096].double().sum(dim=1).abs().max().item()
    assert sums < 1e-3
    del s, t, out, g
    torch.cuda.empty_cache()


@pytest.mark.parametrize("eps", [0.05, 0.5])
def test_large_other_radii(saki_lib, eps):
    s, t = workloads.rows("large", 0, 2048, device=DEV)
    rows = np.array([0, 700, 1500, 2047])
    out, o, R = run_and_compare(saki_lib, s, t, eps, workloads.coupling_seed("large"), rows=rows)
    _row_properties(o, eps)


@pytest.mark.parametrize("variant", ["", "shared"])
def test_stream_chunk(saki_lib, variant):
    chunk = 5
    lo = 4096 * chunk
    s, t = workloads.rows("stream", lo, lo + 4096, device=DEV, variant=variant)
    rows = np.array([0, 1, 2000, 4095])
    out, o, R = run_and_compare(saki_lib, s, t, 0.02, workloads.coupling_seed("stream"),
                                row_offset=lo, rows=rows)
    _row_properties(o, 0.02)


def test_verify_blocks(saki_lib):
    k = 8
    n = 4096 * 2
    s, t = workloads.rows("verify", 0, n, device=DEV)
    draft = workloads.drafts(s)
    eps = 0.2
    seed = workloads.coupling_seed("verify")
    say(f"verify n={n} k={k}")
    out = saki_lib.spec_verify(s, t, k, draft, eps, seed)
    torch.cuda.synchronize()
    gpu = dict(accepted_len=out["accepted_len"].cpu().numpy(),
               correction=out["correction"].cpu().numpy(),
               per_pos=np_out(out["per_pos"]))
    blocks = np.array([0, 1, 2, 500, 1023])
    idx = np.concatenate([np.arange(b * k, (b + 1) * k) for b in blocks])
    ii = torch.as_tensor(idx, device=DEV)
    R = parity.compare_verify(gpu, f64(s[ii]), f64(t[ii]), k, draft[ii].cpu().numpy(), eps, seed, 0,
                              blocks)
    say(R.summary())
    R.check()
    al = gpu["accepted_len"]
    assert al.min() >= 0 and al.max() <= k
    assert np.all((gpu["correction"] >= 0) == (al < k))
    say(f"mean accepted length {al.mean():.3f}")


def test_verify_without_per_position_outputs(saki_lib):
    """Without per-position outputs, drafts whose u lies below min(1, pi(z) / p(z))
    (a lower bound of the accept probability for every lambda in [0, 1]) are
    accepted without the lambda search; results equal the full path's and the
    oracle's."""
    k = 8
    n = 4096 * 2
    s, t = workloads.rows("verify", 0, n, device=DEV)
    draft = workloads.drafts(s)
    eps, seed = 0.2, workloads.coupling_seed("verify")
    say(f"verify without per-position outputs n={n}")
    full = saki_lib.spec_verify(s, t, k, draft, eps, seed)
    lean = saki_lib.spec_verify(s, t, k, draft, eps, seed, per_pos=False)
    torch.cuda.synchronize()
    gpu = dict(accepted_len=lean["accepted_len"].cpu().numpy(), correction=lean["correction"].cpu().numpy())
    same = (gpu["accepted_len"] == full["accepted_len"].cpu().numpy()) & \
           (gpu["correction"] == full["correction"].cpu().numpy())
    diff = np.nonzero(~same)[0]
    say(f"blocks differing from the full path: {diff.size}")
    assert diff.size <= 2
    blocks = np.unique(np.concatenate([[0, 1, 2, 500, 1023], diff]))
    idx = np.concatenate([np.arange(b * k, (b + 1) * k) for b in blocks])
    ii = torch.as_tensor(idx, device=DEV)
    R = parity.compare_verify(gpu, f64(s[ii]), f64(t[ii]), k, draft[ii].cpu().numpy(), eps, seed, 0,
                              blocks)
    say(R.summary())
    R.check()
    # EOS through the shortcut: p = pi accepts every draft
    V = 300
    s2 = torch.randn(2 * 4, V, generator=torch.Generator(device=DEV).manual_seed(3), device=DEV)
    d2 = torch.tensor([3, 7, 5, 1, 2, 2, 2, 2], dtype=torch.int32, device=DEV)
    out = saki_lib.spec_verify(s2, s2.clone(), 4, d2, 0.1, 5, eos_id=7, per_pos=False)
    torch.cuda.synchronize()
    assert out["accepted_len"].cpu().tolist() == [2, 4] and out["correction"].cpu().tolist() == [-1, -1]


def test_verify_full_size_sampled(saki_lib):
    """The verify workload at full size (8,192 blocks of k = 8, V = 151,936
    bf16) in the configuration the benchmark times (accepted lengths and
    corrections only): sampled blocks against the oracle, and the first-
    rejection structure on every block."""
    cfg = workloads.CONFIGS["verify"]
    k, n, V = cfg["k"], cfg["rows"], cfg["V"]
    nb = n // k
    say(f"generate verify {n}x{V}")
    s = torch.empty(n, V, dtype=torch.bfloat16, device=DEV)
    t = torch.empty_like(s)
    workloads.fill("verify", s, t)
    draft = workloads.drafts(s)
    eps, seed = 0.2, workloads.coupling_seed("verify")
    out = saki_lib.spec_verify(s, t, k, draft, eps, seed, per_pos=False)
    torch.cuda.synchronize()
    gpu = dict(accepted_len=out["accepted_len"].cpu().numpy(), correction=out["correction"].cpu().numpy())
    al, co = gpu["accepted_len"], gpu["correction"]
    assert al.shape == (nb,) and al.min() >= 0 and al.max() <= k
    assert np.all((co >= 0) == (al < k)) and co.max() < V
    rng = np.random.default_rng(11)
    blocks = np.unique(np.concatenate([[0, 1, nb // 2, nb - 1], rng.choice(nb, 4, replace=False)]))
    idx = np.concatenate([np.arange(b * k, (b + 1) * k) for b in blocks])
    ii = torch.as_tensor(idx, device=DEV)
    say(f"oracle on blocks {blocks.tolist()}")
    R = parity.compare_verify(gpu, f64(s[ii]), f64(t[ii]), k, draft[ii].cpu().numpy(), eps, seed, 0,
                              blocks)
    say(R.summary())
    R.check()
    del s, t, draft, out
    torch.cuda.empty_cache()


def test_verify_edge_cases(saki_lib):
    k, V = 4, 300
    rng = torch.Generator(device=DEV).manual_seed(1)
    s = torch.randn(3 * k, V, generator=rng, device=DEV)
    t = s.clone()
    t[k:] = torch.randn(2 * k, V, generator=rng, device=DEV)
    draft = torch.tensor([3, 7, 5, 1] * 3, dtype=torch.int32, device=DEV)
    draft[2 * k + 1] = 1000  # out of range
    out = saki_lib.spec_verify(s, t, k, draft, 0.1, 5, eos_id=7)
    torch.cuda.synchronize()
    al, co = out["accepted_len"].cpu().tolist(), out["correction"].cpu().tolist()
    o = verify.verify_blocks(f64(s), f64(t), k, draft.cpu().numpy(), 0.1, 5, 0, 7)
    assert al == o["accepted_len"].tolist() and co == o["correction"].tolist()
    assert al[0] == 2 and co[0] == -1  # p = pi: accepted through the EOS at position 1
    st = out["per_pos"]["row_status"].cpu().tolist()
    assert st[0:4] == [0, 0, 3, 3]
    if al[2] == 1:
        assert st[9] == 2


def padded(x):
    """Copy of a [n, V] tensor in storage whose row pitch is a multiple of 16 bytes."""
    n, V = x.shape
    per = 16 // x.element_size()
    buf = torch.zeros(n, (V + per - 1) // per * per, dtype=x.dtype, device=x.device)
    buf[:, :V] = x
    return buf[:, :V]


def test_edge_vocab_sizes_and_special_rows(saki_lib):
    g = torch.Generator(device=DEV).manual_seed(7)
    for V in (1, 7, 8, 1000, 1025, 3000):
        n = 24
        s = padded((2 * torch.randn(n, V, generator=g, device=DEV)).to(torch.bfloat16))
        t = padded((2 * torch.randn(n, V, generator=g, device=DEV)).to(torch.bfloat16))
        t[3] = s[3]            # p = pi
        t[4] = s[4] + 2.0      # p = pi (exact shift in bf16 for these magnitudes? compare oracle anyway)
        if V > 1:
            s[5, V // 2] = float("inf")
            t[6, 0] = float("nan")
        for eps in (0.0, 0.3):
            valid = np.ones(n, np.uint8)
            valid[::5] = 0
            run_and_compare(saki_lib, s, t, eps, 99, row_offset=10, valid=valid)


@pytest.mark.parametrize("V", [16 * 1024, 17 * 1024 + 5, 256 * 1024, 256 * 1024 + 1])
def test_row_cache_boundaries(saki_lib, V):
    """bf16 rows of up to 256 chunks keep each wave's last four full chunks in
    LDS: every chunk cached (16 chunks), one chunk per wave past that plus a
    ragged tail, the largest cached row (256 chunks), and one entry more (the
    variant without the cache).  Coupling, loss and gradient against the
    oracle on every row; the verify kernel on the same rows, whose blocks
    stop at their first rejection."""
    g = torch.Generator(device=DEV).manual_seed(V)
    n = 8
    s = (3.0 * torch.randn(n, V, generator=g, device=DEV) / 0.7).to(torch.bfloat16)
    t = (0.7 * s.float() + 0.7 * 3.0 * torch.randn(n, V, generator=g, device=DEV)).to(torch.bfloat16)
    s, t = padded(s), padded(t)
    run_and_compare(saki_lib, s, t, 0.2, 4242, row_offset=3)
    k = 4
    draft = workloads.drafts(s)
    out = saki_lib.spec_verify(s, t, k, draft, 0.2, 4242, 3)
    torch.cuda.synchronize()
    gpu = dict(accepted_len=out["accepted_len"].cpu().numpy(),
               correction=out["correction"].cpu().numpy(),
               per_pos=np_out(out["per_pos"]))
    R = parity.compare_verify(gpu, f64(s), f64(t), k, draft.cpu().numpy(), 0.2, 4242, 3,
                              np.arange(n // k))
    say(R.summary())
    R.check()


def test_bf16_gradient_and_masks(saki_lib):
    s, t = workloads.rows("mid", 0, 64, device=DEV)
    valid = (np.arange(64) % 3 != 0).astype(np.uint8)
    out = saki_lib.couple(s, t, 0.2, 3, 0, route=True, grad_dtype=torch.bfloat16,
                          valid_mask=torch.as_tensor(valid, device=DEV), grad_scale=1.0)
    ref = saki_lib.couple(s, t, 0.2, 3, 0, route=True, grad_dtype=torch.float32,
                          valid_mask=torch.as_tensor(valid, device=DEV), grad_scale=1.0)
    torch.cuda.synchronize()
    gb, gf = out["grad"].float(), ref["grad"]
    assert torch.all((gb - gf).abs() <= 2 ** -8 * gf.abs() + 1e-30)
    assert torch.all(gf[torch.as_tensor(valid == 0, device=DEV)] == 0)


def test_loss_sum_and_scale(saki_lib):
    s, t = workloads.rows("tiny", 0, 256, device=DEV)
    valid = (np.arange(256) % 4 != 1).astype(np.uint8)
    scale = 1.0 / valid.sum()
    out = saki_lib.couple(s, t, 0.1, 11, 0, route=True, grad_dtype=torch.float32,
                          valid_mask=torch.as_tensor(valid, device=DEV), grad_scale=scale)
    torch.cuda.synchronize()
    o = np_out(out)
    ev = coupling.couple_rows(f64(s), f64(t), 0.1, 11, 0)
    rl, ls, _ = routing.couple_and_route(ev, f64(s), valid, np.float32(scale), want_grad=False)
    same = (ev["corrected"] == o["corrected"]) & (ev["token"] == o["token"])
    assert same.mean() > 0.99
    if same.all():
        assert abs(o["loss_sum"][0] - ls) <= 1e-5 * np.abs(rl * scale).sum()


def test_route_loss_standalone(saki_lib):
    s, t = workloads.rows("mid", 0, 128, device=DEV)
    ev = saki_lib.couple(s, t, 0.2, 21, 0)
    adv = (ev["logt_token"] - ev["logp_token"]).contiguous()
    valid = torch.as_tensor((np.arange(128) % 7 != 2).astype(np.uint8), device=DEV)
    out = saki_lib.route_loss(s, ev["token"], ev["corrected"], ev["teacher_argmax"], adv,
                              valid_mask=valid, grad_scale=1.0)
    torch.cuda.synchronize()
    rl, ls, grad = routing.route_rows(f64(s), ev["token"].cpu().numpy(), ev["corrected"].cpu().numpy(),
                                      ev["teacher_argmax"].cpu().numpy(), adv.double().cpu().numpy(),
                                      valid.cpu().numpy(), 1.0)
    assert np.all(parity.close(out["row_loss"].cpu().numpy(), rl, atol=1e-6))
    assert abs(out["loss_sum"].item() - ls) <= 1e-5 * np.abs(rl).sum()
    assert np.max(np.abs(out["grad"].cpu().numpy() - grad)) <= parity.GRAD_ATOL


@pytest.mark.parametrize("V", [36 * 1024, 37 * 1024 + 5, 151936])
def test_route_loss_row_cache(saki_lib, V):
    """bf16 rows keep each wave's last nine full chunks of s in LDS between the
    routed loss's two sweeps: every chunk cached (nine per wave), one chunk per
    wave past that plus a ragged tail, and the large vocabulary (36 of its 148
    full chunks cached).  Loss and gradient against the oracle on every row,
    with a masked row and a bf16 gradient."""
    g = torch.Generator(device=DEV).manual_seed(V)
    n = 12
    s = padded((3.0 * torch.randn(n, V, generator=g, device=DEV) / 0.7).to(torch.bfloat16))
    token = torch.randint(0, V, (n,), generator=g, device=DEV, dtype=torch.int32)
    vstar = torch.randint(0, V, (n,), generator=g, device=DEV, dtype=torch.int32)
    corrected = (torch.arange(n, device=DEV) % 3 == 0).to(torch.uint8)
    adv = torch.randn(n, generator=g, device=DEV).float()
    valid = torch.as_tensor((np.arange(n) != 4).astype(np.uint8), device=DEV)
    say(f"route_loss V={V}")
    rl, ls, grad = routing.route_rows(f64(s), token.cpu().numpy(), corrected.cpu().numpy(),
                                      vstar.cpu().numpy(), adv.double().cpu().numpy(), valid.cpu().numpy(), 1.0)
    for gd in (torch.float32, torch.bfloat16):
        out = saki_lib.route_loss(s, token, corrected, vstar, adv, valid_mask=valid, grad_scale=1.0,
                                  grad_dtype=gd)
        torch.cuda.synchronize()
        assert np.all(parity.close(out["row_loss"].cpu().numpy(), rl, atol=1e-6))
        assert abs(out["loss_sum"].item() - ls) <= 1e-5 * np.abs(rl).sum()
        tol = parity.GRAD_ATOL if gd == torch.float32 else parity.GRAD_ATOL + 2.0 ** -8 * np.abs(grad)
        assert np.all(np.abs(out["grad"].float().cpu().numpy() - grad) <= tol)


def test_route_loss_f32_ragged_and_bad_rows(saki_lib):
    """f32 rows of a ragged vocabulary (no row cache), with a supervised index
    outside [0, V) at a valid row and a non-finite logit (both: NaN loss and a
    NaN gradient row), and a masked row with an invalid index (loss 0, gradient
    row 0); the other rows against the oracle."""
    g = torch.Generator(device=DEV).manual_seed(5)
    n, V = 10, 3000
    s = padded(2.0 * torch.randn(n, V, generator=g, device=DEV))
    token = torch.randint(0, V, (n,), generator=g, device=DEV, dtype=torch.int32)
    vstar = torch.randint(0, V, (n,), generator=g, device=DEV, dtype=torch.int32)
    corrected = (torch.arange(n, device=DEV) % 2 == 1).to(torch.uint8)
    adv = torch.randn(n, generator=g, device=DEV).float()
    valid = torch.ones(n, dtype=torch.uint8, device=DEV)
    good = np.ones(n, bool)
    token[2], corrected[2] = V, 0                  # index outside the row
    vstar[3], corrected[3], valid[3] = -1, 1, 0    # masked, invalid index
    s[5, 17] = float("inf")                        # non-finite logit
    good[[2, 3, 5]] = False
    out = saki_lib.route_loss(s, token, corrected, vstar, adv, valid_mask=valid, grad_scale=1.0)
    torch.cuda.synchronize()
    rl_g, gr_g = out["row_loss"].cpu().numpy(), out["grad"].cpu().numpy()
    for r in (2, 5):
        assert np.isnan(rl_g[r]) and np.isnan(gr_g[r]).all()
    assert rl_g[3] == 0 and np.all(gr_g[3] == 0)
    ii = np.nonzero(good)[0]
    it = torch.as_tensor(ii, device=DEV)
    rl, _, grad = routing.route_rows(f64(s[it]), token[it].cpu().numpy(), corrected[it].cpu().numpy(),
                                     vstar[it].cpu().numpy(), adv[it].double().cpu().numpy(), None, 1.0)
    assert np.all(parity.close(rl_g[ii], rl, atol=1e-6))
    assert np.max(np.abs(gr_g[ii] - grad)) <= parity.GRAD_ATOL


def test_determinism_and_row_split_invariance(saki_lib):
    s, t = workloads.rows("mid", 0, 512, device=DEV)
    a = saki_lib.couple(s, t, 0.2, 5, 1000, route=True, grad_dtype=torch.float32)
    b = saki_lib.couple(s, t, 0.2, 5, 1000, route=True, grad_dtype=torch.float32)
    c1 = saki_lib.couple(s[:200].contiguous(), t[:200].contiguous(), 0.2, 5, 1000, route=True,
                         grad_dtype=torch.float32)
    c2 = saki_lib.couple(s[200:].contiguous(), t[200:].contiguous(), 0.2, 5, 1200, route=True,
                         grad_dtype=torch.float32)
    torch.cuda.synchronize()
    for k in ("lambda", "kl", "tv", "proposal", "token", "corrected", "accept_prob", "grad", "row_loss"):
        assert torch.equal(a[k], b[k]), k
        assert torch.equal(a[k][:200], c1[k]) and torch.equal(a[k][200:], c2[k]), k


def test_zero_rows_is_a_no_op(saki_lib):
    s = torch.empty(0, 64, dtype=torch.bfloat16, device=DEV)
    out = saki_lib.couple(s, s, 0.1, 1, 0, route=True, grad_dtype=torch.float32)
    torch.cuda.synchronize()
    assert out["lambda"].numel() == 0
