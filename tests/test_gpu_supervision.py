"""GPU parity of the supervision variants against the float64 oracle:
teacher-sampled correction targets in saki_couple (App. C) and the
Random-TM / TV-Weighted-TM placement controls of saki_select_positions."""
import sys

import numpy as np
import pytest
import torch

from oracle import routing, supervision
from paper_2609_36601_amd import workloads
from tests import parity
from tests.test_gpu_parity import DEV, f64, np_out, run_and_compare, say

pytestmark = pytest.mark.gpu


def test_teacher_sampled_targets_tiny_all_rows(saki_lib):
    s, t = workloads.rows("tiny", 0, 256, device=DEV)
    out, o, R = run_and_compare(saki_lib, s, t, 0.1, workloads.coupling_seed("tiny"), target_sample=True)
    C = o["corrected"] == 1
    assert C.sum() > 10
    # at corrections the target is a teacher draw, not always the mode
    assert (o["target"][C] != o["teacher_argmax"][C]).any()
    assert np.array_equal(o["target"][~C], o["token"][~C])


def test_teacher_sampled_targets_mid_sampled_rows(saki_lib):
    s, t = workloads.rows("mid", 0, 4096, device=DEV)
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([[0, 4095], rng.choice(4096, 40, replace=False)]))
    run_and_compare(saki_lib, s, t, 0.2, workloads.coupling_seed("mid"), rows=rows, target_sample=True)


def _compare_selection(sel_gpu, tv, C, M, off, seed, row_offset, mode):
    sel_o, gaps = supervision.select_positions(tv, C, M, off, seed, row_offset, mode)
    bad = []
    for i in range(len(off) - 1):
        r = slice(off[i], off[i + 1])
        if not np.array_equal(sel_gpu[r], sel_o[r]):
            if gaps[i] < 1e-9:
                say(f"trajectory {i}: near tie (gap {gaps[i]:.2e})")
                continue
            bad.append(i)
    assert not bad, f"selection differs on trajectories {bad[:10]}"


@pytest.mark.parametrize("mode", [0, 1])
def test_selection_on_coupled_rows(saki_lib, mode):
    # mid: 8 sequences x 512 positions; trajectories of mixed lengths over the
    # same rows, TV and corrections from the GPU coupling
    s, t = workloads.rows("mid", 0, 4096, device=DEV)
    seed = workloads.coupling_seed("mid")
    out = saki_lib.couple(s, t, 0.2, seed)
    rng = np.random.default_rng(mode)
    cuts = np.sort(rng.choice(np.arange(1, 4096), 12, replace=False))
    off = np.concatenate([[0], cuts, np.arange(512 * 7, 4096 + 1, 512)])
    off = np.unique(off)
    valid = (rng.random(4096) < 0.9).astype(np.uint8)
    say(f"select mode={mode} trajectories={len(off) - 1}")
    sel = saki_lib.select_positions(mode, torch.as_tensor(off, device=DEV), out["tv"], out["corrected"],
                                    seed, valid_mask=torch.as_tensor(valid, device=DEV), row_offset=0)
    torch.cuda.synchronize()
    tv = out["tv"].cpu().numpy().astype(np.float64)
    C = out["corrected"].cpu().numpy()
    _compare_selection(sel.cpu().numpy(), tv, C, valid, off, seed, 0, mode)


@pytest.mark.parametrize("mode", [0, 1])
def test_selection_edge_cases(saki_lib, mode):
    rng = np.random.default_rng(10 + mode)
    lengths = [0, 1, 2, 7, 300, 5000, 3, 0, 64]
    off = np.concatenate([[0], np.cumsum(lengths)])
    n = int(off[-1])
    tv = rng.random(n).astype(np.float32)
    tv[rng.random(n) < 0.5] = 0.0          # many zeros: the uniform fill is exercised
    tv[rng.random(n) < 0.01] = np.nan      # rows without outputs count as TV 0
    C = (rng.random(n) < 0.35).astype(np.uint8)
    C[off[5]:off[6]] = (rng.random(5000) < 0.8)  # m larger than the positive-TV rows
    valid = (rng.random(n) < 0.85).astype(np.uint8)
    seed, row_offset = 12345, 77777
    for vm in (valid, None):
        say(f"select edge mode={mode} valid={'yes' if vm is not None else 'none'}")
        sel = saki_lib.select_positions(mode, torch.as_tensor(off, device=DEV),
                                        torch.as_tensor(tv, device=DEV), torch.as_tensor(C, device=DEV),
                                        seed, None if vm is None else torch.as_tensor(vm, device=DEV),
                                        row_offset)
        torch.cuda.synchronize()
        g = sel.cpu().numpy()
        _compare_selection(g, tv.astype(np.float64), C, vm, off, seed, row_offset, mode)
        sel2 = saki_lib.select_positions(mode, torch.as_tensor(off, device=DEV),
                                         torch.as_tensor(tv, device=DEV), torch.as_tensor(C, device=DEV),
                                         seed, None if vm is None else torch.as_tensor(vm, device=DEV),
                                         row_offset)
        assert torch.equal(sel, sel2)


def test_selection_routes_through_route_loss(saki_lib):
    # selected rows take the teacher-mode loss, the others RKL on their token
    s, t = workloads.rows("tiny", 0, 256, device=DEV)
    seed = workloads.coupling_seed("tiny")
    out = saki_lib.couple(s, t, 0.1, seed)
    off = torch.as_tensor(np.arange(0, 257, 64), device=DEV)
    sel = saki_lib.select_positions(1, off, out["tv"], out["corrected"], seed)
    adv = (out["logt_token"] - out["logp_token"]).contiguous()
    r = saki_lib.route_loss(s, out["token"], sel, out["teacher_argmax"], adv, grad_scale=1.0 / 256)
    torch.cuda.synchronize()
    rl, ls, g = routing.route_rows(f64(s), out["token"].cpu().numpy(), sel.cpu().numpy(),
                                   out["teacher_argmax"].cpu().numpy(),
                                   adv.cpu().numpy().astype(np.float64), None, 1.0 / 256)
    assert np.allclose(r["row_loss"].cpu().numpy(), rl, rtol=1e-5, atol=1e-6)
    assert abs(float(r["loss_sum"].item()) - ls) <= 1e-5 * abs(ls) + 1e-9
    assert np.max(np.abs(r["grad"].cpu().numpy() * 256 - g * 256)) < 2e-3
    assert int(sel.sum()) == int(out["corrected"].sum())
