"""Captured HIP graphs: saki_couple (with routing, gradient and loss sum),
saki_route_loss and saki_spec_verify replayed several times, with eager work and synchronisations
between the replays, equal the eager calls bit for bit.  The calls clear their
work counters with a kernel, not a memset node, and sum the loss with a kernel
in a fixed order, so every replay starts from the same state."""
import numpy as np
import pytest
import torch

from paper_2609_36601_amd import workloads

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _same(a, b):
    a, b = a.cpu().numpy(), b.cpu().numpy()
    return np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_couple_replays_in_a_graph(saki_lib):
    n = 512
    s, t = workloads.rows("mid", 0, n, device=DEV)
    V = s.shape[1]
    out = saki_lib.alloc_couple_out(n, DEV)
    route = dict(valid_mask=None, grad_scale=1.0 / n,
                 row_loss=torch.empty(n, dtype=torch.float32, device=DEV),
                 loss_sum=torch.empty(1, dtype=torch.float64, device=DEV),
                 grad=torch.empty(n, V, dtype=torch.float32, device=DEV))
    ws = torch.empty(max(saki_lib.workspace_bytes(saki_lib.SAKI_OP_COUPLE, n, V), 8), dtype=torch.uint8,
                     device=DEV)
    saki_lib.saki_couple(s, t, 0.2, 17, 0, out, route, ws)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}
    ref.update({k: route[k].clone() for k in ("row_loss", "loss_sum", "grad")})

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        saki_lib.saki_couple(s, t, 0.2, 17, 0, out, route, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        saki_lib.saki_couple(s, t, 0.2, 17, 0, out, route, ws)
    for rep in range(3):
        for v in out.values():
            v.fill_(0)
        for k in ("row_loss", "loss_sum", "grad"):
            route[k].fill_(float("nan"))
        ws.fill_(0x5A)                     # stale counter and loss slots
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            got = route[k] if k in ("row_loss", "loss_sum", "grad") else out[k]
            assert _same(got, v), f"replay {rep}: {k} differs from the eager call"


def test_verify_replays_in_a_graph(saki_lib):
    k, n = 8, 8 * 64
    s, t = workloads.rows("verify", 0, n, device=DEV)
    draft = workloads.drafts(s)
    V = s.shape[1]
    acc = torch.empty(n // k, dtype=torch.int32, device=DEV)
    corr = torch.empty(n // k, dtype=torch.int32, device=DEV)
    ws = torch.empty(max(saki_lib.workspace_bytes(saki_lib.SAKI_OP_VERIFY, n, V), 8), dtype=torch.uint8,
                     device=DEV)
    saki_lib.saki_spec_verify(s, t, k, draft, 0.2, 5, 0, -1, acc, corr, None, ws)
    torch.cuda.synchronize()
    ref_a, ref_c = acc.clone(), corr.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        saki_lib.saki_spec_verify(s, t, k, draft, 0.2, 5, 0, -1, acc, corr, None, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        saki_lib.saki_spec_verify(s, t, k, draft, 0.2, 5, 0, -1, acc, corr, None, ws)
    for rep in range(3):
        acc.fill_(-7)
        corr.fill_(-7)
        ws.fill_(0x5A)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(acc, ref_a) and torch.equal(corr, ref_c), f"replay {rep} differs"


def test_route_loss_replays_in_a_graph(saki_lib):
    n = 512
    s, t = workloads.rows("mid", 0, n, device=DEV)
    out = saki_lib.couple(s, t, 0.2, 17, 0)
    torch.cuda.synchronize()
    adv = (out["logt_token"] - out["logp_token"]).contiguous()
    args = (s, out["token"], out["corrected"], out["teacher_argmax"], adv)
    ref = saki_lib.route_loss(*args, grad_scale=1.0 / n)
    torch.cuda.synchronize()
    V = s.shape[1]
    row_loss = torch.empty(n, dtype=torch.float32, device=DEV)
    loss_sum = torch.empty(1, dtype=torch.float64, device=DEV)
    grad = torch.empty(n, V, dtype=torch.float32, device=DEV)
    ws = torch.empty(max(saki_lib.workspace_bytes(saki_lib.SAKI_OP_ROUTE, n, V), 8), dtype=torch.uint8,
                     device=DEV)
    kw = dict(grad_scale=1.0 / n, row_loss=row_loss, loss_sum=loss_sum, grad=grad, workspace=ws)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        saki_lib.saki_route_loss(*args, **kw)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        saki_lib.saki_route_loss(*args, **kw)
    for rep in range(3):
        for v in (row_loss, loss_sum, grad):
            v.fill_(float("nan"))
        ws.fill_(0x5A)                     # stale counter and loss slots
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, got in (("row_loss", row_loss), ("loss_sum", loss_sum), ("grad", grad)):
            assert _same(got, ref[name]), f"replay {rep}: {name} differs from the eager call"
