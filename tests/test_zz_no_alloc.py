"""saki_couple_static (no workspace argument: the row counter and the scaled
row losses live in the library's static device scratch) against saki_couple
with a caller workspace, on the same rows: every output bit for bit, on two
calls in a row of which the second has fewer rows, and at the row limit."""
import numpy as np
import pytest
import torch

from paper_2609_36601_amd import workloads

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _buffers(saki, n, V, grad_dtype, row_offset):
    out = saki.alloc_couple_out(n, DEV)
    # the mask follows the global row, the scale is fixed: calls over
    # different row ranges give the same values at the same global rows
    valid = ((row_offset + np.arange(n)) % 5 != 2).astype(np.uint8)
    route = dict(valid_mask=torch.as_tensor(valid, device=DEV),
                 grad_scale=0.25,
                 row_loss=torch.full((n,), 7.0, dtype=torch.float32, device=DEV),
                 loss_sum=torch.full((1,), 7.0, dtype=torch.float64, device=DEV),
                 grad=torch.full((n, V), 7.0, dtype=grad_dtype, device=DEV))
    return out, route


def _same(a, b):
    for k in a:
        x, y = a[k], b[k]
        if x.dtype.is_floating_point:
            ok = torch.equal(torch.nan_to_num(x, nan=123.0), torch.nan_to_num(y, nan=123.0)) and \
                torch.equal(torch.isnan(x), torch.isnan(y))
        else:
            ok = torch.equal(x, y)
        assert ok, k


def _run_pair(saki, s, t, eps, seed, row_offset, grad_dtype):
    n, V = s.shape
    out_a, route_a = _buffers(saki, n, V, grad_dtype, row_offset)
    out_b, route_b = _buffers(saki, n, V, grad_dtype, row_offset)
    saki.saki_couple_static(s, t, eps, seed, row_offset, out_a, route_a)
    ws = torch.empty(saki.workspace_bytes(saki.SAKI_OP_COUPLE, n, V), dtype=torch.uint8, device=DEV)
    saki.saki_couple(s, t, eps, seed, row_offset, out_b, route_b, ws)
    torch.cuda.synchronize()
    _same(out_a, out_b)
    _same({k: route_a[k] for k in ("row_loss", "loss_sum", "grad")},
          {k: route_b[k] for k in ("row_loss", "loss_sum", "grad")})
    return out_a, route_a


def test_static_scratch_matches_workspace_entry(saki_lib):
    seed = workloads.coupling_seed("mid")
    print("static scratch: mid 2048 rows, then 300 rows", flush=True)
    s, t = workloads.rows("mid", 0, 2048, device=DEV)
    a, ra = _run_pair(saki_lib, s, t, 0.2, seed, 0, torch.float32)
    assert ra["loss_sum"].item() != 7.0 and (a["row_status"] == 0).all()
    # a second, smaller call: the scratch keeps the first call's contents
    s2, t2 = workloads.rows("mid", 100, 400, device=DEV)
    b, rb = _run_pair(saki_lib, s2, t2, 0.05, seed, 100, torch.bfloat16)
    # the smaller call's rows equal the larger call's at the same global rows
    # when the radius is the same
    c, rc = _run_pair(saki_lib, s2, t2, 0.2, seed, 100, torch.float32)
    for k in ("lambda", "tv", "token", "corrected"):
        assert torch.equal(c[k], a[k][100:400]), k
    assert torch.equal(rc["grad"], ra["grad"][100:400])
    assert torch.equal(rc["row_loss"], ra["row_loss"][100:400])


def test_static_scratch_at_the_row_limit(saki_lib):
    """SAKI_STATIC_MAX_ROWS rows of a short vocabulary (the whole scratch in
    use), then one row more is refused."""
    n, V = saki_lib.SAKI_STATIC_MAX_ROWS, 64
    print(f"static scratch: {n} rows of V={V}", flush=True)
    g = torch.Generator(device=DEV).manual_seed(12)
    s = (2.0 * torch.randn(n, V, generator=g, device=DEV)).to(torch.bfloat16)
    t = (2.0 * torch.randn(n, V, generator=g, device=DEV)).to(torch.bfloat16)
    _run_pair(saki_lib, s, t, 0.1, 77, 5, torch.float32)
    s1 = torch.zeros(n + 1, V, dtype=torch.bfloat16, device=DEV)
    out = saki_lib.alloc_couple_out(n + 1, DEV)
    with pytest.raises(saki_lib.SakiError) as e:
        saki_lib.saki_couple_static(s1, s1, 0.1, 1, 0, out, None)
    assert e.value.status == 2
