"""GPU parity of saki_probe_metrics (C_1, C_k, KL(T||S), H(S), teacher Top-k)
against the float64 oracle."""
import numpy as np
import pytest
import torch

from oracle import probe
from paper_2609_36601_amd import workloads
from tests.test_gpu_parity import DEV, f64, say

pytestmark = pytest.mark.gpu


def _check(saki, s, t, k, rows=None):
    say(f"probe n={s.shape[0]} V={s.shape[1]} dtype={s.dtype} k={k}")
    out = saki.probe_metrics(s, t, k)
    torch.cuda.synchronize()
    rows = np.arange(s.shape[0]) if rows is None else np.asarray(rows)
    ii = torch.as_tensor(rows, device=DEV)
    o = probe.probe_metrics(f64(s[ii]), f64(t[ii]), k)
    g = {key: v[ii].cpu().numpy() for key, v in out.items()}
    assert np.all(g["row_status"] == 0)
    assert np.array_equal(g["topk"], o["topk"]), "teacher Top-k sets differ"
    for key in ("c1", "ck", "entropy"):
        err = np.abs(g[key] - o[key]) / (np.abs(o[key]) + 1e-9)
        assert err.max() < 1e-5, (key, err.max())
    kerr = np.abs(g["kl_ts"] - o["kl_ts"]) / (np.abs(o["kl_ts"]) + 1e-6)
    assert kerr.max() < 1e-5, ("kl_ts", kerr.max())
    return g, o


@pytest.mark.parametrize("k", [1, 16, 64])
def test_probe_tiny_all_rows(saki_lib, k):
    s, t = workloads.rows("tiny", 0, 256, device=DEV)
    _check(saki_lib, s, t, k)


def test_probe_mid_and_large_sampled(saki_lib):
    s, t = workloads.rows("mid", 0, 4096, device=DEV)
    rng = np.random.default_rng(0)
    _check(saki_lib, s[:1024], t[:1024], 16, rows=rng.choice(1024, 48, replace=False))
    s, t = workloads.rows("large", 0, 64, device=DEV)
    _check(saki_lib, s, t, 16, rows=np.arange(0, 64, 4))


def test_probe_ties_ragged_vocab_and_bad_rows(saki_lib):
    g = torch.Generator(device="cpu").manual_seed(3)
    for V in (5, 1000, 3001):
        s = (torch.randn(40, V, generator=g) * 2).to(torch.bfloat16)
        t = torch.round(torch.randn(40, V, generator=g) * 2).to(torch.bfloat16)  # heavy ties
        t[3] = 1.0  # all equal: the Top-k are the k lowest indices
        S, T = saki_lib.alloc_rows(40, V, torch.bfloat16, DEV), saki_lib.alloc_rows(40, V, torch.bfloat16, DEV)
        S.copy_(s)
        T.copy_(t)
        k = min(16, V)
        _check(saki_lib, S, T, k)
        assert list(_check(saki_lib, S, T, k, rows=[3])[0]["topk"][0]) == list(range(k))
    T[7, 2] = float("nan")
    out = saki_lib.probe_metrics(S, T, 4)
    assert int(out["row_status"][7]) == 1 and torch.isnan(out["c1"][7])
    assert torch.all(out["topk"][7] == -1)
    assert int(out["row_status"][6]) == 0


def test_probe_vocab_beyond_chunk_table(saki_lib):
    # more than 512 chunks of 1024 entries (the per-chunk maxima are then not
    # kept and every gather is a full sweep), with a ragged last chunk
    V = 512 * 1024 + 1001
    g = torch.Generator(device="cpu").manual_seed(5)
    s = (torch.randn(6, V, generator=g) * 3).to(torch.bfloat16)
    t = (torch.randn(6, V, generator=g) * 3).to(torch.bfloat16)
    t[2] = torch.round(t[2].float())  # heavy ties at the threshold
    t[4] = -2.0                       # all equal
    S, T = saki_lib.alloc_rows(6, V, torch.bfloat16, DEV), saki_lib.alloc_rows(6, V, torch.bfloat16, DEV)
    S.copy_(s)
    T.copy_(t)
    _check(saki_lib, S, T, 16)
    assert list(_check(saki_lib, S, T, 16, rows=[4])[0]["topk"][0]) == list(range(16))


def test_probe_signed_zero_ties_past_the_gather_capacity(saki_lib):
    # ten positive teacher logits, then 3,000 zeros of both signs: the 16th
    # largest value is 0, more than 256 entries reach it (the counting search
    # runs), and -0 and +0 tie, so the six lowest-index zeros complete the set
    V, k = 3010, 16
    g = torch.Generator(device="cpu").manual_seed(11)
    s = (torch.randn(4, V, generator=g) * 2).to(torch.bfloat16)
    sign = torch.where(torch.rand(4, V, generator=g) < 0.5, -1.0, 1.0)
    t = sign * 0.0
    pos = torch.stack([torch.randperm(V, generator=g)[:10] for _ in range(4)])
    t.scatter_(1, pos, torch.rand(4, 10, generator=g) + 1.0)
    t[1, :8] = -0.0  # the lowest indices are -0 in this row
    S, T = saki_lib.alloc_rows(4, V, torch.bfloat16, DEV), saki_lib.alloc_rows(4, V, torch.bfloat16, DEV)
    S.copy_(s)
    T.copy_(t.to(torch.bfloat16))
    assert torch.signbit(T.float()).any() and (T.float() == 0).sum() > 4 * 256
    _check(saki_lib, S, T, k)
