"""Laws the GPU path must realise, checked statistically on its own outputs.

These do not compare draws with the oracle's: they check the distributions the
paper states, over many rows that share their logits but not their random keys
(global rows g = row_offset + r).
  * Prop. 1 / Eq. residual (Sec. 3.3): the committed token has law q, the
    proposal law p, the correction rate is TV(p, q), and a correction has law
    [q - p]_+ / TV.
  * Prop. spec_exact (App. F): GPU rollouts with k-token speculative waves have
    the law prod_t q_t of sequential exact-q sampling.
"""
import numpy as np
import pytest
import torch
from scipy.stats import binomtest, chisquare

from oracle import bridge, rollout as orollout
from paper_2609_36601_amd import binding
from paper_2609_36601_amd.workloads import SyntheticAR, SyntheticARTorch
from tests.test_gpu_parity import DEV, say

pytestmark = pytest.mark.gpu


def _pvalue(obs, law, n):
    """Chi-square p-value with the cells of expected count < 5 pooled."""
    e = law * n
    keep = e >= 5
    o2, e2 = obs[keep], e[keep]
    if (~keep).any():
        if e[~keep].sum() > 0:
            o2 = np.append(o2, obs[~keep].sum())
            e2 = np.append(e2, e[~keep].sum())
        elif obs[~keep].sum() > 0:
            return 0.0  # outcomes the law gives probability 0
    return chisquare(o2, e2 * (o2.sum() / e2.sum())).pvalue


@pytest.mark.parametrize("eps", [0.05, 0.3])
def test_coupling_realises_q(saki_lib, eps):
    s0 = np.array([1.0, 0.2, -0.5, 2.0, -1.0])
    t0 = np.array([-0.5, 1.5, 0.3, 0.4, 2.2])
    n, V = 200_000, s0.size
    s = binding.alloc_rows(n, V, torch.float32, DEV)
    t = binding.alloc_rows(n, V, torch.float32, DEV)
    s.copy_(torch.tensor(s0, dtype=torch.float32).expand(n, V))
    t.copy_(torch.tensor(t0, dtype=torch.float32).expand(n, V))
    say(f"coupling law eps={eps} rows={n}")
    out = saki_lib.couple(s, t, eps, seed=4242, row_offset=10 ** 9)
    torch.cuda.synchronize()
    tok = out["token"].cpu().numpy()
    prop = out["proposal"].cpu().numpy()
    C = out["corrected"].cpu().numpy().astype(bool)
    b = bridge.bridge_rows(s0[None].astype(np.float32).astype(np.float64),
                           t0[None].astype(np.float32).astype(np.float64), eps)
    p, q, tv = np.exp(b["logp"][0]), np.exp(b["logq"][0]), float(b["tv"][0])
    assert np.allclose(out["tv"].cpu().numpy(), tv, rtol=1e-5)
    assert _pvalue(np.bincount(prop, minlength=V), p, n) > 1e-4       # z ~ p
    assert _pvalue(np.bincount(tok, minlength=V), q, n) > 1e-4        # y ~ q
    assert _pvalue(np.bincount(tok, minlength=V), p, n) < 1e-12       # and not p
    assert binomtest(int(C.sum()), n, tv).pvalue > 1e-4               # Pr(C) = TV
    r = np.maximum(q - p, 0.0) / tv
    assert _pvalue(np.bincount(tok[C], minlength=V), r, int(C.sum())) > 1e-4  # residual law


def test_gpu_rollout_has_sequential_q_law(saki_lib):
    """Prop. spec_exact end to end on the GPU path: 20,000 sequences of the
    synthetic model (V = 3, L = 3) from one prompt, k = 2 drafts per wave."""
    V, L, k, eps, N = 3, 3, 2, 0.2, 20_000
    law = orollout.sequential_law(SyntheticAR(V, seed=0), 0, V, L, eps).reshape(-1)
    plaw = orollout.sequential_law(SyntheticAR(V, seed=0), 0, V, L, 0.0).reshape(-1)
    mt = SyntheticARTorch(V, seed=0, device=DEV)
    say(f"gpu rollout law N={N}")
    tr, waves = saki_lib.rollout(mt, np.zeros(N, np.int64), k, L, eps, seed=77, dtype=torch.float32)
    torch.cuda.synchronize()
    toks = tr["tokens"].cpu().numpy().astype(np.int64)
    assert (tr["length"].cpu().numpy() == L).all()
    assert tr["corrected"].cpu().numpy().mean() > 0.1
    obs = np.bincount(toks @ (V ** np.arange(L - 1, -1, -1)), minlength=V ** L)
    assert _pvalue(obs, law, N) > 1e-4
    assert _pvalue(obs, plaw, N) < 1e-12
