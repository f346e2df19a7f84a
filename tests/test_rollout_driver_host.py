"""Host logic of the rollout driver (paper_2609_36601_amd/speculative.py) on the CPU.

The three library calls are replaced by stand-ins built on the oracle, with
the same argument conventions as the binding (dense outputs, block-major rows,
strided draft-prefix logits), so the driver's own work is checked: the
logits buffers and their views, the RNG row keys of each call, the
position-major to block-major draft copy, and the model state after each
commit (the rollback).  Its trajectories must equal the oracle rollout's.
"""
import numpy as np
import pytest
import torch

from oracle import rollout as orollout
from oracle.bridge import log_softmax
from oracle.verify import verify_blocks
from paper_2609_36601_amd import binding, speculative
from paper_2609_36601_amd.workloads import SyntheticAR, SyntheticARTorch


def _np(t):
    return t.detach().double().numpy() if t.is_floating_point() else t.numpy()


def fake_sample(student, token, seed, row_offset=0, row_step=1, row_status=None, stream=None):
    assert token.is_contiguous() and student.stride(1) == 1
    z, _, _ = orollout.draft_tokens(_np(student), seed, row_offset, row_step)
    token.copy_(torch.as_tensor(z, dtype=torch.int32))


def fake_verify(student, teacher, k, draft, eps, seed, row_offset=0, eos_id=-1, accepted_len=None,
                correction=None, per_pos=None, workspace=None, stream=None):
    assert draft.is_contiguous()
    s, t, d = _np(student), _np(teacher), _np(draft).astype(np.int64)
    v = verify_blocks(s, t, k, d, eps, seed, row_offset=row_offset, eos_id=eos_id)
    accepted_len.copy_(torch.as_tensor(v["accepted_len"], dtype=torch.int32))
    correction.copy_(torch.as_tensor(v["correction"], dtype=torch.int32))
    R = s.shape[0]
    tok = d.copy()
    for b in range(R // k):
        if v["correction"][b] >= 0:
            tok[b * k + v["accepted_len"][b]] = v["correction"][b]
    logpi = np.stack([log_softmax(t[r]) for r in range(R)])
    vals = dict(token=tok, **{"lambda": v["lam"]}, kl=v["kl"], tv=v["tv"],
                logp_token=v["logp"][np.arange(R), tok], logt_token=logpi[np.arange(R), tok],
                teacher_argmax=np.argmax(t, axis=1))
    for key, val in vals.items():
        if key in per_pos:
            per_pos[key].copy_(torch.as_tensor(val).to(per_pos[key].dtype))


def fake_commit(traj, max_len, k, eos_id, accepted_len, correction, per_pos, n_commit=None,
                stream=None):
    names = dict(lam="lambda", kl="kl", tv="tv", logp="logp_token", logt="logt_token",
                 teacher_argmax="teacher_argmax", tokens="tokens", corrected="corrected",
                 length="length", done="done")
    t_o = {o: _np(traj[g]).astype(np.float64 if traj[g].is_floating_point() else np.int64)
           for o, g in names.items()}
    pp = dict(token=_np(per_pos["token"]).astype(np.int64))
    for o in ("lam", "kl", "tv", "logp", "logt", "teacher_argmax"):
        pp[o] = _np(per_pos[names[o]])
    n = orollout.commit_wave(t_o, k, eos_id, _np(accepted_len), _np(correction), pp)
    for o, g in names.items():
        traj[g].copy_(torch.as_tensor(t_o[o]).to(traj[g].dtype))
    if n_commit is not None:
        n_commit.copy_(torch.as_tensor(n, dtype=torch.int32))


@pytest.fixture
def fakes(monkeypatch):
    monkeypatch.setattr(speculative._b, "saki_sample", fake_sample)
    monkeypatch.setattr(speculative._b, "saki_spec_verify", fake_verify)
    monkeypatch.setattr(speculative._b, "saki_commit", fake_commit)


@pytest.mark.parametrize("k,eos,dtype", [(3, -1, torch.float32), (4, 5, torch.bfloat16),
                                         (1, -1, torch.float32)])
def test_driver_matches_oracle_rollout(fakes, k, eos, dtype):
    V, B, L, eps, seed = 12, 8, 9, 0.1, 17
    mt = SyntheticARTorch(V, seed=3, device="cpu")
    tr, waves = speculative.rollout(mt, np.arange(B), k, L, eps, seed, eos_id=eos, dtype=dtype)
    o = orollout.rollout(SyntheticAR(V, seed=3), np.arange(B), k, L, eps, seed, eos_id=eos)
    assert waves == o["waves"]
    for key, ok in (("tokens", "tokens"), ("corrected", "corrected"), ("length", "length"),
                    ("done", "done"), ("teacher_argmax", "teacher_argmax")):
        np.testing.assert_array_equal(tr[key].numpy(), o[ok], err_msg=key)
    for key, ok in (("lambda", "lam"), ("tv", "tv"), ("kl", "kl")):
        np.testing.assert_allclose(tr[key].double().numpy(), o[ok], rtol=1e-6, atol=1e-9)
    if eos >= 0:
        assert (o["length"] < L).any()


def test_driver_zero_length(fakes):
    mt = SyntheticARTorch(10, seed=0, device="cpu")
    tr, waves = speculative.rollout(mt, np.arange(3), 2, 0, 0.1, 1)
    assert waves == 0 and (tr["done"] == binding.SEQ_FINISHED).all()


def test_dense_outputs_are_required():
    x = torch.zeros(4, 3, dtype=torch.int32)
    with pytest.raises(ValueError):
        binding._dense(x[:, 1])
    binding._dense(x[1], None)
