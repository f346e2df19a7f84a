"""Speculative rollout driver: waves of draft, verify, commit (SAKI App. I).

Each wave, for every sequence of the batch,
  1. the student drafts k tokens from the committed prefix
     (saki_sample on the logits at each draft prefix);
  2. the teacher is evaluated on the k draft prefixes and the block is
     verified with first-rejection semantics (saki_spec_verify);
  3. the accepted drafts and the correction are committed into token-aligned
     trajectories, later draft states are dropped (saki_commit);
and the model continues from the new committed prefix.  Every step of the
method runs in libsaki; this module only orders the calls and keeps the
model's state, all on the device, with one host synchronisation every
`check_every` waves to stop once every sequence is done (finished sequences
are masked on the device, not compacted).  The committed trajectories have
the law of sequential exact-q sampling (App. F, Prop. spec_exact).

`model` is the caller's autoregressive pair of networks, any object with
    V, device
    initial(prompt_ids) -> int64 states [B]
    advance(states, tokens) -> states after appending the tokens
    logits_into(states, s_out, t_out)   student / teacher logits of the
                                        prefixes, written into [n, V] views
(workloads.SyntheticARTorch is a synthetic one).

Keying: draft j of sequence b in wave w and its verification share the
global row g = w * B * k + b * k + j, so drafts equal the proposals the
coupling would draw at those rows.
"""
import torch

from . import binding as _b

META_FIELDS = ["lambda", "kl", "tv", "logp_token", "logt_token", "teacher_argmax", "token",
               "corrected", "row_status"]
# what the routed objective needs per committed token: the token, the
# correction flag, the teacher mode and log p, log pi of the token (for the
# advantage); without lambda*, KL and TV the verification can accept a draft
# below its lambda-free accept bound without the lambda search
OBJECTIVE_FIELDS = ["logp_token", "logt_token", "teacher_argmax", "token", "corrected", "row_status"]


def rollout(model, prompts, k, max_len, eps, seed, eos_id=-1, dtype=torch.bfloat16,
            check_every=1, max_waves=None, stream=None, timing=None, metadata="full"):
    """Runs waves until every sequence is done; returns (trajectories, waves).

    trajectories: dict of device tensors as in binding.alloc_traj: tokens,
    corrected, lambda, kl, tv, logp_token, logt_token, teacher_argmax
    [B, max_len] and length, done [B].
    metadata: "full" (every field above) or "objective" (lambda, kl and tv are
    left NaN: the fields the routed objective needs, and a faster verification).
    timing: optional dict; if given, (start, end) event pairs recorded on the
    current stream around the library calls are appended to timing["sample"],
    timing["verify"] and timing["commit"], and each wave's accepted lengths
    (a device tensor) to timing["accepted_len"].
    """
    dev = torch.device(model.device)
    prompts = torch.as_tensor(prompts, dtype=torch.int64, device=dev)
    B = prompts.numel()
    V = model.V
    traj = _b.alloc_traj(B, max_len, dev)
    if max_len <= 0:
        traj["done"].fill_(_b.SEQ_FINISHED)
        return traj, 0
    # logits of the B * k draft prefixes, block-major rows b * k + j
    S = _b.alloc_rows(B * k, V, dtype, dev)
    T = _b.alloc_rows(B * k, V, dtype, dev)
    S3 = S.view(B, k, V) if S.is_contiguous() else S.as_strided((B, k, V), (k * S.stride(0), S.stride(0), 1))
    H = torch.empty(B, k + 1, dtype=torch.int64, device=dev)
    D = torch.empty(k, B, dtype=torch.int32, device=dev)       # drafts, position-major
    drafts = torch.empty(B, k, dtype=torch.int32, device=dev)  # block-major for verification
    if metadata not in ("full", "objective"):
        raise ValueError("metadata must be 'full' or 'objective'")
    wanted = META_FIELDS if metadata == "full" else OBJECTIVE_FIELDS
    pp = _b.alloc_couple_out(B * k, dev, fields=[f for f in _b.COUPLE_FIELDS if f in wanted])
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    corr = torch.empty(B, dtype=torch.int32, device=dev)
    n_commit = torch.empty(B, dtype=torch.int32, device=dev)
    ws = torch.empty(max(_b.workspace_bytes(_b.SAKI_OP_VERIFY, B * k, V), 8), dtype=torch.uint8, device=dev)
    state = model.initial(prompts)

    def timed(name, fn, *a, **kw):
        if timing is None:
            return fn(*a, **kw)
        st = torch.cuda.current_stream() if stream is None else stream
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        fn(*a, **kw)
        e1.record(st)
        timing.setdefault(name, []).append((e0, e1))

    limit = max_waves if max_waves is not None else max_len + 1
    wave = 0
    while wave < limit:
        g0 = wave * B * k
        H[:, 0] = state
        for j in range(k):
            model.logits_into(H[:, j], S3[:, j], None)
            timed("sample", _b.saki_sample, S3[:, j], D[j], seed, row_offset=g0 + j, row_step=k,
                  stream=stream)
            H[:, j + 1] = model.advance(H[:, j], D[j].clamp(min=0))
        drafts.copy_(D.t())
        model.logits_into(H[:, :k].reshape(-1), None, T)
        timed("verify", _b.saki_spec_verify, S, T, k, drafts.view(-1), eps, seed, row_offset=g0,
              eos_id=eos_id, accepted_len=acc, correction=corr, per_pos=pp, workspace=ws, stream=stream)
        if timing is not None:
            timing.setdefault("accepted_len", []).append(acc.clone())
        timed("commit", _b.saki_commit, traj, max_len, k, eos_id, acc, corr, pp, n_commit,
              stream=stream)
        # the model continues from the committed prefix: the draft state after
        # m - 1 drafts, advanced by the last committed token (rollback of the rest)
        m = n_commit.long()
        prev = H.gather(1, (m - 1).clamp(min=0)[:, None])[:, 0]
        last = traj["tokens"].gather(1, (traj["length"].long() - 1).clamp(min=0)[:, None])[:, 0]
        state = torch.where(m > 0, model.advance(prev, last.long()), state)
        wave += 1
        if wave % check_every == 0 and not bool((traj["done"] == _b.SEQ_RUNNING).any()):
            break
    return traj, wave
