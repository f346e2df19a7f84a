"""GPU-vs-oracle comparison rules for the coupling path.

Bar: accept/correct events, proposals, committed tokens, teacher argmax and
prefix lengths agree exactly, except where the decision was within 1e-6 of a
tie (|u - alpha| < 1e-6 for the accept test, or a relative gap < 1e-6 between
the best and second-best race keys); such rows are counted and reported.
lambda, KL, TV and accept probability agree to 1e-5 relative (absolute floor
1e-9); selected log-probabilities to 1e-5 relative with an absolute floor of
1e-6 (fp32 accumulation of the row's normalisers), row losses to 1e-5
relative with that floor carried through the loss's formula (loss_atol);
unscaled gradients to 2e-3 absolute.
"""
import multiprocessing as mp
import os

import numpy as np

from oracle import coupling, routing, supervision, verify

MARGIN = 1e-6
RTOL = 1e-5
ATOL = 1e-9
GRAD_ATOL = 2e-3
LOGP_ATOL = 1e-6


def loss_atol(corrected, adv, logp_y):
    """Absolute part of the row-loss bound.  A row loss is -log p(target) at a
    correction and -A log p(y) at an accepted row, with A = log pi(y) - log p(y)
    a difference of two log-probabilities: each log-probability carries the
    absolute floor LOGP_ATOL of fp32 accumulation (rounding of the row's
    normalisers), which reaches the loss as LOGP_ATOL (|A| + 2 |log p(y)|) at an
    accepted row (the advantage's cancellation) and LOGP_ATOL at a correction."""
    if corrected:
        return LOGP_ATOL
    return LOGP_ATOL * (1.0 + abs(adv) + 2.0 * abs(logp_y))


def close(a, b, rtol=RTOL, atol=ATOL):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    return both_nan | (np.abs(a - b) <= rtol * np.abs(b) + atol)


def rel_err(a, b, atol=ATOL):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    m = ~(np.isnan(a) & np.isnan(b))
    if not m.any():
        return 0.0
    return float(np.max(np.abs(a[m] - b[m]) / (np.abs(b[m]) + atol / RTOL)))


class Report:
    def __init__(self):
        self.rows = 0
        self.near_margin = 0
        self.near_tie = 0
        self.failures = []
        self.max_rel = {}

    def note(self, key, err):
        self.max_rel[key] = max(self.max_rel.get(key, 0.0), err)

    def fail(self, msg):
        if len(self.failures) < 20:
            self.failures.append(msg)

    def summary(self):
        return (f"rows={self.rows} near_margin={self.near_margin} near_tie={self.near_tie} "
                f"max_rel={ {k: f'{v:.2e}' for k, v in self.max_rel.items()} }")

    def check(self):
        assert not self.failures, "\n".join(self.failures) + "\n" + self.summary()


def compare_couple(gpu, s, t, eps, seed, row_offset, rows, report=None, grad=None,
                   valid=None, grad_scale=1.0, target_sample=False, local=False, grad_rtol=0.0):
    """Compare GPU outputs (dict of numpy arrays indexed by row) on `rows` with
    the oracle run on those rows' logits s, t (float64 arrays [len(rows), V]).
    target_sample: corrections were supervised on a teacher draw (App. C).
    local: gpu arrays and valid hold only the listed rows, in order.
    grad_rtol: relative part of the gradient bound (2^-8 for a bf16 gradient,
    on top of the absolute 2e-3)."""
    R = report or Report()
    rows = np.asarray(rows)
    if not local:
        gpu = {k: (v[rows] if k not in ("grad", "loss_sum") else v) for k, v in gpu.items()}
        valid = None if valid is None else np.asarray(valid)[rows]
    orc_all = [coupling.couple_rows(s[i:i + 1], t[i:i + 1], eps, seed, row_offset + int(r))
               for i, r in enumerate(rows)]
    for i, r in enumerate(rows):
        o = {k: (v[0] if isinstance(v, np.ndarray) and v.ndim >= 1 else v) for k, v in orc_all[i].items()}
        R.rows += 1
        g = {k: v[i] for k, v in gpu.items() if k not in ("grad", "loss_sum")}
        tag = f"row {r}"
        if int(g["row_status"]) != int(o["row_status"]):
            R.fail(f"{tag}: status {g['row_status']} vs {o['row_status']}")
            continue
        if o["row_status"] != 0:
            # no coupling at this row: a masked row carries loss 0 and an
            # all-zero gradient row whatever its logits, a valid row NaN
            masked = valid is not None and not valid[i]
            if "row_loss" in gpu:
                rl = gpu["row_loss"][i]
                if not ((rl == 0.0) if masked else np.isnan(rl)):
                    R.fail(f"{tag}: row_loss {rl!r} at a row with status {o['row_status']} (masked {masked})")
            if grad is not None:
                ok = np.all(grad[i] == 0.0) if masked else np.all(np.isnan(grad[i]))
                if not ok:
                    R.fail(f"{tag}: gradient of a row with status {o['row_status']} (masked {masked}) is not "
                           f"{'all zero' if masked else 'all NaN'}")
            continue
        if int(g["teacher_argmax"]) != int(o["teacher_argmax"]):
            R.fail(f"{tag}: argmax {g['teacher_argmax']} vs {o['teacher_argmax']}")
        for key in ("lambda", "kl", "tv"):
            ok_key = "lam" if key == "lambda" else key
            if not close(g[key], o[ok_key]):
                R.fail(f"{tag}: {key} {g[key]!r} vs {o[ok_key]!r}")
            R.note(key, rel_err(g[key], o[ok_key]))
        gaps = o["gaps"]
        prop_tie = min(gaps[0], gaps[1]) < MARGIN
        if int(g["proposal"]) != int(o["proposal"]):
            if prop_tie:
                R.near_tie += 1
                continue
            R.fail(f"{tag}: proposal {g['proposal']} vs {o['proposal']} (gaps {gaps[:2]})")
            continue
        if not close(g["accept_prob"], o["accept_prob"]):
            R.fail(f"{tag}: alpha {g['accept_prob']!r} vs {o['accept_prob']!r}")
        R.note("accept_prob", rel_err(g["accept_prob"], o["accept_prob"]))
        if int(g["corrected"]) != int(o["corrected"]):
            if o["margin"] < MARGIN:
                R.near_margin += 1
                continue
            R.fail(f"{tag}: corrected {g['corrected']} vs {o['corrected']} margin {o['margin']}")
            continue
        if int(g["token"]) != int(o["token"]):
            if o["corrected"] and min(gaps[2], gaps[3]) < MARGIN:
                R.near_tie += 1
                continue
            R.fail(f"{tag}: token {g['token']} vs {o['token']} (gaps {gaps})")
            continue
        for key in ("logp_token", "logt_token", "logq_token"):
            if not close(g[key], o[key], atol=LOGP_ATOL):
                R.fail(f"{tag}: {key} {g[key]!r} vs {o[key]!r}")
            R.note(key, rel_err(g[key], o[key], atol=LOGP_ATOL))
        # the gradient's target: y, or at a correction v* / the teacher draw
        tgt, tgaps = supervision.correction_targets(orc_all[i], t[i:i + 1], seed, row_offset + int(r),
                                                    sample=target_sample)
        target = int(tgt[0])
        if "target" in g and int(g["target"]) != target:
            if min(tgaps[0]) < MARGIN:
                R.near_tie += 1
                continue
            R.fail(f"{tag}: target {g['target']} vs {target} (gaps {tgaps[0]})")
            continue
        if "row_loss" in gpu:
            M = None if valid is None else valid[i:i + 1]
            adv = o["logt_token"] - o["logp_token"]
            rl, _, og = routing.route_rows(s[i:i + 1], [o["token"]], [o["corrected"]], [target], [adv],
                                           M, grad_scale, want_grad=grad is not None)
            if not close(gpu["row_loss"][i], rl[0], atol=loss_atol(o["corrected"], adv, o["logp_token"])):
                R.fail(f"{tag}: row_loss {gpu['row_loss'][i]!r} vs {rl[0]!r} (A {adv!r})")
            R.note("row_loss", rel_err(gpu["row_loss"][i], rl[0], atol=1e-6))
            if grad is not None:
                dif = np.abs(grad[i] - og[0])
                err = float(np.max(dif))
                R.note("grad_abs", err)
                if not np.all(dif <= GRAD_ATOL + grad_rtol * np.abs(og[0])):
                    R.fail(f"{tag}: grad max abs err {err}")
    return R


def compare_verify(gpu, s, t, k, draft, eps, seed, row_offset, blocks, eos_id=-1, report=None):
    """gpu: dict with accepted_len, correction (per block) and per_pos arrays.
    s, t, draft: the rows of the listed blocks only (block-major)."""
    R = report or Report()
    for i, b in enumerate(blocks):
        sl = slice(i * k, (i + 1) * k)
        o = verify.verify_blocks(s[sl], t[sl], k, draft[sl], eps, seed,
                                 row_offset + int(b) * k, eos_id)
        R.rows += 1
        n_g, c_g = int(gpu["accepted_len"][b]), int(gpu["correction"][b])
        n_o, c_o = int(o["accepted_len"][0]), int(o["correction"][0])
        # near-tie accept decisions inside the evaluated prefix excuse a mismatch
        first = min(n_g, n_o)
        if n_g != n_o:
            j = first
            if j < k and o["evaluated"][j] and o["margin"][j] < MARGIN:
                R.near_margin += 1
                continue
            R.fail(f"block {b}: n {n_g} vs {n_o} (margins {o['margin']})")
            continue
        if c_g != c_o:
            if min(o["gaps"][0]) < MARGIN:
                R.near_tie += 1
                continue
            R.fail(f"block {b}: correction {c_g} vs {c_o}")
            continue
        pp = gpu.get("per_pos")
        if pp is not None:
            for j in range(k):
                r = int(b) * k + j
                if not o["evaluated"][j]:
                    continue
                for key, okey in (("lambda", "lam"), ("kl", "kl"), ("accept_prob", "accept_prob")):
                    if not close(pp[key][r], o[okey][j]):
                        R.fail(f"block {b} pos {j}: {key} {pp[key][r]!r} vs {o[okey][j]!r}")
                    R.note(key, rel_err(pp[key][r], o[okey][j]))
    return R


def merge(reports):
    R = Report()
    for r in reports:
        R.rows += r.rows
        R.near_margin += r.near_margin
        R.near_tie += r.near_tie
        for f in r.failures:
            R.fail(f)
        for k, v in r.max_rel.items():
            R.note(k, v)
    return R


def workers():
    """Worker processes for oracle comparisons: the CPU share of the machine,
    at most 16 (the share of one GPU on the test machines)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _couple_job(args):
    gpu, s, t, eps, seed, row_offset, rows, grad, valid, grad_scale, target_sample, grad_rtol = args
    return compare_couple(gpu, s, t, eps, seed, row_offset, rows, grad=grad, valid=valid,
                          grad_scale=grad_scale, target_sample=target_sample, local=True,
                          grad_rtol=grad_rtol)


def _verify_job(args):
    gpu, s, t, k, draft, eps, seed, row_offset, blocks, eos_id = args
    return compare_verify(gpu, s, t, k, draft, eps, seed, row_offset, blocks, eos_id)


THREAD_VARS = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")


def _pool_map(fn, jobs):
    if len(jobs) == 1:
        return [fn(jobs[0])]
    # spawned workers (the parent has a GPU context, which must not be
    # forked), whose numerical libraries start single-threaded: the variables
    # are set before the workers import numpy
    saved = {k: os.environ.get(k) for k in THREAD_VARS}
    for k in THREAD_VARS:
        os.environ[k] = "1"
    try:
        pool = mp.get_context("spawn").Pool(len(jobs))
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    with pool:
        return pool.map(fn, jobs)


def compare_couple_pool(gpu, s, t, eps, seed, row_offset, rows, grad=None, valid=None,
                        grad_scale=1.0, target_sample=False, n_workers=None, grad_rtol=0.0):
    """compare_couple with the listed rows split over worker processes.
    gpu: per-row outputs of all rows (indexed by row); s, t, grad: the listed
    rows only, in order (float64)."""
    rows = np.asarray(rows)
    parts = [p for p in np.array_split(np.arange(len(rows)), min(n_workers or workers(), max(1, len(rows))))
             if len(p)]
    jobs = []
    for p in parts:
        sub = rows[p]
        g = {k: v[sub] for k, v in gpu.items() if k not in ("grad", "loss_sum", "row_loss_sum")}
        jobs.append((g, s[p], t[p], eps, seed, row_offset, sub, None if grad is None else grad[p],
                     None if valid is None else np.asarray(valid)[sub], grad_scale, target_sample, grad_rtol))
    return merge(_pool_map(_couple_job, jobs))


def compare_verify_pool(gpu, s, t, k, draft, eps, seed, row_offset, blocks, eos_id=-1, n_workers=None):
    """compare_verify with the listed blocks split over worker processes.
    s, t, draft: the rows of the listed blocks only (block-major, in order)."""
    blocks = np.asarray(blocks)
    parts = [p for p in np.array_split(np.arange(len(blocks)), min(n_workers or workers(), max(1, len(blocks))))
             if len(p)]
    jobs = []
    for p in parts:
        idx = np.concatenate([np.arange(i * k, (i + 1) * k) for i in p])
        jobs.append((gpu, s[idx], t[idx], k, draft[idx], eps, seed, row_offset, blocks[p], eos_id))
    return merge(_pool_map(_verify_job, jobs))
