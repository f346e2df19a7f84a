"""GPU-vs-oracle comparison rules for the coupling path.

Bar: accept/correct events, proposals, committed tokens, teacher argmax and
prefix lengths agree exactly, except where the decision was within 1e-6 of a
tie (|u - alpha| < 1e-6 for the accept test, or a relative gap < 1e-6 between
the best and second-best race keys); such rows are counted and reported.
lambda, KL, TV, accept probability, selected log-probabilities and row losses
agree to 1e-5 relative (absolute floor 1e-9, or 1e-6 for log-probabilities
and losses of magnitude below one); unscaled gradients to 2e-3 absolute.
"""
import numpy as np

from oracle import coupling, routing, supervision, verify

MARGIN = 1e-6
RTOL = 1e-5
ATOL = 1e-9
GRAD_ATOL = 2e-3


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
                   valid=None, grad_scale=1.0, target_sample=False):
    """Compare GPU outputs (dict of numpy arrays indexed by row) on `rows` with
    the oracle run on those rows' logits s, t (float64 arrays [len(rows), V]).
    target_sample: corrections were supervised on a teacher draw (App. C)."""
    R = report or Report()
    rows = np.asarray(rows)
    orc_all = [coupling.couple_rows(s[i:i + 1], t[i:i + 1], eps, seed, row_offset + int(r))
               for i, r in enumerate(rows)]
    for i, r in enumerate(rows):
        o = {k: (v[0] if isinstance(v, np.ndarray) and v.ndim >= 1 else v) for k, v in orc_all[i].items()}
        R.rows += 1
        g = {k: v[r] for k, v in gpu.items() if k not in ("grad", "loss_sum")}
        tag = f"row {r}"
        if int(g["row_status"]) != int(o["row_status"]):
            R.fail(f"{tag}: status {g['row_status']} vs {o['row_status']}")
            continue
        if o["row_status"] != 0:
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
            if not close(g[key], o[key], atol=1e-6):
                R.fail(f"{tag}: {key} {g[key]!r} vs {o[key]!r}")
            R.note(key, rel_err(g[key], o[key], atol=1e-6))
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
            M = None if valid is None else valid[r:r + 1]
            adv = o["logt_token"] - o["logp_token"]
            rl, _, og = routing.route_rows(s[i:i + 1], [o["token"]], [o["corrected"]], [target], [adv],
                                           M, grad_scale, want_grad=grad is not None)
            if not close(gpu["row_loss"][r], rl[0], atol=1e-6):
                R.fail(f"{tag}: row_loss {gpu['row_loss'][r]!r} vs {rl[0]!r}")
            R.note("row_loss", rel_err(gpu["row_loss"][r], rl[0], atol=1e-6))
            if grad is not None:
                err = float(np.max(np.abs(grad[i] - og[0])))
                R.note("grad_abs", err)
                if not err <= GRAD_ATOL:
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
