"""Throughput of the coupled + routed path (with gradient) on one MI355X.

One step = one saki_couple call with fused routing and an fp32 gradient over
the whole 'large' workload: 64 sequences x 1024 positions = 65,536 rows of
V = 151,936 bf16 student and teacher logits, resident in HBM.  Prints one
JSON line.  --gpus N with N > 1 exits: the library runs on one GPU.
"""
import argparse
import json
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s

# The sources each measured kernel is built from (the rollout kernels live in a
# header of their own, which these kernels do not use).
_CORE_SOURCES = ["include/saki.h", "paper_2609_36601_amd/csrc/saki.hip", "paper_2609_36601_amd/csrc/row_engine.hpp",
                 "paper_2609_36601_amd/csrc/device_util.hpp"]
KERNEL_SOURCES = {"couple": _CORE_SOURCES, "route": _CORE_SOURCES, "verify": _CORE_SOURCES, "stream": _CORE_SOURCES,
                  "probe": _CORE_SOURCES + ["paper_2609_36601_amd/csrc/probe.hpp"]}

# HBM traffic of one step of the dominant kernel, from two rocprofv3 --pmc runs
# (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch): the couple kernel on the large
# workload at eps 0.2 (its main launch and the short launch that redoes flagged
# rows, profiles/couple_kernel_large.md), the verify kernel on the verification
# workload (profiles/verify_kernel.md), the couple kernel on one 4,096-row chunk
# of the long-rollout workload (mean of five chunks, profiles/couple_kernel_stream.md),
# the route kernel on the large workload's coupled rows
# (profiles/route_kernel_large.md) and the probe kernel on 4,096 of them
# (profiles/probe_kernel_large.md).  A plain 1 GiB device copy in the same runs
# reads FETCH_SIZE = 524,300-524,320 KiB and WRITE_SIZE = 1,048,576 KiB, so
# FETCH_SIZE is scaled by 2.0 and WRITE_SIZE by 1.0.  Keyed by the SHA-256 of
# the kernel's sources: a changed kernel reports traffic = null until re-measured.
_CORE_HASH = "fab9e12252029b7344abf907affbc80908491c42be492c4d9797e374b81230dd"
MEASURED_TRAFFIC = {
    "couple": {_CORE_HASH: dict(fetch_kib=38406715.5 + 59.8, write_kib=41888169.2 + 5648.0,
                                fetch_scale=2.0, write_scale=1.0)},
    "verify": {_CORE_HASH: dict(fetch_kib=13062836.5, write_kib=97980.9, fetch_scale=2.0, write_scale=1.0)},
    "stream": {_CORE_HASH: dict(fetch_kib=2662206.5, write_kib=2924365.7, fetch_scale=2.0, write_scale=1.0)},
    "route": {_CORE_HASH: dict(fetch_kib=17097281.9, write_kib=41756980.5, fetch_scale=2.0, write_scale=1.0)},
    "probe": {"a242e6a694f019423bc917d1dada40291711f9267150294d94c60238e7bdba2c":
              dict(fetch_kib=1284932.0, write_kib=975.4, fetch_scale=2.0, write_scale=1.0)},
}


# VALU instructions (wave64, SQ_INSTS_VALU) of one launch of the dominant
# kernel, from the rocprofv3 --pmc run of the same sources (the couple kernel
# on the large workload at eps 0.2, the verify kernel on the verification
# workload).  Their issue rate is the bound these kernels meet first: a CU
# issues at most one wave64 VALU instruction per cycle (four SIMDs of 16 lanes,
# four cycles each), 256 CUs x 2.4 GHz = 6.14e11 per second.
VALU_ISSUE_PEAK = 256 * 2.4e9
MEASURED_VALU = {
    "couple": {_CORE_HASH: 9.762e9},
    "verify": {_CORE_HASH: 3.113e9},
}


def valu_issue(workload, ms):
    """The measured VALU instructions per launch over the launch time, against
    the issue peak (None when the kernel changed after its counters)."""
    n = MEASURED_VALU.get(workload, {}).get(kernel_source_hash(workload))
    if n is None:
        return None
    achieved = n / (ms * 1e-3)
    return {"instructions": n, "achieved": achieved, "peak": VALU_ISSUE_PEAK, "unit": "wave64 instr/s",
            "frac": achieved / VALU_ISSUE_PEAK}


def kernel_source_hash(workload="couple"):
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[workload]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic_bytes(workload="couple"):
    m = MEASURED_TRAFFIC.get(workload, {}).get(kernel_source_hash(workload))
    if m is None:
        return None
    return (m["fetch_kib"] * m["fetch_scale"] + m["write_kib"] * m["write_scale"]) * 1024.0


def stream_traffic_bytes(n_chunks, rows):
    """HBM bytes of the whole long-rollout step: the measured mean of one
    4,096-row launch times the launches, for the full 262,144 rows only."""
    per = measured_traffic_bytes("stream")
    if per is None or rows != 262144 or n_chunks != 64:
        return None
    return per * n_chunks


def _oracle_rows(args):
    """CPU oracle on rows, in order, until `budget` seconds of work (a worker process)."""
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    import numpy as np
    from oracle import coupling, routing
    s, t, eps, seed, offsets, budget = args
    t0 = time.perf_counter()
    done = 0
    for i in range(s.shape[0]):
        si = s[i:i + 1].astype(np.float64)
        ti = t[i:i + 1].astype(np.float64)
        ev = coupling.couple_rows(si, ti, eps, seed, int(offsets[i]))
        routing.couple_and_route(ev, si, None, 1.0, want_grad=True)
        done += 1
        if time.perf_counter() - t0 >= budget:
            break
    return done, time.perf_counter() - t0


def cpu_info():
    """The host's CPU model (from /proc/cpuinfo), its logical CPUs and the
    CPUs this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count() or 1
    return model, os.cpu_count() or 1, affinity


def cpu_workers():
    """Worker processes for the CPU baseline: every CPU this process may run
    on, at most 16 (the CPU share of one GPU on the measuring machines)."""
    return max(1, min(16, cpu_info()[2]))


THREAD_VARS = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")


def single_threaded_pool(n):
    """A pool of n spawned worker processes whose numerical libraries start
    single-threaded (the variables are set before the workers import numpy)."""
    saved = {k: os.environ.get(k) for k in THREAD_VARS}
    for k in THREAD_VARS:
        os.environ[k] = "1"
    try:
        return mp.get_context("spawn").Pool(n)
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def _pool_rows(S, T, eps, seed, rows, workers, budget):
    parts = [np.arange(w, len(rows), workers) for w in range(workers)]
    jobs = [(S[p], T[p], eps, seed, rows[p], budget) for p in parts if len(p)]
    with single_threaded_pool(len(jobs)) as pool:
        pool.map(_noop, range(len(jobs)))  # start the workers before timing
        t0 = time.perf_counter()
        res = pool.map(_oracle_rows, jobs)
        wall = time.perf_counter() - t0
    return sum(r[0] for r in res), sum(r[1] for r in res), wall, len(jobs)


def cpu_baseline(s, t, eps, seed, n_sample=512, budget=1.5, budget_single=6.0, n_full=None):
    """The float64 oracle (as it stands) on a bounded sample of the same rows:
    n_sample evenly spaced rows, split over one single-threaded worker process
    per available CPU (at most 16), each stopping after `budget` seconds of
    work; then one worker alone for `budget_single` seconds (the single-core
    rate).  n_full: rows of the full configuration, for the extrapolated time
    the oracle would take on all of them."""
    import torch
    n = s.shape[0]
    rows = np.linspace(0, n - 1, n_sample).astype(np.int64)
    idx = torch.as_tensor(rows, device=s.device)
    S = s[idx].float().cpu().numpy()
    T = t[idx].float().cpu().numpy()
    workers = cpu_workers()
    done, busy, wall, used = _pool_rows(S, T, eps, seed, rows, workers, budget)
    done1, busy1, wall1, _ = _pool_rows(S, T, eps, seed, rows, 1, budget_single)
    model, host_cpus, affinity = cpu_info()
    value, single = done / wall, done1 / wall1
    n_full = n_full or n
    return dict(value=value, unit="positions/s", cores=used, kind="oracle",
                sample=f"{done} rows of the same workload (from {n_sample} evenly spaced), coupling + "
                       f"routed loss + gradient, {used} single-threaded worker processes each stopping "
                       f"after {budget:.2f} s ({busy:.1f} s of CPU work in {wall:.1f} s wall); then "
                       f"{done1} rows on one core in {wall1:.1f} s",
                cpu_model=model, host_cpus=host_cpus, affinity_cpus=affinity,
                single_core_value=single,
                full_config_rows=n_full,
                full_config_oracle_s=n_full / value, full_config_oracle_s_single_core=n_full / single)


def _noop(x):
    return x


def attainable_read_gbs(dev, gib=4, reps=5):
    """HBM read bandwidth a plain streaming reduction reaches on this GPU (GB/s).

    A reference point for the roofline, measured with torch's own sum over a
    buffer larger than every cache (read as float64, the fastest of torch's
    reductions here); it is not part of the coupling path.
    """
    import torch
    x = torch.ones(gib << 27, dtype=torch.float64, device=dev)
    x.sum()
    torch.cuda.synchronize()
    best = float("inf")
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        x.sum()
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    n = x.numel() * x.element_size()
    del x
    torch.cuda.empty_cache()
    return n / (best * 1e-3) / 1e9


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--eps", type=float, default=0.2)
    ap.add_argument("--rows", type=int, default=None, help="override the row count (debug)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the headline configuration (no other radii, verify or stream keys)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one 1 GiB device copy before timing (counter calibration)")
    ap.add_argument("--metadata", choices=("full", "objective"), default="objective",
                    help="rollout workload: per-token metadata kept (objective: without lambda, KL, TV)")
    ap.add_argument("--workload", choices=("couple", "verify", "stream", "rollout", "route", "probe"), default="couple",
                    help="couple: the headline (coupling + routed loss + fp32 gradient); "
                         "verify: speculative verification of 8,192 blocks of k = 8; "
                         "route: saki_route_loss alone on the large workload's coupled rows; "
                         "probe: probe metrics (Top-16) on 4,096 rows of the large workload; "
                         "stream: the long-rollout stress workload, 262,144 rows in 64 chunks; "
                         "rollout: speculative rollout waves, 256 sequences x 64 tokens, k = 8")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(rows shard across GPUs without communication: each GPU takes a row range with its own row_offset)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_36601_amd as saki
    from paper_2609_36601_amd import workloads

    saki.load()
    dev = torch.device("cuda:0")
    if args.workload == "verify":
        return bench_verify(args, saki, workloads, dev)
    if args.workload == "rollout":
        return bench_rollout(args, saki, workloads, dev)
    if args.workload == "stream":
        return bench_stream(args, saki, workloads, dev)
    if args.workload == "route":
        return bench_route(args, saki, workloads, dev)
    if args.workload == "probe":
        return bench_probe(args, saki, workloads, dev)
    cfg = workloads.CONFIGS["large"]
    n = args.rows or cfg["rows"]
    V = cfg["V"]
    seed = workloads.coupling_seed("large")
    print(f"# generating {n} x {V} bf16 student/teacher rows", file=sys.stderr, flush=True)
    s = torch.empty(n, V, dtype=torch.bfloat16, device=dev)
    t = torch.empty_like(s)
    workloads.fill("large", s, t)
    grad = torch.empty(n, V, dtype=torch.float32, device=dev)
    out = saki.alloc_couple_out(n, dev)
    route = dict(valid_mask=None, grad_scale=1.0 / n,
                 row_loss=torch.empty(n, dtype=torch.float32, device=dev),
                 loss_sum=torch.empty(1, dtype=torch.float64, device=dev), grad=grad)
    ws = torch.empty(max(saki.workspace_bytes(saki.SAKI_OP_COUPLE, n, V), 8), dtype=torch.uint8,
                     device=dev)
    torch.cuda.synchronize()
    if args.calibrate_copy:
        calibration_copy(dev)

    ms, per, wall = time_calls(lambda: saki.saki_couple(s, t, args.eps, seed, 0, out, route, ws),
                               args.steps, args.warmup)
    print(f"# per-step ms: {[round(x, 3) for x in per]} (wall {wall:.3f} s)", file=sys.stderr, flush=True)

    bytes_per_row = 2 * V * 2 + V * 4  # s + t read once (bf16), fp32 gradient written once
    achieved = n * bytes_per_row / (ms * 1e-3) / 1e9
    corr_rate = float(out["corrected"].float().mean())
    near_margin = near_margin_rows(out)
    mean_tv = float(out["tv"].mean())
    mean_lam = float(out["lambda"].mean())
    print(f"# correction rate {corr_rate:.4f}, mean TV {mean_tv:.4f}, mean lambda {mean_lam:.4f}",
          file=sys.stderr, flush=True)

    attainable = attainable_read_gbs(dev)
    print(f"# attainable HBM read bandwidth (streaming reduction): {attainable:.0f} GB/s", file=sys.stderr,
          flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(s, t, args.eps, seed, n_full=n)
        print(f"# cpu baseline: {cpu}", file=sys.stderr, flush=True)

    # the rest of the metric's configurations, in the same run: the large
    # workload at the sweep's other radii, speculative verification and the
    # long-rollout stress workload
    others = {}
    if not args.headline_only and n == cfg["rows"]:
        steps_o = max(1, min(args.steps, 10))
        for eps_o in cfg["eps"]:
            if eps_o == args.eps:
                continue
            ms_o, per_o, _ = time_calls(lambda: saki.saki_couple(s, t, eps_o, seed, 0, out, route, ws),
                                        steps_o, 1)
            ach_o = n * bytes_per_row / (ms_o * 1e-3) / 1e9
            others[f"large_eps{eps_o}"] = dict(
                workload=f"large at eps {eps_o}: 65,536 rows, V=151,936 bf16, coupling + routed loss + fp32 grad",
                value=n / (ms_o * 1e-3), unit="positions/s", ms_per_step=ms_o, steps=steps_o,
                roofline=dict(bound="hbm", achieved=ach_o, peak=HBM_PEAK_GBS, unit="GB/s", frac=ach_o / HBM_PEAK_GBS),
                stats=dict(correction_rate=float(out["corrected"].float().mean()),
                           mean_tv=float(out["tv"].mean()), mean_lambda=float(out["lambda"].mean()),
                           near_margin_rows=near_margin_rows(out)))
            print(f"# large eps {eps_o}: {ms_o:.3f} ms", file=sys.stderr, flush=True)
        del out, route, ws
        # the verify workload in the same (n, V) buffers
        others["verify"] = verify_suite(saki, workloads, dev, s, t, steps_o, 1)
        print(f"# verify: {others['verify']['ms_per_step']:.3f} ms", file=sys.stderr, flush=True)
        # the long-rollout workload in the first 4,096 rows of the buffers
        others["stream"] = stream_suite(saki, workloads, dev, s, t, grad, 1)
        print(f"# stream: {others['stream']['ms_per_step']:.2f} ms", file=sys.stderr, flush=True)

    line = {
        "metric": "coupled+routed positions/sec at V=151,936 bf16; % of MI355X peak HBM GB/s",
        "value": n / (ms * 1e-3),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"logits": "bf16", "arithmetic": "f32, row sums and the lambda solve in f64", "workload": "large: 64 seq x 1024 pos = 65,536 rows, V=151,936 bf16, "
                               "rho~U(0.3,0.95), coupling + routed loss + fp32 grad",
                   "rows": n, "vocab": V, "eps": args.eps, "grad_dtype": "f32"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "attainable_read": attainable, "frac_attainable": achieved / attainable,
                     "traffic": measured_traffic_bytes() if n == cfg["rows"] and args.eps == 0.2 else None,
                     "valu_issue": valu_issue("couple", ms) if n == cfg["rows"] and args.eps == 0.2 else None},
        "cpu_baseline": cpu,
        "stats": {"correction_rate": corr_rate, "mean_tv": mean_tv, "mean_lambda": mean_lam,
                  "near_margin_rows": near_margin},
        "other_configs": others,
    }
    print(json.dumps(line), flush=True)


def near_margin_rows(out):
    """Rows whose accept decision lies within 1e-6 of its threshold (|u - alpha|):
    the rows a comparison with the oracle may excuse."""
    return int((out["margin"] < 1e-6).sum())


def calibration_copy(dev):
    """One plain 1 GiB device-to-device copy: its FETCH_SIZE / WRITE_SIZE per
    byte moved scales the counters read for the measured kernel in the same run."""
    import torch
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def time_calls(call, steps, warmup):
    """Times `call` (library calls enqueued on torch's current stream) with HIP
    events: `warmup` untimed calls, then `steps` timed ones; returns the mean
    ms, the per-call ms and the wall time of the timed calls."""
    import torch
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t_wall = time.perf_counter()
    ev[0].record(stream)
    for i in range(steps):
        call()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return sum(per) / len(per), per, wall


def verify_suite(saki, workloads, dev, s, t, steps, warmup):
    """The verify workload (8,192 blocks of k = 8, V = 151,936 bf16, eps 0.2,
    accepted lengths and corrections only) generated into the buffers s, t."""
    import torch
    cfg = workloads.CONFIGS["verify"]
    k, V = cfg["k"], cfg["V"]
    n = s.shape[0] - s.shape[0] % k
    nb = n // k
    workloads.fill("verify", s[:n], t[:n])
    draft = workloads.drafts(s[:n])
    seed = workloads.coupling_seed("verify")
    acc = torch.empty(nb, dtype=torch.int32, device=dev)
    corr = torch.empty(nb, dtype=torch.int32, device=dev)
    ws = torch.empty(max(saki.workspace_bytes(saki.SAKI_OP_VERIFY, n, V), 8), dtype=torch.uint8, device=dev)
    ms, per, _ = time_calls(lambda: saki.saki_spec_verify(s[:n], t[:n], k, draft, 0.2, seed, 0, -1, acc, corr,
                                                          None, ws), steps, warmup)
    al = acc.cpu().numpy()
    evaluated = int(np.minimum(al + 1, k).sum())  # positions each block reads before it stops
    achieved = evaluated * 2 * V * 2 / (ms * 1e-3) / 1e9
    return dict(workload="verify: 256 seq x 32 blocks x k=8 = 65,536 rows, V=151,936 bf16, rho~U(0.2,0.99) "
                         "per block, drafts z~softmax(s), eps 0.2, accepted lengths and corrections",
                value=nb / (ms * 1e-3), unit="blocks/s", ms_per_step=ms, steps=steps,
                mean_accepted_length=float(al.mean()), positions_evaluated=evaluated,
                roofline=dict(bound="hbm", achieved=achieved, peak=HBM_PEAK_GBS, unit="GB/s",
                              frac=achieved / HBM_PEAK_GBS, traffic=measured_traffic_bytes("verify"),
                              valu_issue=valu_issue("verify", ms)))


def stream_suite(saki, workloads, dev, s_buf, t_buf, grad_buf, warmup):
    """The long-rollout stress workload: 262,144 rows of V = 151,936 bf16 in 64
    chunks of 4,096 (row_offset = 4,096 x chunk, grad_scale = 1 / 262,144),
    eps 0.02, coupling + routed loss + fp32 gradient; each chunk generated into
    the first 4,096 rows of the buffers before its call; only the calls are
    timed (HIP events), and summed."""
    import torch
    cfg = workloads.CONFIGS["stream"]
    V, chunk, n_total = cfg["V"], cfg["chunk"], cfg["rows"]
    s, t, grad = s_buf[:chunk], t_buf[:chunk], grad_buf[:chunk]
    eps, seed = 0.02, workloads.coupling_seed("stream")
    out = saki.alloc_couple_out(chunk, dev)
    route = dict(valid_mask=None, grad_scale=1.0 / n_total,
                 row_loss=torch.empty(chunk, dtype=torch.float32, device=dev),
                 loss_sum=torch.empty(1, dtype=torch.float64, device=dev), grad=grad)
    ws = torch.empty(max(saki.workspace_bytes(saki.SAKI_OP_COUPLE, chunk, V), 8), dtype=torch.uint8, device=dev)
    total_ms, corr, tv = 0.0, 0.0, 0.0
    for c in range(n_total // chunk):
        lo = c * chunk
        workloads.fill("stream", s, t, lo=lo)
        torch.cuda.synchronize()
        call = lambda: saki.saki_couple(s, t, eps, seed, lo, out, route, ws)  # noqa: E731
        ms, _, _ = time_calls(call, 1, warmup if c == 0 else 0)
        total_ms += ms
        corr += float(out["corrected"].float().sum())
        tv += float(out["tv"].double().sum())
    achieved = n_total * (2 * V * 2 + V * 4) / (total_ms * 1e-3) / 1e9
    return dict(workload="stream: 32 seq x 8192 pos = 262,144 rows in 64 chunks of 4,096, V=151,936 bf16, "
                         "peaked rows, eps 0.02, coupling + routed loss + fp32 grad",
                value=n_total / (total_ms * 1e-3), unit="positions/s", ms_per_step=total_ms,
                chunks=n_total // chunk,
                roofline=dict(bound="hbm", achieved=achieved, peak=HBM_PEAK_GBS, unit="GB/s",
                              frac=achieved / HBM_PEAK_GBS,
                              traffic=stream_traffic_bytes(n_total // chunk, n_total)),
                stats=dict(correction_rate=corr / n_total, mean_tv=tv / n_total))


def _oracle_blocks(args):
    """CPU oracle on blocks, in order, until `budget` seconds of work (a worker process)."""
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    from oracle import verify
    s, t, draft, k, eps, seed, offsets, budget = args
    t0 = time.perf_counter()
    done = 0
    for i in range(len(offsets)):
        sl = slice(i * k, (i + 1) * k)
        verify.verify_blocks(s[sl], t[sl], k, draft[sl], eps, seed, int(offsets[i]))
        done += 1
        if time.perf_counter() - t0 >= budget:
            break
    return done, time.perf_counter() - t0


def bench_verify(args, saki, workloads, dev):
    """Speculative verification (Sec. 3.5): 256 sequences x 32 blocks of k = 8
    draft positions, V = 151,936 bf16, eps 0.2; accepted-prefix length and the
    correction of every block."""
    import numpy as np
    import torch
    cfg = workloads.CONFIGS["verify"]
    k, V = cfg["k"], cfg["V"]
    n = args.rows or cfg["rows"]
    n -= n % k
    nb = n // k
    seed = workloads.coupling_seed("verify")
    print(f"# generating {n} x {V} bf16 rows and student drafts", file=sys.stderr, flush=True)
    s = torch.empty(n, V, dtype=torch.bfloat16, device=dev)
    t = torch.empty_like(s)
    workloads.fill("verify", s, t)
    draft = workloads.drafts(s)
    acc = torch.empty(nb, dtype=torch.int32, device=dev)
    corr = torch.empty(nb, dtype=torch.int32, device=dev)
    ws = torch.empty(max(saki.workspace_bytes(saki.SAKI_OP_VERIFY, n, V), 8), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    if args.calibrate_copy:
        calibration_copy(dev)

    def step():
        saki.saki_spec_verify(s, t, k, draft, args.eps, seed, 0, -1, acc, corr, None, ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev[0].record(stream)
    for i in range(args.steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    ms = sum(per) / len(per)
    al = acc.cpu().numpy()
    evaluated = int(np.minimum(al + 1, k).sum())  # positions each block reads before it stops
    print(f"# per-step ms: {[round(x, 3) for x in per]}; mean accepted length {al.mean():.3f}; "
          f"positions evaluated {evaluated} of {n}", file=sys.stderr, flush=True)
    achieved = evaluated * 2 * V * 2 / (ms * 1e-3) / 1e9
    attainable = attainable_read_gbs(dev)
    cpu = None
    if not args.no_cpu_baseline:
        n_sample = 32
        blocks = np.linspace(0, nb - 1, n_sample).astype(np.int64)
        idx = torch.as_tensor(np.concatenate([np.arange(b * k, (b + 1) * k) for b in blocks]), device=dev)
        S = s[idx].float().cpu().numpy().astype(np.float64)
        T = t[idx].float().cpu().numpy().astype(np.float64)
        D = draft[idx].cpu().numpy()
        workers = cpu_workers()
        budget = 20.0
        parts = [np.arange(w, n_sample, workers) for w in range(workers)]
        jobs = [(np.concatenate([S[b * k:(b + 1) * k] for b in p]), np.concatenate([T[b * k:(b + 1) * k] for b in p]),
                 np.concatenate([D[b * k:(b + 1) * k] for b in p]), k, args.eps, seed, blocks[p] * k,
                 budget / workers)
                for p in parts if len(p)]
        with single_threaded_pool(len(jobs)) as pool:
            pool.map(_noop, range(len(jobs)))
            t0 = time.perf_counter()
            res = pool.map(_oracle_blocks, jobs)
            wall = time.perf_counter() - t0
        done = sum(r[0] for r in res)
        cpu = dict(value=done / wall, unit="blocks/s", cores=len(jobs), kind="oracle",
                   sample=f"{done} blocks of the same workload (from {n_sample} evenly spaced), {len(jobs)} "
                          f"single-threaded worker processes each stopping after {budget / len(jobs):.2f} s; "
                          f"{sum(r[1] for r in res):.1f} s of CPU work in {wall:.1f} s wall")
    line = {
        "metric": "speculative-verify blocks/sec (k=8, V=151,936 bf16)",
        "value": nb / (ms * 1e-3),
        "unit": "blocks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"logits": "bf16", "arithmetic": "f32, row sums and the lambda solve in f64", "workload": "verify: 256 seq x 32 blocks x k=8 = 65,536 rows, V=151,936 bf16, "
                               "rho~U(0.2,0.99) per block, drafts z~softmax(s)",
                   "blocks": nb, "k": k, "vocab": V, "eps": args.eps,
                   "mean_accepted_length": float(al.mean()), "positions_evaluated": evaluated},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "attainable_read": attainable,
                     "frac_attainable": achieved / attainable,
                     "traffic": measured_traffic_bytes("verify") if n == cfg["rows"] and args.eps == 0.2 else None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def bench_route(args, saki, workloads, dev):
    """saki_route_loss on its own: the routed loss (Eq. general_objective) and its
    f32 gradient over the large workload's 65,536 rows (V = 151,936 bf16), with
    the coupling outputs of one saki_couple call (made before timing) as input."""
    import torch
    cfg = workloads.CONFIGS["large"]
    n = args.rows or cfg["rows"]
    V = cfg["V"]
    seed = workloads.coupling_seed("large")
    print(f"# generating {n} x {V} bf16 rows and their coupling", file=sys.stderr, flush=True)
    s = torch.empty(n, V, dtype=torch.bfloat16, device=dev)
    t = torch.empty_like(s)
    workloads.fill("large", s, t)
    out = saki.alloc_couple_out(n, dev)
    ws_c = torch.empty(max(saki.workspace_bytes(saki.SAKI_OP_COUPLE, n, V), 8), dtype=torch.uint8, device=dev)
    saki.saki_couple(s, t, args.eps, seed, 0, out, None, ws_c)
    torch.cuda.synchronize()
    del t, ws_c
    torch.cuda.empty_cache()
    adv = (out["logt_token"] - out["logp_token"]).contiguous()
    grad = torch.empty(n, V, dtype=torch.float32, device=dev)
    row_loss = torch.empty(n, dtype=torch.float32, device=dev)
    loss_sum = torch.empty(1, dtype=torch.float64, device=dev)
    ws = torch.empty(max(saki.workspace_bytes(saki.SAKI_OP_ROUTE, n, V), 8), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    if args.calibrate_copy:
        calibration_copy(dev)

    def step():
        saki.saki_route_loss(s, out["token"], out["corrected"], out["teacher_argmax"], adv,
                             grad_scale=1.0 / n, row_loss=row_loss, loss_sum=loss_sum, grad=grad,
                             workspace=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev[0].record(stream)
    for i in range(args.steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    ms = sum(per) / len(per)
    print(f"# per-step ms: {[round(x, 3) for x in per]}", file=sys.stderr, flush=True)
    achieved = n * (2 * V + 4 * V) / (ms * 1e-3) / 1e9  # s read once (bf16), f32 gradient written once
    attainable = attainable_read_gbs(dev)
    line = {
        "metric": "routed-loss positions/sec at V=151,936 bf16 (saki_route_loss, f32 gradient)",
        "value": n / (ms * 1e-3),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"logits": "bf16", "arithmetic": "f32, row sums in f64", "workload": "route: the large workload's 65,536 coupled rows, V=151,936 bf16, "
                               "routed loss + loss sum + fp32 grad",
                   "rows": n, "vocab": V, "eps": args.eps, "grad_dtype": "f32",
                   "loss_sum": float(loss_sum.item())},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "attainable_read": attainable,
                     "frac_attainable": achieved / attainable,
                     "traffic": measured_traffic_bytes("route") if n == cfg["rows"] and args.eps == 0.2 else None},
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def bench_probe(args, saki, workloads, dev):
    """Probe metrics (C_1, C_16, KL(T || S), H(S) and the teacher's Top-16) on
    4,096 rows of the large workload (V = 151,936 bf16)."""
    import torch
    cfg = workloads.CONFIGS["large"]
    n = args.rows or 4096
    V, k = cfg["V"], 16
    s, t = workloads.rows("large", 0, n, device=dev)
    out = dict(c1=torch.empty(n, dtype=torch.float32, device=dev),
               ck=torch.empty(n, dtype=torch.float32, device=dev),
               kl_ts=torch.empty(n, dtype=torch.float32, device=dev),
               entropy=torch.empty(n, dtype=torch.float32, device=dev),
               topk=torch.empty(n, k, dtype=torch.int32, device=dev),
               row_status=torch.empty(n, dtype=torch.uint8, device=dev))
    torch.cuda.synchronize()
    if args.calibrate_copy:
        calibration_copy(dev)

    def step():
        saki.saki_probe_metrics(s, t, k, **out)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev[0].record(stream)
    for i in range(args.steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    ms = sum(per) / len(per)
    print(f"# per-step ms: {[round(x, 3) for x in per]}", file=sys.stderr, flush=True)
    achieved = n * (2 * V * 2) / (ms * 1e-3) / 1e9  # s and t read once (bf16)
    line = {
        "metric": "probe positions/sec at V=151,936 bf16 (C_1, C_16, KL(T||S), H(S), teacher Top-16)",
        "value": n / (ms * 1e-3),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"logits": "bf16", "arithmetic": "f32, row sums in f64",
                   "workload": "probe: 4,096 rows of the large workload, V=151,936 bf16, k=16",
                   "rows": n, "vocab": V, "k": k, "mean_c16": float(out["ck"].mean())},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic_bytes("probe") if n == 4096 else None},
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


ROLLOUT = dict(B=256, k=8, max_len=64, V=151936, eps=0.2, model_seed=4, seed=0x5A4B49 + 6)


def _oracle_rollout(job):
    import numpy as np
    from oracle import rollout as orollout
    from paper_2609_36601_amd import workloads
    B, k, L, V, eps, seed, model_seed = job
    t0 = time.process_time()
    o = orollout.rollout(workloads.SyntheticAR(V, seed=model_seed), np.arange(B), k, L, eps, seed)
    return time.process_time() - t0, int(o["length"].sum())


def bench_rollout(args, saki, workloads, dev):
    """Speculative rollout waves (App. I): 256 sequences x 64 tokens, k = 8 drafts
    per wave, V = 151,936 bf16, eps 0.2, on the synthetic prefix-hash model.  The
    timed figure is the library's work per rollout (draft sampling, verification,
    commit), from events around its calls; the synthetic model's logits (the
    stand-in for the networks) are reported apart."""
    import torch
    R = dict(ROLLOUT)
    B, k, L, V, eps = R["B"], R["k"], R["max_len"], R["V"], R["eps"]
    mt = workloads.SyntheticARTorch(V, seed=R["model_seed"], device=dev)
    prompts = torch.arange(B)

    def run(timing=None):
        return saki.rollout(mt, prompts, k, L, eps, R["seed"], dtype=torch.bfloat16,
                            check_every=4, timing=timing, metadata=args.metadata)

    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    lib_ms, wall_ms, tokens, waves_all, evaluated = [], [], 0, [], 0
    parts = {"sample": 0.0, "verify": 0.0, "commit": 0.0}
    for _ in range(args.steps):
        timing = {}
        t0 = time.perf_counter()
        tr, waves = run(timing)
        torch.cuda.synchronize()
        wall_ms.append((time.perf_counter() - t0) * 1e3)
        ms = 0.0
        for name in parts:
            x = sum(a.elapsed_time(b) for a, b in timing.get(name, []))
            parts[name] += x
            ms += x
        lib_ms.append(ms)
        tokens += int(tr["length"].sum().item())
        waves_all.append(waves)
        for a in timing["accepted_len"]:
            evaluated += int(torch.clamp(a.long() + 1, max=k).sum().item())
    n = args.steps
    ms = sum(lib_ms) / n
    tok = tokens / n
    # algorithmic bytes of the library per rollout: each draft step reads the B
    # student rows once (2 V bytes each), verification reads student and teacher
    # rows up to each block's first rejection
    waves_mean = sum(waves_all) / n
    bytes_per = waves_mean * k * B * V * 2 + (evaluated / n) * 2 * V * 2
    achieved = bytes_per / (ms * 1e-3) / 1e9
    print(f"# library ms per rollout {[round(x, 2) for x in lib_ms]}; wall ms {[round(x, 1) for x in wall_ms]}; "
          f"waves {waves_all}; parts (ms per rollout) "
          f"{ {k_: round(v / n, 3) for k_, v in parts.items()} }", file=sys.stderr, flush=True)
    cpu = None
    if not args.no_cpu_baseline:
        # the oracle on a bounded sample of the same workload: 2 sequences x 8 tokens
        job = (2, k, 8, V, eps, R["seed"], R["model_seed"])
        with single_threaded_pool(1) as pool:
            pool.map(_noop, range(1))
            t0 = time.perf_counter()
            busy, ntok = pool.map(_oracle_rollout, [job])[0]
            wall = time.perf_counter() - t0
        cpu = dict(value=ntok / wall, unit="committed tokens/s", cores=1, kind="oracle",
                   sample=f"oracle rollout of 2 sequences x 8 tokens, k={k}, same V, eps and model "
                          f"(one single-threaded process, {busy:.1f} s of CPU work)")
    line = {
        "metric": "speculative rollout committed tokens/sec (k=8, V=151,936 bf16; library steps)",
        "value": tok / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"logits": "bf16", "arithmetic": "f32, row sums and the lambda solve in f64", "workload": "rollout: 256 sequences x 64 tokens, k=8 drafts per wave, V=151,936 bf16, "
                               "eps 0.2, synthetic prefix-hash student/teacher",
                   "metadata": args.metadata,
                   "tokens_per_rollout": tok, "waves_per_rollout": waves_mean,
                   "positions_verified_per_rollout": evaluated / n,
                   "library_ms": {k_: v / n for k_, v in parts.items()},
                   "wall_ms_with_model": sum(wall_ms) / n},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def bench_stream(args, saki, workloads, dev):
    """Long-rollout stress workload: 32 sequences x 8,192 positions = 262,144 rows of
    V = 151,936 bf16 (peaked rows), eps 0.02, coupling + routed loss + fp32 gradient,
    streamed in 64 chunks of 4,096 rows with row_offset = 4,096 x chunk and
    grad_scale = 1 / 262,144.  Only the library calls are timed (one per chunk, HIP
    events), and summed; each chunk is generated before its call."""
    import torch
    cfg = workloads.CONFIGS["stream"]
    V, chunk = cfg["V"], cfg["chunk"]
    n_total = args.rows or cfg["rows"]
    n_chunks = (n_total + chunk - 1) // chunk
    eps = 0.02
    seed = workloads.coupling_seed("stream")
    s = torch.empty(chunk, V, dtype=torch.bfloat16, device=dev)
    t = torch.empty_like(s)
    grad = torch.empty(chunk, V, dtype=torch.float32, device=dev)
    out = saki.alloc_couple_out(chunk, dev)
    route = dict(valid_mask=None, grad_scale=1.0 / n_total,
                 row_loss=torch.empty(chunk, dtype=torch.float32, device=dev),
                 loss_sum=torch.empty(1, dtype=torch.float64, device=dev), grad=grad)
    ws = torch.empty(max(saki.workspace_bytes(saki.SAKI_OP_COUPLE, chunk, V), 8), dtype=torch.uint8,
                     device=dev)
    total_ms, rows, corr, tv = 0.0, 0, 0.0, 0.0
    if args.calibrate_copy:
        calibration_copy(dev)
    for c in range(n_chunks):
        lo = c * chunk
        n = min(chunk, n_total - lo)
        workloads.fill("stream", s[:n], t[:n], lo=lo)
        torch.cuda.synchronize()
        if c == 0:
            for _ in range(max(args.warmup, 1)):
                saki.saki_couple(s[:n], t[:n], eps, seed, lo, out, route, ws)
            torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        saki.saki_couple(s[:n], t[:n], eps, seed, lo, out, route, ws)
        e1.record()
        torch.cuda.synchronize()
        total_ms += e0.elapsed_time(e1)
        rows += n
        corr += float(out["corrected"][:n].float().sum())
        tv += float(out["tv"][:n].double().sum())
    print(f"# {n_chunks} chunks, {rows} rows, {total_ms:.2f} ms of library time; correction rate "
          f"{corr / rows:.4f}, mean TV {tv / rows:.4f}", file=sys.stderr, flush=True)
    achieved = rows * (2 * V * 2 + V * 4) / (total_ms * 1e-3) / 1e9
    attainable = attainable_read_gbs(dev)
    line = {
        "metric": "coupled+routed positions/sec, long-rollout stress (V=151,936 bf16, eps 0.02)",
        "value": rows / (total_ms * 1e-3),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": 1,
        "warmup": max(args.warmup, 1),
        "ms_per_step": total_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"logits": "bf16", "arithmetic": "f32, row sums and the lambda solve in f64", "workload": "stream: 32 seq x 8192 pos = 262,144 rows in 64 chunks of 4,096, "
                               "V=151,936 bf16, peaked rows, eps 0.02, coupling + routed loss + fp32 grad",
                   "rows": rows, "vocab": V, "eps": eps, "chunks": n_chunks},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "attainable_read": attainable,
                     "frac_attainable": achieved / attainable, "traffic": stream_traffic_bytes(n_chunks, rows)},
        "cpu_baseline": None,
        "stats": {"correction_rate": corr / rows, "mean_tv": tv / rows},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
