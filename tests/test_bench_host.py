"""Host-side behaviour of bench.py that needs no GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, env=None):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=120, env=env)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    env = dict(os.environ, WORLD_SIZE="4")
    r = _run(env=env)
    assert r.returncode == 2


def test_help_lists_the_workloads():
    r = _run("--help")
    assert r.returncode == 0
    for w in ("couple", "verify", "stream", "rollout"):
        assert w in r.stdout


def test_traffic_table_is_keyed_by_source_hash():
    sys.path.insert(0, ROOT)
    import bench
    # algorithmic bytes per launch: couple 79.7 GB, route 59.7 GB, probe 2.49 GB
    floor = {"couple": 79e9, "route": 59e9, "probe": 2.4e9}
    for w in ("couple", "route", "probe"):
        h = bench.kernel_source_hash(w)
        assert len(h) == 64
        t = bench.measured_traffic_bytes(w)
        # either the counters were taken for exactly these sources, or traffic is unknown
        assert (t is None) == (h not in bench.MEASURED_TRAFFIC[w])
        if t is not None:
            assert floor[w] < t < 5 * floor[w]


def test_valu_issue_is_keyed_by_source_hash():
    sys.path.insert(0, ROOT)
    import bench
    for w in ("couple", "verify"):
        v = bench.valu_issue(w, 20.0)
        assert (v is None) == (bench.kernel_source_hash(w) not in bench.MEASURED_VALU[w])
        if v is not None:
            # at most one wave64 VALU instruction per CU and cycle
            assert 0.0 < v["frac"] and v["peak"] == 256 * 2.4e9
            assert v["achieved"] == v["instructions"] / 20e-3
