"""Builds libsaki.so (the gfx950 HIP library behind include/saki.h) in-tree."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libsaki.so")
SOURCES = [os.path.join(HERE, "csrc", "saki.hip")]
DEPS = SOURCES + [os.path.join(HERE, "csrc", f) for f in ("device_util.hpp", "row_engine.hpp", "probe.hpp", "rollout.hpp")] + [
    os.path.join(ROOT, "include", "saki.h")]

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
    # no packed FP32 instructions (v_pk_*_f32) in any kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no machine-level hoisting of loop invariants: in the persistent kernels it
    # lifts the double constants of the per-row serial math (log / exp
    # coefficients) out of the row loop, where they stay live across the
    # sweeps and are spilled to scratch, then reloaded at memory latency in the
    # serial steps of every row
    "-mllvm", "-disable-machine-licm",
]


def hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def build(verbose=False):
    """Compile libsaki.so for gfx950 (always recompiles)."""
    tmp = LIB + ".tmp"
    cmd = [hipcc()] + HIPCC_FLAGS + SOURCES + ["-o", tmp]
    res = subprocess.run(cmd, cwd=HERE, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libsaki.so")
    if verbose:
        out = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in l)
        if out.strip():
            print(out)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
