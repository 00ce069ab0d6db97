"""Builds the HIP library libroutepack.so for gfx950 with hipcc (in-tree),
and the measurement aid libroutepack_probe.so (the LDS read-bandwidth probe,
not part of the method) from rp_probe.hip.

Each source compiles to its own object in parallel (no device code crosses a
translation unit), then one hipcc line links each shared library."""
from __future__ import annotations

import glob
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libroutepack.so")
PROBE_LIB = os.path.join(HERE, "libroutepack_probe.so")
PROBE_SOURCE = "rp_probe.hip"
OBJ_DIR = os.path.join(ROOT, "_build", "obj")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no fused multiply-add: accept tests and resampling weights are fixed
    # sequences of IEEE binary64 operations
    "-ffp-contract=off",
    # no packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]

# Flags for single sources on top of HIPCC_FLAGS.  The chain kernels run one
# wave per SIMD, a latency-bound chain of dependent moves: the scheduler
# strategy that groups memory instructions into clauses issues the row loads
# and LDS reads of a stage together (1% shorter annealing launch at mid than
# the default occupancy-driven strategy; it reorders the same instructions).
FILE_FLAGS = {
    "rp_anneal_chain.hip": ["-mllvm", "-amdgpu-sched-strategy=max-memory-clause"],
}


def flags_for(src: str) -> list:
    """The hipcc flags one source compiles with."""
    return HIPCC_FLAGS + FILE_FLAGS.get(os.path.basename(src), [])


def sources():
    """The library's sources (every .hip file but the probe's)."""
    return sorted(f for f in glob.glob(os.path.join(HERE, "csrc", "*.hip")) if os.path.basename(f) != PROBE_SOURCE)


def _jobs() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n, int(os.environ.get("MAX_JOBS", "16"))))


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link one shared library (always rebuilds)."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJ_DIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
    tag = os.getpid()

    def compile_one(src):
        obj = os.path.join(OBJ_DIR, os.path.basename(src)[:-4] + f".{tag}.o")
        cmd = [hipcc, *flags_for(src), *inc, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        return obj

    with ThreadPoolExecutor(_jobs()) as ex:
        objs = list(ex.map(compile_one, sources() + [os.path.join(HERE, "csrc", PROBE_SOURCE)]))
    probe_obj = objs.pop()
    try:
        for target, parts in ((LIB, objs), (PROBE_LIB, [probe_obj])):
            tmp = target + f".tmp{tag}"
            cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *parts, "-o", tmp]
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.check_call(cmd)
            os.replace(tmp, target)
    finally:
        for o in objs + [probe_obj]:
            try:
                os.remove(o)
            except OSError:
                pass
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
