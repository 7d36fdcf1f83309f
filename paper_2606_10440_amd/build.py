"""Build libsimgpu.so (host builder + HIP engines) for gfx950 with hipcc.

Each source is compiled to an object in parallel, then linked into the
shared library next to this file."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libsimgpu.so")
CSRC = os.path.join(HERE, "csrc")
SOURCES = ["api.cpp", "engine_launch.cpp", "engine_wg.hip", "engine_lane.hip", "engine_b1.hip",
           "engine_wave.hip", "engine_grid.hip", "engine_res.hip", "noalloc.hip"]
ARCH = os.environ.get("SIMGPU_ARCH", "gfx950")
OBJDIR = os.path.join(ROOT, "_build", "simgpu")

FLAGS = [
    "-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC",
    "-Wall", "-Wno-unused-result",
    # keep the compiler from forming packed fp32 ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature; that warning is noise
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if err.strip():
        print(err, file=sys.stderr, flush=True)
    if r.returncode:
        raise subprocess.CalledProcessError(r.returncode, cmd)


# per-source flags: the resident engine's same-address LDS atomics with
# lane-varying operands are combined per wave by a DPP scan instead of a
# scalar loop over the active lanes; the wave and lane engines, whose
# lone wavefronts wait on LDS each simulated cycle, are scheduled for
# instruction-level parallelism (measured: the wave engine 3-7 % and the
# lane engine about 3 % less time per launch; the resident and grid
# engines ran slower so)
EXTRA = {"engine_res.hip": ["-mllvm", "-amdgpu-atomic-optimizer-strategy=DPP"],
         "engine_wave.hip": ["-mllvm", "-amdgpu-sched-strategy=iterative-ilp"],
         "engine_lane.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"]}


def build(verbose: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = [s for s in SOURCES if os.path.exists(os.path.join(CSRC, s))]
    objs = [os.path.join(OBJDIR, s + ".o") for s in srcs]
    jobs = [[hipcc, *FLAGS, *EXTRA.get(s, []), "-c", "-o", o, os.path.join(CSRC, s)] for s, o in zip(srcs, objs)]
    with ThreadPoolExecutor(max_workers=min(len(jobs), 8)) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
