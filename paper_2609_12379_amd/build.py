"""Compile the HIP library for gfx950 in-tree (paper_2609_12379_amd/libfm.so).

The step kernel is instantiated once per batch specialisation (1, 2, 4, 8) in separate
translation units, compiled in parallel, then linked with the C-ABI and scheduler objects.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libfm.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # atomics stay as written: the optimizer would turn the one-lane chunk claims into
    # wave-wide ones that wait for their result at once
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    "-I", os.path.join(ROOT, "include"),
]
BATCHES = (1, 2, 4, 8)


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed: " + " ".join(cmd) + "\n" + res.stderr[-4000:])
    return res.stderr


def build(verbose: bool = False, jobs: int = 0, batches=None) -> str:
    """Build libfm.so. ``batches`` (or FM_BUILD_BATCHES="1,4") limits the batch
    specialisations compiled, for development only; the default builds all of them."""
    if batches is None:
        env = os.environ.get("FM_BUILD_BATCHES", "")
        batches = tuple(int(x) for x in env.split(",") if x) or BATCHES
    out = tempfile.mkdtemp(prefix="fm_build_")
    try:
        units = [([os.path.join(CSRC, "fm_kernels.hip"), f"-DFM_B={b}"] + ([] if b in batches else ["-DFM_STUB"]),
                  os.path.join(out, f"k{b}.o")) for b in BATCHES]
        units.append(([os.path.join(CSRC, "fm_lib.hip")], os.path.join(out, "lib.o")))
        units.append(([os.path.join(CSRC, "fm_plan.cpp")], os.path.join(out, "plan.o")))
        jobs = jobs or min(len(units), max(1, os.cpu_count() or 1))
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            logs = list(ex.map(lambda u: _run([HIPCC] + FLAGS + ["-c"] + u[0] + ["-o", u[1]]), units))
        tmp = LIB + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + [u[1] for u in units] + ["-o", tmp])
        os.replace(tmp, LIB)
        if verbose:
            print("".join(l[-1500:] for l in logs))
    finally:
        shutil.rmtree(out, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build())
