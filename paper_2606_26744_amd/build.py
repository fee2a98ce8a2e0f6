"""Build libhdf.so (the HIP kernels and the C ABI) for gfx950, in-tree.

    python -m paper_2606_26744_amd.build

Compiles every csrc/*.hip to an object with hipcc (in parallel) and links the
shared library next to this file; also builds libhdf_probe.so from csrc/probe/ (a
memory-system probe that only bench.py loads, not part of the library).  Always
recompiles.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libhdf.so")
PROBE_OUT = os.path.join(HERE, "libhdf_probe.so")
ARCH = "gfx950"

# Packed-fp32 instructions are disabled for all device code (they are generated
# from plain float code otherwise); the host pass reports the feature as unknown,
# which is harmless.
CFLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-Wall",
          "-Wno-unused-function", "-Wno-unused-variable",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    for c in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, jobs: int | None = None) -> str:
    hipcc = _hipcc()
    bdir = os.path.join(HERE, "_build")
    os.makedirs(bdir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    if not srcs:
        raise RuntimeError("no HIP sources under " + CSRC)

    def compile_one(src):
        obj = os.path.join(bdir, os.path.basename(src)[:-4] + ".o")
        cmd = [hipcc, *CFLAGS, "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        errs = "\n".join(l for l in r.stderr.splitlines()
                         if "packed-fp32-ops" not in l)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{errs}")
        if verbose and errs.strip():
            print(errs, file=sys.stderr)
        return obj

    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 4)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(compile_one, srcs))
    tmp = OUT + ".tmp"
    cmd = [hipcc, "-shared", f"--offload-arch={ARCH}", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, OUT)
    probes = sorted(glob.glob(os.path.join(CSRC, "probe", "*.hip")))
    if probes:
        tmp = PROBE_OUT + ".tmp"
        cmd = [hipcc, "-shared", *CFLAGS, "-o", tmp, *probes]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("probe build failed:\n" + r.stderr)
        os.replace(tmp, PROBE_OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
