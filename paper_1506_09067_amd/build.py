"""Build libchaos.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libchaos.so")
SOURCES = ["worker.hip", "fused_large.hip", "fused_t1.hip", "fused_cpcp.hip", "batch_grad.hip",
           "chaos_api.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions stay disabled in every HIP build
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no implicit multiply-add contraction: every fused multiply-add in the
    # kernels is an explicit fmaf, so results do not depend on the compiler
    "-ffp-contract=off",
    "-Wall", "-Wno-unused-function",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = [ln for ln in r.stderr.splitlines() if ln.strip() and "packed-fp32-ops" not in ln]
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
    elif verbose and noise:
        sys.stderr.write("\n".join(noise) + "\n")
    return r.returncode


def build_library(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every HIP source into libchaos.so (always recompiles): one
    object per source, compiled concurrently, then one link."""
    tmpdir = tempfile.mkdtemp(prefix="chaos_build_")
    try:
        objs = [os.path.join(tmpdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
        cmds = [[HIPCC, *FLAGS, "-c", os.path.join(CSRC, s), "-o", o]
                for s, o in zip(SOURCES, objs)]
        jobs = jobs or min(len(cmds), max(1, min(os.cpu_count() or 1, 16)))
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            rcs = list(ex.map(lambda c: _run(c, verbose), cmds))
        for s, rc in zip(SOURCES, rcs):
            if rc != 0:
                raise RuntimeError("hipcc failed compiling %s" % s)
        tmp = LIB + ".tmp%d" % os.getpid()
        if _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose):
            raise RuntimeError("hipcc failed linking libchaos.so")
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
