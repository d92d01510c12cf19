"""Compile the gfx950 HIP library ``libdlvm.so`` in-tree with hipcc.

Run ``python -m paper_1711_03016_amd.build``. Objects go to ``_build/`` at the
repository root and the shared library next to this file, where the binding
loads it from.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libdlvm.so")
SOURCES = ["gemm.hip", "gemm_nn.hip", "gemm_nt.hip", "gemm_tn.hip", "gemm_pair.hip",
           "elementwise.hip", "small_step.hip", "api.cpp"]

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
ARCH = "gfx950"
# Packed float32 instructions are disabled for all device code.
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
]


def _compile(src: str, obj: str) -> tuple[str, int, str]:
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    p = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(line for line in (p.stdout + p.stderr).splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in line)
    return src, p.returncode, out


def build(verbose: bool = False) -> str:
    """Compile every source and link ``libdlvm.so``; return its path."""
    objdir = os.path.join(ROOT, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        results = list(ex.map(_compile, SOURCES, objs))
    failed = [r for r in results if r[1] != 0]
    for src, rc, out in results:
        if out.strip() and (verbose or rc != 0):
            print(f"--- {src} ---\n{out}", file=sys.stderr)
    if failed:
        raise RuntimeError("hipcc failed for " + ", ".join(r[0] for r in failed))
    tmp = LIB + ".tmp"
    p = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs],
                       capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError("link failed:\n" + p.stdout + p.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
