"""Builds libim2win.so (the C-ABI library and its gfx950 kernels) in-tree.

Every HIP source is compiled for gfx950 only, with packed fp32 VALU
instructions disabled (``-packed-fp32-ops``): the fp32 path uses plain
v_fma_f32 / v_fmac_f32.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libim2win.so")
SOURCES = ["api.cpp", "plan.cpp", "chunked.cpp", "transform.hip", "conv_fp32.hip", "conv_fp16.hip", "conv_fp16_col.hip", "conv_fp32_dma.hip", "conv_fp16_seg.hip", "conv_fp32_mfma.hip", "conv_fp16_stem.hip", "conv_fp32_stem.hip", "conv_fp32_cols.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "-x", "hip", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"),
]


def _run(cmd):
    p = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the gfx950 feature name: drop that warning
    noise = [l for l in (p.stdout + p.stderr).splitlines()
             if l.strip() and "packed-fp32-ops" not in l]
    return p.returncode, noise


def build(verbose: bool = False) -> str:
    """Compiles every source to an object (in parallel), then links them."""
    from concurrent.futures import ThreadPoolExecutor
    objdir = os.path.join(ROOT, "_build", "obj")
    os.makedirs(objdir, exist_ok=True)
    compile_flags = [f for f in FLAGS if f != "-shared"]
    jobs = []
    for s in SOURCES:
        obj = os.path.join(objdir, os.path.splitext(s)[0] + ".o")
        jobs.append((obj, [HIPCC] + compile_flags + ["-c", os.path.join(CSRC, s), "-o", obj]))
    workers = max(1, min(len(jobs), os.cpu_count() or 1, 16))
    with ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(lambda j: _run(j[1]), jobs))
    failed = False
    for (obj, cmd), (rc, noise) in zip(jobs, results):
        if verbose:
            print(" ".join(cmd), flush=True)
        if noise and (verbose or rc != 0):
            sys.stderr.write("\n".join(noise) + "\n")
        failed |= rc != 0
    if failed:
        raise RuntimeError("hipcc failed building libim2win.so")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + [j[0] for j in jobs] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    rc, noise = _run(cmd)
    if rc != 0:
        sys.stderr.write("\n".join(noise) + "\n")
        raise RuntimeError("linking libim2win.so failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
