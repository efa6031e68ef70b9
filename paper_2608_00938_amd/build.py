"""Build libgrace.so in-tree with hipcc for gfx950.

Usage: ``python -m paper_2608_00938_amd.build`` (also called by the repo's
``__graft_entry__.build()``).  Every HIP source is compiled on each call, once
for libgrace.so and once with -DGRACE_DEBUG for libgrace_debug.so.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libgrace.so")
SOURCES = ["grace_api.hip", "cross_attn.hip", "self_attn.hip", "beam.hip", "graph.hip", "gtm.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    # Keep the compiler from forming packed-fp32 VALU instructions.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd):
    p = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(ln for ln in (p.stderr or "").splitlines() if noise not in ln)
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{err}")
    return err


DEBUG_LIB = os.path.join(PKG, "libgrace_debug.so")
DEBUG_OBJ = os.path.join(OBJ, "debug")


def build(verbose: bool = False) -> str:
    """Build libgrace.so and its debug twin libgrace_debug.so (-DGRACE_DEBUG:
    device-side index checks counted, see grace_debug_counts); returns the
    release library's path."""
    os.makedirs(DEBUG_OBJ, exist_ok=True)
    jobs = []
    for out_dir, extra in ((OBJ, []), (DEBUG_OBJ, ["-DGRACE_DEBUG"])):
        for src in SOURCES:
            jobs.append((src, os.path.join(out_dir, src.replace(".hip", ".o")), extra))

    def compile_one(job):
        src, obj, extra = job
        return _run([HIPCC, *CFLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj])

    with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as ex:
        logs = list(ex.map(compile_one, jobs))
    for lib, out_dir in ((LIB, OBJ), (DEBUG_LIB, DEBUG_OBJ)):
        objs = [os.path.join(out_dir, s.replace(".hip", ".o")) for s in SOURCES]
        tmp = lib + ".tmp"
        logs.append(_run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]))
        os.replace(tmp, lib)
    if verbose:
        for lg in logs:
            if lg.strip():
                print(lg, file=sys.stderr)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
