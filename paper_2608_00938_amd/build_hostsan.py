"""Host-sanitizer build of the C ABI (CPU only).

Compiles ``grace_api.hip`` -- the host-side argument validation, overlap checks
and dispatch -- with AddressSanitizer and UndefinedBehaviorSanitizer on its host
code only (the device code of that file is built as usual), and links it with
the kernels of the normal build into ``_build/libgrace_hostsan.so``.  The host
ABI tests then run against it with the ASan runtime preloaded
(``tests/test_host_sanitizers.py``).  Run ``python -m
paper_2608_00938_amd.build`` first: the kernel objects come from there.
"""
from __future__ import annotations

import os
import subprocess
import sys

from . import build as B

LIB = os.path.join(B.OBJ, "libgrace_hostsan.so")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]


def asan_runtime() -> str:
    """Path of the ASan runtime that the sanitized library needs preloaded."""
    clang = os.path.join(os.path.dirname(B.HIPCC), "..", "lib", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    return subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                          capture_output=True, text=True, check=True).stdout.strip()


def build(verbose: bool = False) -> str:
    objs = [os.path.join(B.OBJ, s.replace(".hip", ".o")) for s in B.SOURCES if s != "grace_api.hip"]
    missing = [o for o in objs if not os.path.exists(o)]
    if missing:
        raise RuntimeError(f"build the library first (missing {missing[0]})")
    api = os.path.join(B.OBJ, "grace_api_hostsan.o")
    logs = [B._run([B.HIPCC, *B.CFLAGS, "-O1", *SAN, "-c", os.path.join(B.CSRC, "grace_api.hip"),
                    "-o", api])]
    tmp = LIB + ".tmp"
    logs.append(B._run([B.HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *SAN, "-o", tmp,
                        api, *objs]))
    os.replace(tmp, LIB)
    if verbose:
        for lg in logs:
            if lg.strip():
                print(lg, file=sys.stderr)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
