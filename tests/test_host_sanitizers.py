"""The host side of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only).

``python -m paper_2608_00938_amd.build_hostsan`` builds the library with its
argument validation, overlap checks and dispatch instrumented.  Every host ABI
test then runs in a child process against that build, with the ASan runtime
preloaded; any sanitizer report or failed test fails this test.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_LIB = os.path.join(ROOT, "paper_2608_00938_amd", "_build", "libgrace_hostsan.so")

RUN = """
import sys
sys.path.insert(0, {root!r})
from paper_2608_00938_amd import grace as G
G._LIB_PATH = {lib!r}
import pytest
sys.exit(pytest.main([{tests!r}, "-q", "-p", "no:cacheprovider", "-m", "not gpu"]))
"""


@pytest.mark.skipif(not os.path.exists(SAN_LIB), reason="host-sanitizer build not present")
def test_abi_host_checks_under_asan_and_ubsan():
    from paper_2608_00938_amd import build_hostsan
    env = dict(os.environ)
    env["LD_PRELOAD"] = build_hostsan.asan_runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["HIP_VISIBLE_DEVICES"] = ""   # host checks only: the child never touches a GPU
    code = RUN.format(root=ROOT, lib=SAN_LIB, tests=os.path.join(ROOT, "tests", "test_abi_host.py"))
    p = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600, cwd=ROOT)
    out = p.stdout + p.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert p.returncode == 0, out[-4000:]
    assert " passed" in p.stdout, out[-2000:]
