"""The library's host code under clang's undefined-behaviour checks.

A second copy of libcl.so is built with every UBSan check on the host side
made fatal, and the CPU tests that drive the C ABI (argument validation of
every entry point, workspace queries, the binding's checks, the rank
allocator and sensitivity scores) run against it in a child process.  A
report from the sanitizer (an overflowing size product, a misaligned or
out-of-range access, an invalid shift or enum value) ends that process with
a nonzero status and is printed here.
"""

import os
import subprocess
import sys

from paper_2605_05819_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ABI_TESTS = ["tests/test_abi.py", "tests/test_binding.py", "tests/test_ranks.py"]


def test_abi_tests_pass_on_the_ubsan_build(tmp_path):
    lib = build.build_ubsan(str(tmp_path / "ubsan"))
    env = dict(os.environ, CL_LIBRARY=lib,
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:report_error_type=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider"] + ABI_TESTS,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert "runtime error" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    # a child with this environment loads the sanitized copy, and with it the
    # UBSan runtime, not the in-tree library
    probe = ("from paper_2605_05819_amd import cl; cl.lib(); print(cl.LIB_PATH); "
             "maps = open('/proc/self/maps').read(); "
             "print('ubsan' if 'libclang_rt.ubsan_standalone' in maps else 'none')")
    check = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True,
                           timeout=300)
    assert check.stdout.split() == [lib, "ubsan"], check.stdout + check.stderr
