"""The host code (argument and state checks, page allocator, workspace
layout) under AddressSanitizer and UndefinedBehaviorSanitizer: the CPU ABI
tests run in a child process against a host-instrumented build of the
library, with the clang ASan runtime loaded first.  CPU only."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(shutil.which(os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")) is None,
                                reason="hipcc not available")


def test_abi_cpu_tests_pass_under_host_sanitizers():
    sys.path.insert(0, ROOT)
    from paper_2608_12385_amd import build as B
    lib = B.build(sanitize=True)
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms, "host code is not instrumented"
    rt = B.asan_runtime()
    assert rt and os.path.exists(rt), "clang ASan runtime not found"
    runner = ("import sys; sys.path.insert(0, %r)\n"
              "from paper_2608_12385_amd import binding\n"
              "binding.LIB_PATH = %r\n"
              "import pytest\n"
              "sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider', %r]))\n"
              % (ROOT, lib, os.path.join(ROOT, "tests", "test_abi_cpu.py")))
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-c", runner], capture_output=True, text=True, env=env, cwd=ROOT,
                       timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out, out[-2000:]
