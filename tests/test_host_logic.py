"""Host-side logic under sanitizers, on the CPU (no GPU needed):

  * the kernel-dispatch predicates (wq_limits.h) at the 32-bit buffer-offset
    boundaries, in a small C++ program built with g++ and ASan/UBSan;
  * the whole C-ABI validation suite (tests/test_abi.py) against a build of
    the library whose host code carries AddressSanitizer: argument checks,
    span bookkeeping and the error paths run instrumented.
"""

import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2412_15803_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_dispatch_predicates_at_offset_limits(tmp_path):
    exe = str(tmp_path / "limits_test")
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-I", CSRC, os.path.join(HERE, "host", "limits_test.cpp"),
                    "-o", exe], check=True, capture_output=True, text=True)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip() == "ok"


@pytest.mark.skipif(not os.path.exists("/opt/rocm/bin/hipcc"), reason="hipcc not available")
def test_abi_suite_under_host_address_sanitizer(tmp_path):
    sys.path.insert(0, os.path.join(HERE, "host"))
    import asan_build

    lib = asan_build.build_asan(str(tmp_path / "asan"))
    nm = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_report" in nm, "the library's host code is not instrumented"
    env = dict(os.environ, LD_PRELOAD=asan_build.asan_runtime(), WQ_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1")
    out = subprocess.run([sys.executable, "-m", "pytest", os.path.join(HERE, "test_abi.py"), "-q", "-x",
                          "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=600)
    text = out.stdout + out.stderr
    assert "AddressSanitizer" not in text, text[-4000:]
    assert out.returncode == 0, text[-4000:]
    assert " passed" in out.stdout
