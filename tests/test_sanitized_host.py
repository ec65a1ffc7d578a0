"""CPU tier under sanitizers: the oracle and the library's host code (argument validation,
workspace queries, planning) built with AddressSanitizer and UndefinedBehaviorSanitizer, and
the CPU tests of the C ABI and of the oracle run against those builds in a child process."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None, reason="gcc/g++ not available")
def test_cpu_tier_under_asan_and_ubsan():
    sys.path.insert(0, ROOT)
    import oracle
    from paper_1810_09958_amd import build as B
    try:
        B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available for the device objects")
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not found")
    lib = B.build_sanitized()
    ref = oracle.build(force=True, sanitize=True)
    env = dict(os.environ, ISAM_LIB=lib, ISAM_REF_LIB=ref, LD_PRELOAD=f"{asan} {ubsan}",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    tests = ["tests/test_abi.py", "tests/test_oracle_gemm.py", "tests/test_oracle_dwsep.py",
             "tests/test_oracle_gru.py", "tests/test_oracle_conv1d.py", "tests/test_synth.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider", *tests],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error:" not in tail, tail
