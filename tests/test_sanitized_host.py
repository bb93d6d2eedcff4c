"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The library's host layer (hils_api.cpp: argument checks, workspace sizing and
dispatch, linked with the regular kernel objects as libhils_san.so) and the
oracle (both precisions, built with clang) are compiled with ASan + UBSan; the
ABI tests and the oracle's pins then run in a child process that preloads
clang's ASan runtime and loads those builds (HILS_LIB, HILS_ORACLE_SANITIZED).
Any sanitizer report fails the child (halt_on_error) and this test.  No GPU
call is made: the ABI tests stop at the host checks."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RUNTIME = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
TESTS = ["tests/test_abi.py", "tests/test_oracle_pins.py", "tests/test_oracle_headnorm.py",
         "tests/test_oracle_decode.py", "tests/test_oracle_landmark.py"]


@pytest.mark.skipif(not RUNTIME, reason="clang's ASan runtime is not installed")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    import oracle
    from paper_2607_02980_amd import build

    oracle.build_sanitized()
    lib = build.build_sanitized()
    logs = tmp_path / "san"
    env = dict(os.environ,
               LD_PRELOAD=RUNTIME[-1],
               ASAN_OPTIONS=f"detect_leaks=0:halt_on_error=1:verify_asan_link_order=0:log_path={logs}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:log_path={logs}",
               HILS_LIB=lib, HILS_ORACLE_SANITIZED="1")
    r = subprocess.run([sys.executable, "-m", "pytest", *TESTS, "-q", "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    reports = "".join(open(f).read() for f in glob.glob(str(logs) + "*"))
    assert r.returncode == 0 and not reports, (r.stdout[-3000:] + r.stderr[-3000:] + reports[:6000])
    assert " passed" in r.stdout
