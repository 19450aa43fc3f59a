"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

* The library's host planner (argument validation, the splice plan, the
  attention work list, the XCD weighting, the SA_DEBUG slot checks) is plain
  C++ in paper_2607_00151_amd/csrc/plan.h; tests/host/plan_check.cpp builds it
  on its own with both sanitizers and checks the plans' invariants over
  thousands of seeded shapes.
* The oracle's C source is built with both sanitizers and the oracle's pin
  suite runs against that build in a child process that preloads the ASan
  runtime.
Any sanitizer report aborts the child, which fails the test.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gcc_lib(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.timeout(300)
def test_planner_under_asan_ubsan(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "plan_check")
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-Wall", "-Werror",
                           "-I", os.path.join(ROOT, "include"),
                           "-I", os.path.join(ROOT, "paper_2607_00151_amd", "csrc"),
                           os.path.join(ROOT, "tests", "host", "plan_check.cpp"), "-o", exe])
    r = subprocess.run([exe], capture_output=True, text=True, timeout=240)
    print(r.stdout[-2000:], r.stderr[-4000:])
    assert r.returncode == 0 and "ALL OK" in r.stdout


@pytest.mark.timeout(600)
def test_oracle_pins_under_asan_ubsan():
    asan = _gcc_lib("libasan.so")
    if asan is None:
        pytest.skip("gcc's ASan runtime not available")
    import oracle
    oracle.build(force=True, sanitize=True)
    env = dict(os.environ, LD_PRELOAD=asan, ORACLE_SANITIZED="1",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=540)
    print(r.stdout[-3000:], r.stderr[-3000:])
    assert r.returncode == 0, "oracle pins failed under the sanitizers"
    assert "passed" in r.stdout
