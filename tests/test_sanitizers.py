"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

  * the oracle's C code: a driver calls every oracle function on random
    inputs;
  * the library's host-only code (host.cpp: job build, claim decisions,
    validation, commitment rule, retrieve planner; controller.cpp: the
    controller simulation and TTR estimators), built with plain g++ and the
    sanitizers into a shared library of its own, which the host-call tests
    then use in place of libtempokv.so (event-by-event controller parity,
    job build, routed job build, claim decisions, validation, TTR, planner);
  * the index's host table (index_table.cpp) under a randomised check
    against std::unordered_map that also replays its change lists onto a
    mirror, as the device upload does.
GPU code is not built here: only host code is instrumented."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_35065_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = tmp_path / "selftest"
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", *SAN, "-o", str(exe),
                           os.path.join(ROOT, "oracle", "selftest.c"),
                           os.path.join(ROOT, "oracle", "tempokv_oracle.c"), "-lm"])
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120,
                       env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"})
    assert r.returncode == 0, r.stdout + r.stderr
    assert "oracle selftest ok" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ missing")
def test_index_table_under_asan_ubsan(tmp_path):
    exe = tmp_path / "index_table_check"
    subprocess.check_call(["g++", "-O1", "-g", "-std=c++17", *SAN, "-I", INCLUDE, "-I", CSRC, "-o", str(exe),
                           os.path.join(ROOT, "tests", "native", "index_table_check.cpp"),
                           os.path.join(CSRC, "index_table.cpp")])
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300,
                       env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"})
    assert r.returncode == 0, r.stdout + r.stderr
    assert "index table check ok" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ missing")
def test_library_host_calls_under_asan_ubsan(tmp_path):
    so = tmp_path / "libtempokv_host_san.so"
    # -ffp-contract=off as in the library build: the controller's event times must match the oracle's exactly
    subprocess.check_call(["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off", *SAN,
                           "-I", INCLUDE, "-I", CSRC, "-o", str(so),
                           os.path.join(CSRC, "host.cpp"), os.path.join(CSRC, "controller.cpp")])
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    assert os.path.isabs(asan), "libasan.so not found"
    env = {**os.environ, "LD_PRELOAD": asan, "HYPOTHESIS_PROFILE": "default",
           # Python itself is not built with the sanitizer: its own allocations are not reported as leaks
           "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1", "UBSAN_OPTIONS": "print_stacktrace=1"}
    tests = ["tests/test_claims.py", "tests/test_controller_parity.py",
             "tests/test_abi.py", "-k", "not exports and not copy_calls and not stage_calls and not pipeline_calls "
             "and not hash_and_lookup and not retrieve_as and not index and not device_validate and not probe"]
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "native", "host_calls_runner.py"), str(so),
                        *tests], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-4000:] + r.stderr[-4000:])
    assert " passed" in r.stdout and "error" not in r.stdout.splitlines()[-1]
