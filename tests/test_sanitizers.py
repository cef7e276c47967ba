"""The host code of libstepq (layout derivation, launch planning and its
check, the CPU setup step) and the fp64 oracle, built with AddressSanitizer
and UndefinedBehaviorSanitizer and run on the CPU (tests/native/)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
CSRC = os.path.join(ROOT, "paper_2609_38169_amd", "csrc")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(cmd_build, exe, tmp_path):
    r = subprocess.run(cmd_build, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    # verify_asan_link_order=0: a library preloaded by the environment may
    # come before the sanitizer runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    return r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_checks")
    out = _run(["g++", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                os.path.join(NATIVE, "host_checks.cpp"), os.path.join(CSRC, "stepq_plan.cpp"),
                os.path.join(CSRC, "stepq_setup.cpp"), "-pthread", "-o", exe], exe, tmp_path)
    assert "host checks ok" in out


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_checks")
    out = _run(["gcc", "-std=c11", *SAN, "-ffp-contract=off", os.path.join(NATIVE, "oracle_checks.c"),
                os.path.join(ROOT, "oracle", "stepq_oracle.c"), "-lm", "-o", exe], exe, tmp_path)
    assert "oracle checks ok" in out
