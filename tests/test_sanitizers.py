"""AddressSanitizer and UndefinedBehaviorSanitizer over the host-side code, on the CPU: the
library's argument checks and lane/chunk planner (csrc/lif_host.h, compiled by g++ as
host code only) and the CPU oracle (oracle/lif_oracle.c), driven by
tests/sanitize/host_harness.cpp.  No GPU code is built here."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None, reason="needs gcc and g++")
def test_host_code_under_sanitizers(tmp_path):
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    obj = tmp_path / "lif_oracle.o"
    exe = tmp_path / "host_harness"
    subprocess.run(["gcc", "-std=c11", "-ffp-contract=off", *SAN, "-I", os.path.join(ROOT, "oracle"), "-c",
                    os.path.join(ROOT, "oracle", "lif_oracle.c"), "-o", str(obj)], check=True)
    subprocess.run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(rocm, "include"),
                    "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "oracle"),
                    "-I", os.path.join(ROOT, "paper_2408_00280_amd", "csrc"),
                    os.path.join(ROOT, "tests", "sanitize", "host_harness.cpp"), str(obj), "-lm",
                    "-o", str(exe)], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([str(exe)], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
