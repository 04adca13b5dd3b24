"""The library's host code (argument validation, size arithmetic, workspace
layout, the launch sequence up to the first HIP call) built with
AddressSanitizer and UndefinedBehaviorSanitizer and run without a GPU.  The
device code is compiled as usual but never runs: every call in
tests/host_checks.cpp either fails validation or fails its first launch.
The sanitizers apply to host code only (each flag behind -Xarch_host)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_12370_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
HOST_SANITIZERS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                   "-Xarch_host", "-fno-sanitize-recover=undefined"]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc is needed to build the library")
def test_host_code_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    common = ["-O1", "-g", "-std=c++17", *HOST_SANITIZERS, "-I" + INCLUDE]
    steps = [
        [HIPCC, "--offload-arch=gfx950", *common, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + CSRC, "-c", os.path.join(CSRC, "specverify.hip"), "-o", str(tmp_path / "sv.o")],
        [HIPCC, "-x", "c++", *common, "-c", os.path.join(ROOT, "tests", "host_checks.cpp"), "-o",
         str(tmp_path / "checks.o")],
        [HIPCC, "--offload-arch=gfx950", *HOST_SANITIZERS, str(tmp_path / "sv.o"), str(tmp_path / "checks.o"), "-o",
         str(tmp_path / "checks")],
    ]
    for cmd in steps:
        r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([str(tmp_path / "checks")], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "0 failures" in r.stdout
