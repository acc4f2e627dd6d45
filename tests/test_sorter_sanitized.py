"""The host sorter of the chunk-sorted code form (csrc/sorted.hip) built with
AddressSanitizer and UndefinedBehaviorSanitizer on its host code and run by
tests/sorter_sanitize_driver.cpp, which checks the output against the codes
(see the driver).  CPU only: the driver launches no kernel."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def test_sorter_under_sanitizers(tmp_path):
    if not (os.path.exists(HIPCC) or shutil.which("hipcc")):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "sorter_asan")
    cmd = [HIPCC, "-std=c++17", "-O1", "-g", "--offload-arch=gfx950",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "paper_2401_06118_amd", "csrc"),
           os.path.join(ROOT, "tests", "sorter_sanitize_driver.cpp"),
           os.path.join(ROOT, "paper_2401_06118_amd", "csrc", "sorted.hip"), "-o", exe]
    b = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert b.returncode == 0, b.stdout + b.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "sorter sanitize ok" in r.stdout
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
