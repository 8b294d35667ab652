"""Host AddressSanitizer / UndefinedBehaviorSanitizer run over the CPU oracle
and the seeded input generator (tests/sanitize_driver.c)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def test_oracle_and_generator_under_asan_and_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "sanitize_driver")
    build = subprocess.run(
        [gcc, "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=off",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         os.path.join(HERE, "sanitize_driver.c"), "-lm", "-o", exe],
        capture_output=True, text=True)
    if build.returncode != 0 and "sanitize" in build.stderr and "cannot find" in build.stderr:
        pytest.skip("sanitizer runtime not installed")
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stderr[-4000:]
    assert "sanitized cases: 400" in run.stdout


def test_c_abi_host_code_under_asan_and_ubsan(tmp_path):
    """The library's host code (argument checks, plans, workspaces, status
    strings) under AddressSanitizer and UndefinedBehaviorSanitizer, driven by
    tests/api_sanitize_driver.cpp.  The sanitizers instrument host code only."""
    root = os.path.dirname(HERE)
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    csrc = os.path.join(root, "paper_2608_03447_amd", "csrc")
    exe = str(tmp_path / "api_sanitize_driver")
    build = subprocess.run(
        [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
         "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
         "-fno-gpu-sanitize", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(root, "include"), os.path.join(csrc, "asd_api.cpp"),
         os.path.join(csrc, "asd_kernels.hip"), os.path.join(HERE, "api_sanitize_driver.cpp"),
         "-o", exe],
        capture_output=True, text=True)
    assert build.returncode == 0, build.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1",
               HIP_VISIBLE_DEVICES="")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "0 failures" in run.stdout
    assert "runtime error" not in run.stderr
