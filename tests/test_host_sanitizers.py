"""Host entry points under AddressSanitizer + UndefinedBehaviorSanitizer (CPU only).

Builds tests/host_fuzz.cpp with the library's host sources (planner and schedule emitter) using
g++ and runs it over random shard geometries and document mixes; a sanitizer finding aborts the
program and fails the test.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_30460_amd", "csrc")


@pytest.fixture(scope="module")
def fuzz_binary(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("host_fuzz") / "host_fuzz")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I/opt/rocm/include", os.path.join(ROOT, "tests", "host_fuzz.cpp"),
           os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "schedule.cpp"), "-o", out]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        if "asan" in proc.stderr.lower() or "ubsan" in proc.stderr.lower():
            pytest.skip("sanitizer runtime not available: " + proc.stderr[-300:])
        raise AssertionError("build failed:\n" + proc.stderr[-3000:])
    return out


@pytest.mark.parametrize("seed", [1, 2])
def test_host_entry_points_clean_under_sanitizers(fuzz_binary, seed):
    env = dict(os.environ, SEED=str(seed), ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    proc = subprocess.run([fuzz_binary, "800"], capture_output=True, text=True, env=env, timeout=300)
    assert proc.returncode == 0, proc.stdout[-2000:] + proc.stderr[-4000:]
    assert proc.stdout.startswith("ok "), proc.stdout
