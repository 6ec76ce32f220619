"""The library's host code (plans, reshard, cost evaluator, RolloutDP, prefix tree,
routing) built with AddressSanitizer and UndefinedBehaviorSanitizer and fuzzed by a
seeded C++ driver (tests/host_asan/driver.cpp).  Host code only: no device code is built
and the driver calls no entry point that launches work."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_03077_amd", "csrc")
HOST_SOURCES = ["api.cpp", "plan.cpp", "migrate.cpp", "cost_model.cpp", "scheduler.cpp"]


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the ROCm headers")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "host_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC]
    cmd += [os.path.join(CSRC, f) for f in HOST_SOURCES]
    cmd += [os.path.join(ROOT, "tests", "host_asan", f) for f in ("stubs.cpp", "driver.cpp")]
    cmd += ["-L/opt/rocm/lib", "-lamdhip64", "-pthread", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, LD_LIBRARY_PATH="/opt/rocm/lib:" + os.environ.get("LD_LIBRARY_PATH", ""),
               ASAN_OPTIONS="detect_leaks=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and "host fuzz ok" in r.stdout, (r.stdout + r.stderr)[-4000:]
