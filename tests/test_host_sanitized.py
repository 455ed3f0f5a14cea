"""The scheduler and the C ABI under AddressSanitizer and
UndefinedBehaviorSanitizer (no GPU): tests/host_harness/abi_harness.cpp,
built with g++ together with plan.cpp and abi.cpp, replaces the kernel
launchers and HIP runtime calls with stubs that check every address range a
kernel or copy would touch against the buffers passed, then drives every
entry point over the layer workloads, the streaming history lengths, several
attention block counts and 150 seeded random descriptors, plus the
invalid-descriptor and invalid-call paths."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_20940_amd", "csrc")


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("g++ and the HIP headers are needed to build the host harness")
    exe = str(tmp_path_factory.mktemp("harness") / "abi_harness")
    cmd = [gxx, "-std=c++17", "-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-include", "algorithm",
           os.path.join(ROOT, "tests", "host_harness", "abi_harness.cpp"),
           os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "abi.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    return subprocess.run([exe, *args], capture_output=True, text=True, env=env, timeout=300)


def test_entry_points_clean_under_sanitizers(harness):
    r = _run(harness)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " 0 failures" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr


def test_range_checks_report_a_planted_overrun(harness):
    """The stubs' range checks have teeth: a workspace shorter than the size
    passed is reported."""
    r = _run(harness, "plant")
    assert r.returncode != 0
    assert "overrun" in r.stderr
