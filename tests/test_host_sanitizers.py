"""The library's host code (frame construction, plan building, plan groups, the argument checks of
the C entry points) built with AddressSanitizer, LeakSanitizer and UndefinedBehaviorSanitizer and
run on the CPU against a stand-in for the HIP runtime (tests/sanitize/): status codes, and a
device allocation failing at every point of the creation sequence (FF_ENOMEM, NULL handles, no
leaks).  No GPU; g++ builds host code only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_26430_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "sanitize")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_driver")
    srcs = [os.path.join(CSRC, f) for f in ("capi.cpp", "framegen.cpp", "plan.cpp", "group.cpp")] + \
           [os.path.join(HERE, "hip_host_stub.cpp"), os.path.join(HERE, "driver.cpp")]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-D__HIP_PLATFORM_AMD__", "-D__align__(x)=__attribute__((aligned(x)))", "-DHIP_SYMBOL(x)=(&(x))",
           "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, *srcs, "-o", exe, "-lpthread"]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert build.returncode == 0, build.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    out = run.stdout + run.stderr
    assert "ERROR: AddressSanitizer" not in out and "ERROR: LeakSanitizer" not in out, out[-6000:]
    assert "runtime error" not in out, out[-6000:]
    assert run.returncode == 0, out[-6000:]
    assert "host driver: 0 failed checks" in out
    injected = int(out.split("allocation failures injected: ")[1].split()[0])
    assert injected >= 2 * 5, out[-2000:]    # at least frame and plan allocations of the 5 frames
