"""The library's host logic (api.cpp: argument checks, page bookkeeping, pass
planning, the failure path of build and append) under AddressSanitizer and
UndefinedBehaviorSanitizer, on a machine without a GPU: api.cpp is linked with
host-only stand-ins for the kernel launchers (tests/host_harness) into a
driver executable that exercises the C ABI."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HARNESS = os.path.join(ROOT, "tests", "host_harness")


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU is present: the driver's fake device pointers "
                                                       "would reach real copies")
def test_host_logic_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_driver")
    cmd = ["/opt/rocm/bin/hipcc", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-I" + os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2607_28940_amd", "csrc", "api.cpp"),
           os.path.join(ROOT, "paper_2607_28940_amd", "csrc", "xplan.cpp"),
           os.path.join(HARNESS, "stub_kernels.cpp"), os.path.join(HARNESS, "driver.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "all checks passed" in r.stdout
