"""The library's host code under AddressSanitizer (no GPU needed).

The C ABI validates every argument on the host before any HIP call. This
builds the library with AddressSanitizer on its host code only (the device
code is compiled as usual, unsanitised) together with
tests/host_asan_driver.c, which
walks every size query and argument rejection over valid and invalid
configurations, and runs it: any out-of-bounds access or leak in those paths
aborts with a sanitizer report, and every expected status must come back.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_paths_under_asan(tmp_path):
    src = os.path.join(ROOT, "paper_2608_10392_amd", "csrc", "unif_moe.hip")
    drv = os.path.join(ROOT, "tests", "host_asan_driver.c")
    inc = os.path.join(ROOT, "include")
    lib_o = tmp_path / "unif_moe_host.o"
    drv_o = tmp_path / "driver.o"
    exe = tmp_path / "host_asan"
    asan = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-std=c++17", "-O1", "-g", *asan, "-Xclang", "-target-feature",
                    "-Xclang", "-packed-fp32-ops", "-c", src, "-o", str(lib_o)], check=True, capture_output=True)
    gcc = shutil.which("gcc")
    subprocess.run([gcc, "-O1", "-g", "-fsanitize=address", "-I", inc, "-c", drv, "-o", str(drv_o)], check=True,
                   capture_output=True)
    subprocess.run([HIPCC, *asan, str(drv_o), str(lib_o), "-o", str(exe)], check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=23")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "host paths ok" in r.stdout, r.stdout
