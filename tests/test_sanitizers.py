"""AddressSanitizer + UndefinedBehaviorSanitizer builds of the CPU code, on
the CPU (no GPU).

* The oracle (oracle/chaos_oracle.c) with a driver that calls every exported
  function on the small and large nets, two tiny nets, the conv primitives
  and the error paths; leak detection on.
* The library's host side (paper_1506_09067_amd/csrc/chaos_api.hip, host
  part sanitized; its device part is only data) with a driver that walks
  every argument and shape error of the C ABI and a valid net up to the
  device query; the kernel launchers are stubs that fail, so nothing here
  runs on a GPU.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    return r.returncode, r.stdout + r.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_drv")
    rc, out = _run(["gcc", "-std=c11", "-g", "-O1", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "oracle", "chaos_oracle.c"),
                    os.path.join(SAN, "oracle_driver.c"), "-lm", "-o", exe])
    assert rc == 0, out
    rc, out = _run([exe], env=SAN_ENV, timeout=300)
    assert rc == 0 and "oracle driver ok" in out, out


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_host_api_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "host_drv")
    rc, out = _run([HIPCC, "-std=c++17", "-g", "-O1", "-fno-omit-frame-pointer",
                    "--offload-arch=gfx950",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "paper_1506_09067_amd", "csrc", "chaos_api.hip"),
                    os.path.join(SAN, "host_driver.cpp"), "-o", exe])
    assert rc == 0, out
    # no GPU is used: hide any from the driver so a valid net stops at the device query
    env = dict(SAN_ENV, HIP_VISIBLE_DEVICES="-1", ROCR_VISIBLE_DEVICES="-1")
    rc, out = _run([exe], env=env, timeout=300)
    assert rc == 0 and "host driver ok" in out, out
