"""The C ABI's argument validation under the host sanitizers (CPU only).

The library sources and tests/abi_validation_host.hip are compiled with
AddressSanitizer and UndefinedBehaviorSanitizer on the host code (the device code
is built as usual, about 40 s), then the driver runs every validation branch of the entry points on a hand-built
context without a GPU, including sizes at the int32 limits.  Any out-of-bounds access,
signed overflow or other undefined behaviour aborts the driver.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_24391_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_abi_validation_under_host_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_validation")
    from paper_2604_24391_amd import build as fcbuild
    srcs = [os.path.join(CSRC, s) for s in fcbuild.SOURCES]
    srcs.append(os.path.join(ROOT, "tests", "abi_validation_host.hip"))
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-std=c++17", "-Xarch_host", "-g",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wno-unused-value", "-Wno-unused-result",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
           *srcs, "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    env = dict(os.environ)
    env.pop("FC_DEBUG", None)
    env["HIP_VISIBLE_DEVICES"] = ""          # never a device, even where one exists
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-6000:]
    assert "OK (0 failed expectations)" in run.stdout
    assert "runtime error" not in out and "AddressSanitizer" not in out
