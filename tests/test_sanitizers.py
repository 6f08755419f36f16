"""The host code of the C ABI (api.cpp, with host-only launcher stand-ins) and the oracle, built
with AddressSanitizer and UndefinedBehaviorSanitizer and driven over valid and invalid inputs
(no GPU: nothing is launched). Any out-of-bounds access, use of freed memory or undefined
behaviour aborts the driver."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SAN = os.path.join(HERE, "sanitize")
HIPCC = "/opt/rocm/bin/hipcc"
CSRC = os.path.join(os.path.dirname(HERE), "paper_2605_06554_amd", "csrc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
           OMP_NUM_THREADS="2")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_abi_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_driver")
    # sanitizers on the host side only: the device side of the HIP headers is not instrumented
    flags = ["-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all"]
    objs = []
    for src in (os.path.join(CSRC, "api.cpp"), os.path.join(SAN, "launch_stubs.cpp"), os.path.join(SAN, "abi_driver.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([HIPCC, *flags, "-c", src, "-o", obj])
        objs.append(obj)
    _run([HIPCC, "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
          "-o", exe, *objs])
    r = _run([exe], env=ENV)
    assert "all checks passed" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-o", exe, os.path.join(SAN, "oracle_driver.c"), "-lm"])
    r = _run([exe], env=ENV)
    assert r.stdout.count("checksum") == 10
