"""The oracle and the host side of the C ABI (configuration and argument
checks, status strings, profiling arrays, test hooks) run clean under
AddressSanitizer (with leak detection) and UndefinedBehaviorSanitizer.  CPU
only: the sanitizers instrument host code; the GPU kernels are linked
unchanged and never launched."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
# host-only sanitizer flags for hipcc: each one applies to the host pass only
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-std=c99", *SAN, "-o", exe, os.path.join(HERE, "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "rr_oracle.c"), "-lm"])
    r = _run([exe], env=ENV, timeout=300)
    assert "oracle driver ok" in r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC) or shutil.which("gcc") is None, reason="needs hipcc and gcc")
def test_host_abi_under_sanitizers(tmp_path):
    from paper_2609_07306_amd import build as hipbuild
    objdir = os.path.join(ROOT, "paper_2609_07306_amd", "_build")
    kernels = [os.path.join(objdir, os.path.splitext(s)[0] + ".o") for s in hipbuild.SOURCES if s != "rr_api.hip"]
    if not all(os.path.exists(o) for o in kernels):
        hipbuild.build()
    api = str(tmp_path / "rr_api_san.o")
    _run([HIPCC, f"--offload-arch={hipbuild.ARCH}", "-O1", "-g", "-std=c++17", "-fPIC",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *HOST_SAN,
          "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2609_07306_amd", "csrc"),
          "-c", os.path.join(ROOT, "paper_2609_07306_amd", "csrc", "rr_api.hip"), "-o", api])
    drv = str(tmp_path / "abi_driver.o")
    _run(["gcc", "-std=c99", *SAN, "-I", os.path.join(ROOT, "include"), "-c",
          os.path.join(HERE, "abi_driver.c"), "-o", drv])
    exe = str(tmp_path / "abi_san")
    _run([HIPCC, f"--offload-arch={hipbuild.ARCH}", *HOST_SAN[:4], "-o", exe, drv, api, *kernels])
    r = _run([exe], env=ENV, timeout=300)
    assert "abi driver ok" in r.stdout
