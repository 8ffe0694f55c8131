"""The routing kernel's exact small-divisor arithmetic (the 64-bit remainder
by 16-bit digits, the Barrett constant floor((2^64 - 1) / m)) and its bit
select, compiled as host code from the kernels' own header and compared with
exact integer arithmetic.  CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_small_divisor_arithmetic_is_exact(tmp_path):
    exe = str(tmp_path / "arith")
    r = subprocess.run([HIPCC, "-O2", "-std=c++17", "-I", os.path.join(ROOT, "paper_2609_07306_amd", "csrc"),
                        "-o", exe, os.path.join(ROOT, "tests", "sanitize", "arith_driver.hip")],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0 and "arith driver ok" in out.stdout
    n = {"mod": 0, "div": 0, "sel": 0}
    for line in out.stdout.splitlines():
        f = line.split()
        if f[0] == "mod":
            x, m, got = int(f[1]), int(f[2]), int(f[3])
            assert got == x % m, line
        elif f[0] == "div":
            m, got = int(f[1]), int(f[2])
            assert got == (2 ** 64 - 1) // m, line
        elif f[0] == "sel":
            z, y, got = int(f[1]), int(f[2]), int(f[3])
            ones = [i for i in range(32) if (z >> i) & 1]
            assert got == ones[y], line
        else:
            continue
        n[f[0]] += 1
    assert n["mod"] > 20000 and n["div"] > 2000 and n["sel"] == 20000
