"""Host check of the kernels' fixed-divisor division (na::FastDiv, CPU only).

tests/fastdiv_check.cpp is compiled against the library's header with the host
C++ compiler and run: for every divisor below 2^20 the device's multiplier
(one double division) equals the host's (64-bit integers), and the quotients
of edge and pseudo-random dividends below 2^31 are exact, for those divisors
and for sampled divisors up to 2^31 - 1.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_fastdiv_is_exact(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "fastdiv_check")
    subprocess.check_call([cxx, "-O2", "-std=c++17", "-Wall", "-Werror",
                           "-I", os.path.join(ROOT, "paper_2403_04690_amd", "csrc"),
                           os.path.join(ROOT, "tests", "fastdiv_check.cpp"), "-o", exe])
    res = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    words = res.stdout.split()
    assert words[0] == "ok" and int(words[1]) > (1 << 20), res.stdout
