"""Host check of the kernels' window functions (na_index.h, CPU only).

tests/index_dump.cpp is compiled against the library's header with the host
C++ compiler; for every axis of length 1..40, window k and dilation d with
k * d <= L, causal or not, the window start and end of each query, the start
the kernels' mask test uses and the inverse range of each key are compared
with the oracle's brute-force neighbour lists and axis relation.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _problems():
    for L in range(1, 41):
        for d in range(1, 5):
            for k in range(1, L // d + 1):
                for c in (0, 1):
                    yield L, k, d, c


def test_window_functions_match_the_oracle(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "index_dump")
    subprocess.check_call([cxx, "-O2", "-std=c++17", "-Wall", "-Werror",
                           "-I", os.path.join(ROOT, "paper_2403_04690_amd", "csrc"),
                           os.path.join(ROOT, "tests", "index_dump.cpp"), "-o", exe])
    probs = list(_problems())
    text = "".join(f"{L} {k} {d} {c}\n" for L, k, d, c in probs)
    res = subprocess.run([exe], input=text, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stderr
    rows = np.array(res.stdout.split(), dtype=np.int64).reshape(-1, 5)
    at = 0
    for L, k, d, c in probs:
        got = rows[at:at + L]
        at += L
        first, inv_lo, inv_hi, inv_cnt = oracle.axis_relation(L, k, d, causal=bool(c))
        nb = oracle.neighbors((L,), (k,), (d,), causal=(bool(c),))
        what = (L, k, d, c)
        np.testing.assert_array_equal(got[:, 0], first, err_msg=str(what))
        last = np.where(nb >= 0, nb, -1).max(axis=1)
        np.testing.assert_array_equal(got[:, 1], last, err_msg=str(what))
        np.testing.assert_array_equal(got[:, 3], inv_lo, err_msg=str(what))
        np.testing.assert_array_equal(got[:, 4], inv_hi, err_msg=str(what))
        # the inverse range holds exactly inv_count queries of the key's group
        np.testing.assert_array_equal((got[:, 4] - got[:, 3]) // d + 1, inv_cnt, err_msg=str(what))
        # the mask test (unsigned)(j - s) < k over the query's group admits
        # exactly its neighbours (s may lie before the axis on a causal one)
        for x in range(L):
            g = x % d
            js = np.arange(g, L, d)
            s = got[x, 2]
            admitted = js[((js - s) // d >= 0) & ((js - s) // d < k)]
            want = np.sort(nb[x][nb[x] >= 0])
            np.testing.assert_array_equal(admitted, want, err_msg=f"{what} x={x}")
    assert at == len(rows)
