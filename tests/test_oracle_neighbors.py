"""Pins of the oracle's neighbourhood rule (CPU only).

The oracle's window-start formula is checked against (a) hand-derived windows
from the paper's definition (tests/golden), (b) an independent brute-force
"k nearest same-group coordinates" search, (c) the closed-form special cases
k = 1 and k = extent, (d) flip and axis-permutation symmetry, and (e) the
sizes of inverse neighbourhoods (Sec. 3.1: the query->key relation is not
symmetric and a key can be attended by more than k queries).
"""
import os

import numpy as np
import pytest

import oracle
from tests import na_bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "windows_1d.txt")


def _sets(idx):
    return [sorted(int(t) for t in row) for row in idx]


def test_golden_hand_derived_windows():
    blocks = bf.read_golden_windows(GOLDEN)
    assert len(blocks) >= 6
    for (L, k, d), rows in blocks.items():
        got = _sets(oracle.neighbors([L], [k], [d]))
        assert len(rows) == L
        for x, want in rows.items():
            assert got[x] == want, (L, k, d, x)
        # the independent brute force agrees with the hand derivation too
        assert [bf.axis_neighbours(x, L, k, d) for x in range(L)] == [rows[x] for x in range(L)]


# every legal (L, k, d) of a small grid (k * d <= L)
LEGAL_1D = [(L, k, d) for L in (1, 2, 5, 7, 10, 13, 16) for d in (1, 2, 3) for k in (1, 2, 3, 4, 5)
            if k * d <= L]


@pytest.mark.parametrize("L,k,d", LEGAL_1D)
def test_1d_matches_bruteforce(L, k, d):
    assert _sets(oracle.neighbors([L], [k], [d])) == bf.neighbours([L], [k], [d])


def test_illegal_windows_are_refused():
    # k * d > L has no window of k same-group neighbours: the oracle refuses it
    for L, k, d in [(1, 2, 1), (5, 3, 2), (7, 4, 2), (10, 4, 3)]:
        with pytest.raises(Exception):
            oracle.neighbors([L], [k], [d])


@pytest.mark.parametrize("case", [
    ((5, 7), (3, 5), (1, 1)),
    ((9, 6), (3, 3), (2, 2)),
    ((10, 11), (5, 3), (2, 3)),
    ((8, 8), (8, 1), (1, 4)),
    ((7, 9), (4, 2), (1, 2)),
])
def test_2d_matches_bruteforce(case):
    ext, ks, ds = case
    assert _sets(oracle.neighbors(ext, ks, ds)) == bf.neighbours(ext, ks, ds)


@pytest.mark.parametrize("case", [
    ((4, 5, 6), (3, 3, 3), (1, 1, 2)),
    ((5, 6, 7), (3, 1, 5), (1, 3, 1)),
    ((6, 4, 9), (2, 3, 3), (3, 1, 3)),
])
def test_3d_matches_bruteforce(case):
    ext, ks, ds = case
    assert _sets(oracle.neighbors(ext, ks, ds)) == bf.neighbours(ext, ks, ds)


def test_window_size_is_exact_everywhere():
    # Every query keeps exactly prod k neighbours, all distinct (shifted, never truncated).
    for ext, ks, ds in [((13,), (5,), (2,)), ((9, 10), (3, 5), (3, 2)), ((5, 6, 7), (3, 3, 3), (1, 2, 2))]:
        idx = oracle.neighbors(ext, ks, ds)
        assert idx.shape == (int(np.prod(ext)), int(np.prod(ks)))
        for row in idx:
            assert len(set(row.tolist())) == idx.shape[1]


def test_k1_is_identity_and_full_window_is_everything():
    idx = oracle.neighbors([9, 4], [1, 1], [3, 2])
    assert (idx[:, 0] == np.arange(36)).all()
    idx = oracle.neighbors([6, 5], [6, 5], [1, 1])
    for row in idx:
        assert sorted(row.tolist()) == list(range(30))
    # k * d = L: every query sees its whole dilation group
    idx = oracle.neighbors([12], [4], [3])
    for x, row in enumerate(idx):
        assert sorted(row.tolist()) == [j for j in range(12) if j % 3 == x % 3]


@pytest.mark.parametrize("L,k,d", [(11, 3, 1), (17, 5, 2), (10, 3, 3), (23, 7, 3), (40, 7, 4)])
def test_flip_equivariance_odd_k(L, k, d):
    idx = _sets(oracle.neighbors([L], [k], [d]))
    for x in range(L):
        assert sorted(L - 1 - j for j in idx[L - 1 - x]) == idx[x]


def test_axis_permutation_equivariance():
    ext, ks, ds = (7, 10), (3, 5), (2, 1)
    a = _sets(oracle.neighbors(ext, ks, ds))
    b = _sets(oracle.neighbors(ext[::-1], ks[::-1], ds[::-1]))
    H, W = ext
    for y in range(H):
        for x in range(W):
            mapped = sorted((j % W) * H + (j // W) for j in a[y * W + x])
            assert mapped == b[x * H + y]


@pytest.mark.parametrize("L,k,d", [(23, 7, 1), (40, 7, 3), (19, 4, 2), (30, 1, 5), (12, 12, 1)])
def test_axis_relation_matches_transpose_of_lists(L, k, d):
    first, lo, hi, cnt = oracle.axis_relation(L, k, d)
    lists = bf.neighbours([L], [k], [d])
    for x in range(L):
        assert first[x] == min(lists[x])
    for j in range(L):
        qs = [x for x in range(L) if j in lists[x]]
        assert cnt[j] == len(qs)
        assert lo[j] == min(qs) and hi[j] == max(qs)


def test_inverse_neighbourhood_size_bounds():
    # For odd k and a group long enough (n >= 2k), inverse neighbourhoods
    # range from ceil(k/2) queries (at the border) to k + floor(k/2).
    for L, k, d in [(40, 7, 1), (80, 7, 2), (32768, 1023, 4)]:
        _, _, _, cnt = oracle.axis_relation(L, k, d)
        assert cnt.min() == (k + 1) // 2
        assert cnt.max() == k + k // 2
        assert cnt.sum() == L * k
