"""Pins of the oracle's causal neighborhood attention (CPU only).

Causal masking per axis (Sec. 3.4 "Dilation and causal masking", caption of
Fig. "neighborhoodattention"): along a causal axis a query never attends to a
token of larger coordinate.  Pinned against what the definition fixes without
the oracle's own index code:
  * brute force: the k nearest same-group coordinates not after the query
    (pure Python, ranks 1-3, with dilation and windows longer than the
    available history);
  * a causal 1-D window as long as the axis is ordinary causal self
    attention: torch's fp64 scaled_dot_product_attention(is_causal=True);
  * 3-D with a causal first axis and full windows on the others is exact
    spatio-temporal attention with causal time (the example of Sec. 3.4):
    dense attention under the mask t_j <= t_i, written with numpy;
  * window 1 returns V; the first query of a causal axis sees only itself
    along it;
  * dilation is the union of independent undilated causal problems;
  * backward: fp64 finite differences, torch autograd of the masked dense
    attention, and the softmax gradient identities.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
from tests import na_bruteforce as bf


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _sets(idx):
    return [sorted(int(t) for t in row if t >= 0) for row in idx]


@pytest.mark.parametrize("L,k,d", [(9, 3, 1), (9, 4, 1), (10, 3, 2), (11, 5, 2), (12, 4, 3),
                                   (7, 7, 1), (20, 6, 3), (5, 1, 1), (16, 9, 1)])
def test_1d_causal_matches_bruteforce(L, k, d):
    got = _sets(oracle.neighbors((L,), (k,), (d,), causal=(1,)))
    assert got == bf.neighbours((L,), (k,), (d,), [True])
    # window length min(k, p + 1) with p the position in the group
    for x, row in enumerate(got):
        assert len(row) == min(k, x // d + 1)
        assert max(row) == x


@pytest.mark.parametrize("ext,ks,ds,cs", [
    ((6, 7), (3, 3), (1, 1), (1, 0)), ((8, 7), (4, 3), (2, 1), (0, 1)),
    ((5, 10), (3, 5), (1, 2), (1, 1)), ((4, 5, 6), (3, 3, 3), (1, 1, 2), (1, 0, 0)),
    ((5, 4, 6), (2, 3, 5), (2, 1, 1), (0, 1, 1)),
])
def test_multi_axis_causal_matches_bruteforce(ext, ks, ds, cs):
    got = _sets(oracle.neighbors(ext, ks, ds, causal=cs))
    assert got == bf.neighbours(ext, ks, ds, [bool(c) for c in cs])


def test_axis_relation_causal_closed_form():
    # inverse range of key j: queries j .. min(j + k - 1, n - 1) of its group
    for L, k, d in [(13, 4, 1), (17, 3, 2), (9, 9, 1), (20, 5, 3)]:
        first, lo, hi, cnt = oracle.axis_relation(L, k, d, causal=True)
        for j in range(L):
            g, p = j % d, j // d
            n = (L - g + d - 1) // d
            assert lo[j] == j and hi[j] == g + d * min(p + k - 1, n - 1)
            assert cnt[j] == min(p + k - 1, n - 1) - p + 1
            assert first[j] == g + d * max(0, p - k + 1)


def test_full_causal_window_is_causal_self_attention():
    B, H, L, D = 2, 3, 17, 8
    q, k, v = (_rand((B, H, L, D), s) for s in (1, 2, 3))
    scale = 0.29
    out, lse = oracle.forward(q, k, v, (L,), (1,), scale, causal=(1,))
    ref = torch.nn.functional.scaled_dot_product_attention(
        *(torch.from_numpy(a) for a in (q, k, v)), is_causal=True, scale=scale)
    np.testing.assert_allclose(out, ref.numpy(), atol=1e-12)
    s = scale * np.einsum("bhid,bhjd->bhij", q, k)
    s = np.where(np.tril(np.ones((L, L), dtype=bool)), s, -np.inf)
    m = s.max(-1)
    np.testing.assert_allclose(lse, m + np.log(np.exp(s - m[..., None]).sum(-1)), atol=1e-12)


def test_spatio_temporal_causal_time_is_masked_dense_attention():
    B, H, D = 1, 2, 4
    ext = (4, 3, 5)
    shape = (B, H) + ext + (D,)
    q, k, v = (_rand(shape, s) for s in (4, 5, 6))
    scale = 0.5
    # windows as long as every axis, causal along time (axis 0)
    out, lse = oracle.forward(q, k, v, ext, (1, 1, 1), scale, causal=(1, 0, 0))
    N = int(np.prod(ext))
    t = np.array([c[0] for c in itertools.product(*[range(e) for e in ext])])
    mask = t[None, :] <= t[:, None]
    qf, kf, vf = (a.reshape(B, H, N, D) for a in (q, k, v))
    s = np.where(mask, scale * np.einsum("bhid,bhjd->bhij", qf, kf), -np.inf)
    m = s.max(-1, keepdims=True)
    e = np.exp(s - m)
    np.testing.assert_allclose(out.reshape(B, H, N, D),
                               np.einsum("bhij,bhjd->bhid", e / e.sum(-1, keepdims=True), vf),
                               atol=1e-12)


def test_window_one_and_first_query():
    B, H, D = 1, 2, 5
    ext = (6, 7)
    shape = (B, H) + ext + (D,)
    q, k, v = (_rand(shape, s) for s in (7, 8, 9))
    out, lse = oracle.forward(q, k, v, (1, 1), (1, 1), 0.3, causal=(1, 1))
    np.testing.assert_allclose(out, v, atol=0)
    # k = 3 causal along axis 0: the first row's queries see only row 0
    out, _ = oracle.forward(q, k, v, (3, 1), (1, 1), 0.3, causal=(1, 0))
    np.testing.assert_allclose(out[:, :, 0], v[:, :, 0], atol=0)


def test_causal_dilation_is_union_of_undilated_problems():
    B, H, D = 1, 1, 3
    ext, ks, ds = (8, 9), (3, 2), (2, 3)
    shape = (B, H) + ext + (D,)
    q, k, v = (_rand(shape, s) for s in (10, 11, 12))
    out, lse = oracle.forward(q, k, v, ks, ds, 0.8, causal=(1, 1))
    for g0, g1 in itertools.product(range(ds[0]), range(ds[1])):
        sl = (slice(None), slice(None), slice(g0, None, ds[0]), slice(g1, None, ds[1]))
        o2, l2 = oracle.forward(q[sl], k[sl], v[sl], ks, (1, 1), 0.8, causal=(1, 1))
        assert np.array_equal(out[sl], o2) and np.array_equal(lse[sl[:4]], l2)


BWD = [((9,), (4,), (1,), (1,)), ((6, 7), (3, 3), (1, 2), (1, 0)),
       ((4, 3, 5), (3, 3, 3), (1, 1, 1), (1, 0, 1))]


@pytest.mark.parametrize("ext,ks,ds,cs", BWD)
def test_causal_finite_differences(ext, ks, ds, cs):
    B, H, D = 1, 1, 4
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (13, 14, 15, 16))
    dq, dk, dv = oracle.backward(q, k, v, g, ks, ds, 0.6, causal=cs)

    def loss(qq, kk, vv):
        return float((oracle.forward(qq, kk, vv, ks, ds, 0.6, causal=cs)[0] * g).sum())

    rng = np.random.default_rng(17)
    h = 1e-6
    for name, grad in (("q", dq), ("k", dk), ("v", dv)):
        for _ in range(6):
            pos = tuple(rng.integers(0, n) for n in shape)
            args = {"q": q.copy(), "k": k.copy(), "v": v.copy()}
            args[name][pos] += h
            fp = loss(args["q"], args["k"], args["v"])
            args[name][pos] -= 2 * h
            fd = (fp - loss(args["q"], args["k"], args["v"])) / (2 * h)
            assert abs(fd - grad[pos]) <= 1e-6 * max(1.0, abs(fd)), (name, pos, fd, grad[pos])


@pytest.mark.parametrize("ext,ks,ds,cs", BWD)
def test_causal_matches_torch_autograd_and_identities(ext, ks, ds, cs):
    B, H, D = 2, 1, 5
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (18, 19, 20, 21))
    dq, dk, dv = oracle.backward(q, k, v, g, ks, ds, 0.45, causal=cs)
    N = int(np.prod(ext))
    mask = torch.zeros(N, N, dtype=torch.bool)
    for t, row in enumerate(bf.neighbours(ext, ks, ds, [bool(c) for c in cs])):
        mask[t, row] = True
    tq, tk, tv = (torch.from_numpy(a.reshape(B, H, N, D)).requires_grad_(True) for a in (q, k, v))
    s = 0.45 * torch.matmul(tq, tk.transpose(-1, -2).contiguous())
    o = torch.matmul(torch.softmax(s.masked_fill(~mask, float("-inf")), -1), tv)
    o.backward(torch.from_numpy(g.reshape(B, H, N, D)))
    for mine, ref in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        np.testing.assert_allclose(mine.reshape(B, H, N, D), ref.numpy(), atol=1e-12)
    f = lambda a: a.reshape(B, H, N, D)
    np.testing.assert_allclose(f(dv).sum(2), f(g).sum(2), atol=1e-11)
    np.testing.assert_allclose(f(dk).sum(2), 0.0, atol=1e-11)


def test_causal_rows_match_full():
    B, H, D = 1, 2, 4
    ext, ks, ds, cs = (7, 9), (3, 4), (2, 1), (1, 1)
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (22, 23, 24, 25))
    out, lse = oracle.forward(q, k, v, ks, ds, 0.5, causal=cs)
    rows = np.array([0, 5, 40, 62, 100, 125])
    ro, rl = oracle.forward_rows(q, k, v, ks, ds, 0.5, rows, causal=cs)
    np.testing.assert_allclose(ro, out.reshape(-1, D)[rows], atol=1e-13)
    dq, dk, dv = oracle.backward(q, k, v, g, ks, ds, 0.5, causal=cs)
    rq, rk, rv = oracle.backward_rows(q, k, v, g, ks, ds, 0.5, rows, rows, causal=cs)
    np.testing.assert_allclose(rq, dq.reshape(-1, D)[rows], atol=1e-13)
    np.testing.assert_allclose(rk, dk.reshape(-1, D)[rows], atol=1e-13)
    np.testing.assert_allclose(rv, dv.reshape(-1, D)[rows], atol=1e-13)
