"""Pins of the oracle's forward pass (CPU only).

Closed forms and invariants that the definition fixes independently of the
oracle's own code:
  * window = extent, dilation 1: dense scaled dot-product attention (Eq. 1),
    written here directly with numpy;
  * window * dilation = extent: dense attention inside each dilation
    sub-lattice (Sec. 3.4);
  * window 1: the output is V at the query's own position (Sec. 1, Fig.
    "neighborhoodattention" caption) and LSE = scale q.k;
  * dilation = the union of independent non-dilated problems (Sec. 3.4);
  * Q = 0: uniform attention, LSE = log(prod k) and O = mean of V over the
    brute-force neighbour set;
  * general NA = dense attention under the brute-force neighbour mask, with
    torch's own softmax in fp64.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle
from tests import na_bruteforce as bf


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _dense(q, k, v, scale):
    """Eq. 1 over all tokens of each (b, h): q,k,v [B,H,N,D]."""
    s = scale * np.einsum("bhid,bhjd->bhij", q, k)
    m = s.max(-1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(-1, keepdims=True)
    return np.einsum("bhij,bhjd->bhid", e / z, v), (m + np.log(z))[..., 0]


@pytest.mark.parametrize("ext", [(9,), (5, 7), (3, 4, 5)])
def test_full_window_is_dense_attention(ext):
    B, H, D = 2, 3, 8
    shape = (B, H) + ext + (D,)
    q, k, v = _rand(shape, 1), _rand(shape, 2), _rand(shape, 3)
    scale = 0.37
    out, lse = oracle.forward(q, k, v, ext, [1] * len(ext), scale)
    N = int(np.prod(ext))
    ro, rl = _dense(q.reshape(B, H, N, D), k.reshape(B, H, N, D), v.reshape(B, H, N, D), scale)
    np.testing.assert_allclose(out.reshape(B, H, N, D), ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse.reshape(B, H, N), rl, rtol=0, atol=1e-12)


def test_window_times_dilation_equals_extent_is_dense_per_sublattice():
    B, H, D = 1, 2, 4
    ext, ks, ds = (6, 9), (3, 3), (2, 3)
    shape = (B, H) + ext + (D,)
    q, k, v = _rand(shape, 4), _rand(shape, 5), _rand(shape, 6)
    out, lse = oracle.forward(q, k, v, ks, ds, 0.5)
    for g0, g1 in itertools.product(range(ds[0]), range(ds[1])):
        sl = (slice(None), slice(None), slice(g0, None, ds[0]), slice(g1, None, ds[1]))
        qs, kk, vs = q[sl], k[sl], v[sl]
        n = qs.shape[2] * qs.shape[3]
        ro, rl = _dense(qs.reshape(B, H, n, D), kk.reshape(B, H, n, D), vs.reshape(B, H, n, D), 0.5)
        np.testing.assert_allclose(out[sl].reshape(B, H, n, D), ro, atol=1e-12)
        np.testing.assert_allclose(lse[sl[:4]].reshape(B, H, n), rl, atol=1e-12)


@pytest.mark.parametrize("ext,ds", [((11,), (3,)), ((6, 5), (2, 1)), ((4, 3, 5), (1, 3, 2))])
def test_window_one_returns_v(ext, ds):
    B, H, D = 2, 2, 6
    shape = (B, H) + ext + (D,)
    q, k, v = _rand(shape, 7), _rand(shape, 8), _rand(shape, 9)
    out, lse = oracle.forward(q, k, v, [1] * len(ext), ds, 0.25)
    np.testing.assert_array_equal(out, v)
    np.testing.assert_allclose(lse, 0.25 * (q * k).sum(-1), atol=1e-13)


@pytest.mark.parametrize("ext,ks,ds", [((14,), (3,), (3,)), ((9, 8), (3, 3), (2, 2)),
                                       ((6, 7, 5), (3, 3, 3), (2, 1, 1))])
def test_dilation_is_union_of_undilated_problems(ext, ks, ds):
    B, H, D = 1, 2, 5
    shape = (B, H) + ext + (D,)
    q, k, v = _rand(shape, 10), _rand(shape, 11), _rand(shape, 12)
    out, lse = oracle.forward(q, k, v, ks, ds, 0.3)
    for g in itertools.product(*[range(d) for d in ds]):
        sl = (slice(None), slice(None)) + tuple(slice(gi, None, di) for gi, di in zip(g, ds))
        so, sls = oracle.forward(q[sl], k[sl], v[sl], ks, [1] * len(ks), 0.3)
        np.testing.assert_array_equal(out[sl], so)
        np.testing.assert_array_equal(lse[sl], sls)


@pytest.mark.parametrize("ext,ks,ds", [((13,), (5,), (2,)), ((7, 9), (3, 5), (2, 1)),
                                       ((5, 4, 6), (3, 3, 3), (1, 1, 2))])
def test_zero_query_is_uniform_average(ext, ks, ds):
    B, H, D = 1, 2, 3
    shape = (B, H) + ext + (D,)
    q = np.zeros(shape)
    k, v = _rand(shape, 13), _rand(shape, 14)
    out, lse = oracle.forward(q, k, v, ks, ds, 1.0)
    ell = int(np.prod(ks))
    np.testing.assert_allclose(lse, math.log(ell), atol=1e-13)
    lists = bf.neighbours(ext, ks, ds)
    N = int(np.prod(ext))
    vf = v.reshape(B, H, N, D)
    of = out.reshape(B, H, N, D)
    for t in range(N):
        np.testing.assert_allclose(of[:, :, t], vf[:, :, lists[t]].mean(axis=2), atol=1e-13)


@pytest.mark.parametrize("ext,ks,ds", [((15,), (4,), (3,)), ((7, 8), (3, 5), (2, 1)),
                                       ((4, 5, 6), (3, 3, 3), (1, 1, 2)), ((9, 7), (2, 3), (4, 2))])
def test_matches_masked_dense_attention_in_torch(ext, ks, ds):
    B, H, D = 2, 2, 6
    shape = (B, H) + ext + (D,)
    q, k, v = _rand(shape, 15), _rand(shape, 16), _rand(shape, 17)
    scale = 0.41
    out, lse = oracle.forward(q, k, v, ks, ds, scale)
    N = int(np.prod(ext))
    mask = torch.zeros(N, N, dtype=torch.bool)
    for t, row in enumerate(bf.neighbours(ext, ks, ds)):
        mask[t, row] = True
    tq, tk, tv = (torch.from_numpy(a.reshape(B, H, N, D)) for a in (q, k, v))
    s = scale * torch.matmul(tq, tk.transpose(-1, -2).contiguous())
    s = s.masked_fill(~mask, float("-inf"))
    ref = torch.matmul(torch.softmax(s, dim=-1), tv)
    np.testing.assert_allclose(out.reshape(B, H, N, D), ref.numpy(), atol=1e-12)
    np.testing.assert_allclose(lse.reshape(B, H, N), torch.logsumexp(s, -1).numpy(), atol=1e-12)


def test_probabilities_sum_to_one_and_output_in_hull():
    B, H, D = 1, 2, 4
    ext, ks, ds = (10, 9), (5, 3), (2, 3)
    shape = (B, H) + ext + (D,)
    q, k = _rand(shape, 18), _rand(shape, 19)
    ones = np.ones(shape)
    out, _ = oracle.forward(q, k, ones, ks, ds, 1.0)
    np.testing.assert_allclose(out, 1.0, atol=1e-14)
    v = _rand(shape, 20)
    out, _ = oracle.forward(q, k, v, ks, ds, 1.0)
    N = int(np.prod(ext))
    lists = bf.neighbours(ext, ks, ds)
    vf, of = v.reshape(B, H, N, D), out.reshape(B, H, N, D)
    for t in range(N):
        nb = vf[:, :, lists[t]]
        assert (of[:, :, t] <= nb.max(axis=2) + 1e-12).all()
        assert (of[:, :, t] >= nb.min(axis=2) - 1e-12).all()


def test_forward_rows_matches_full_forward():
    B, H, D = 2, 3, 8
    ext, ks, ds = (12, 10), (5, 3), (2, 3)
    shape = (B, H) + ext + (D,)
    q, k, v = _rand(shape, 21), _rand(shape, 22), _rand(shape, 23)
    out, lse = oracle.forward(q, k, v, ks, ds, 0.3)
    rows = np.array([0, 5, 119, 120, 300, 719])
    ro, rl = oracle.forward_rows(q, k, v, ks, ds, 0.3, rows)
    np.testing.assert_array_equal(ro, out.reshape(-1, D)[rows])
    np.testing.assert_array_equal(rl, lse.reshape(-1)[rows])


def test_rejects_illegal_problems():
    x = np.zeros((1, 1, 5, 2))
    with pytest.raises(ValueError):
        oracle.forward(x, x, x, [3], [2], 1.0)  # 3 * 2 > 5
    with pytest.raises(ValueError):
        oracle.forward(x, x, x, [0], [1], 1.0)
    with pytest.raises(ValueError):
        oracle.forward(x, x, x, [1], [0], 1.0)


def test_thread_count_does_not_change_results():
    """Each thread owns whole (b, h) slices, so one thread gives the same bits."""
    B, H, D = 3, 2, 8
    ext, ks, ds = (11, 9), (5, 3), (2, 1)
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (31, 32, 33, 34))
    n0 = oracle.num_threads()
    out, lse = oracle.forward(q, k, v, ks, ds, 0.4)
    grads = oracle.backward(q, k, v, g, ks, ds, 0.4)
    try:
        oracle.set_num_threads(1)
        assert oracle.num_threads() == 1
        out1, lse1 = oracle.forward(q, k, v, ks, ds, 0.4)
        grads1 = oracle.backward(q, k, v, g, ks, ds, 0.4)
    finally:
        oracle.set_num_threads(n0)
    assert oracle.num_threads() == n0
    np.testing.assert_array_equal(out1, out)
    np.testing.assert_array_equal(lse1, lse)
    for a, b in zip(grads1, grads):
        np.testing.assert_array_equal(a, b)
