"""Pins of the oracle's backward pass (CPU only).

  * fp64 central finite differences of the scalar loss <O, dO> with respect to
    q, k and v on tiny 1-D, 2-D and 3-D problems with dilation;
  * torch autograd (fp64) of dense attention under the brute-force neighbour
    mask;
  * exact identities of softmax attention: sum_j dV_j = sum_i dO_i,
    sum_j dK_j = 0, sum_i q_i.dQ_i = sum_j k_j.dK_j per (b, h);
  * the row-sampled backward equals the full one.
"""
import numpy as np
import pytest
import torch

import oracle
from tests import na_bruteforce as bf

CASES = [((9,), (3,), (2,)), ((5, 6), (3, 3), (1, 2)), ((4, 3, 5), (3, 3, 3), (1, 1, 1)),
         ((6, 7), (2, 3), (3, 2))]


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("ext,ks,ds", CASES)
def test_finite_differences(ext, ks, ds):
    B, H, D = 1, 2, 4
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (31, 32, 33, 34))
    scale = 0.6
    dq, dk, dv = oracle.backward(q, k, v, g, ks, ds, scale)

    def loss(qq, kk, vv):
        o, _ = oracle.forward(qq, kk, vv, ks, ds, scale)
        return float((o * g).sum())

    rng = np.random.default_rng(35)
    h = 1e-6
    for name, grad in (("q", dq), ("k", dk), ("v", dv)):
        for _ in range(6):
            pos = tuple(rng.integers(0, n) for n in shape)
            args = {"q": q.copy(), "k": k.copy(), "v": v.copy()}
            args[name][pos] += h
            fp = loss(args["q"], args["k"], args["v"])
            args[name][pos] -= 2 * h
            fm = loss(args["q"], args["k"], args["v"])
            fd = (fp - fm) / (2 * h)
            assert abs(fd - grad[pos]) <= 1e-6 * max(1.0, abs(fd)), (name, pos, fd, grad[pos])


@pytest.mark.parametrize("ext,ks,ds", CASES + [((8,), (8,), (1,))])
def test_matches_torch_autograd_of_masked_dense_attention(ext, ks, ds):
    B, H, D = 2, 2, 5
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (41, 42, 43, 44))
    scale = 0.45
    dq, dk, dv = oracle.backward(q, k, v, g, ks, ds, scale)
    N = int(np.prod(ext))
    mask = torch.zeros(N, N, dtype=torch.bool)
    for t, row in enumerate(bf.neighbours(ext, ks, ds)):
        mask[t, row] = True
    tq, tk, tv = (torch.from_numpy(a.reshape(B, H, N, D)).requires_grad_(True) for a in (q, k, v))
    s = scale * torch.matmul(tq, tk.transpose(-1, -2).contiguous())
    o = torch.matmul(torch.softmax(s.masked_fill(~mask, float("-inf")), -1), tv)
    o.backward(torch.from_numpy(g.reshape(B, H, N, D)))
    for mine, ref in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        np.testing.assert_allclose(mine.reshape(B, H, N, D), ref.numpy(), atol=1e-12)


@pytest.mark.parametrize("ext,ks,ds", CASES)
def test_gradient_identities(ext, ks, ds):
    B, H, D = 2, 2, 6
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (51, 52, 53, 54))
    dq, dk, dv = oracle.backward(q, k, v, g, ks, ds, 0.7)
    N = int(np.prod(ext))
    f = lambda a: a.reshape(B, H, N, D)
    np.testing.assert_allclose(f(dv).sum(2), f(g).sum(2), atol=1e-11)
    np.testing.assert_allclose(f(dk).sum(2), 0.0, atol=1e-11)
    np.testing.assert_allclose((f(q) * f(dq)).sum((2, 3)), (f(k) * f(dk)).sum((2, 3)), atol=1e-11)


def test_backward_rows_matches_full_backward():
    B, H, D = 2, 2, 4
    ext, ks, ds = (7, 9), (3, 5), (2, 1)
    shape = (B, H) + ext + (D,)
    q, k, v, g = (_rand(shape, s) for s in (61, 62, 63, 64))
    dq, dk, dv = oracle.backward(q, k, v, g, ks, ds, 0.5)
    qrows = np.array([0, 17, 62, 63, 200, 251])
    krows = np.array([1, 30, 64, 125, 190, 250])
    rq, rk, rv = oracle.backward_rows(q, k, v, g, ks, ds, 0.5, qrows, krows)
    np.testing.assert_allclose(rq, dq.reshape(-1, D)[qrows], atol=1e-13)
    np.testing.assert_allclose(rk, dk.reshape(-1, D)[krows], atol=1e-13)
    np.testing.assert_allclose(rv, dv.reshape(-1, D)[krows], atol=1e-13)


def test_window_one_gradients():
    # k = 1: O = V, so dV = dO and dQ = dK = 0.
    B, H, D = 1, 2, 3
    shape = (B, H, 10, D)
    q, k, v, g = (_rand(shape, s) for s in (71, 72, 73, 74))
    dq, dk, dv = oracle.backward(q, k, v, g, [1], [2], 1.0)
    np.testing.assert_array_equal(dv, g)
    np.testing.assert_allclose(dq, 0.0, atol=1e-15)
    np.testing.assert_allclose(dk, 0.0, atol=1e-15)
