"""Pins of the oracle's backward operator from stored forward results (CPU only).

``oracle.backward_given`` takes the forward's output and logsumexp as the
library's backward does (P rebuilt from the logsumexp, Delta from the stored
output).  Pinned by:
  * with the exact forward results it is the plain backward (itself pinned by
    finite differences and autograd in test_oracle_backward.py);
  * it is affine in the stored output: adding E to `out` moves Delta_i by
    dO_i.E_i, which moves dQ_i by -scale (dO_i.E_i) sum_j P_ij k_j (the
    forward with V replaced by K) and dK_j by -scale sum_i P_ij (dO_i.E_i) q_i
    (the IN product that gives dV, with dO_i replaced by (dO_i.E_i) q_i), and
    leaves dV alone;
  * shifting the logsumexp by c scales every P, hence every gradient, by e^-c;
  * the sums of absolute terms bound the results and equal them when every
    term is non-negative.
"""
import numpy as np
import pytest

import oracle

CASES = [((9,), (3,), (2,), None), ((5, 6), (3, 3), (1, 2), None),
         ((4, 3, 5), (3, 3, 3), (1, 1, 1), None), ((6, 7), (2, 3), (3, 2), (True, False))]


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("ext,ks,ds,cs", CASES)
def test_exact_forward_results_give_the_plain_backward(ext, ks, ds, cs):
    shape = (2, 2) + ext + (5,)
    q, k, v, g = (_rand(shape, s) for s in (81, 82, 83, 84))
    out, lse = oracle.forward(q, k, v, ks, ds, 0.55, causal=cs)
    want = oracle.backward(q, k, v, g, ks, ds, 0.55, causal=cs)
    got = oracle.backward_given(q, k, v, out, lse, g, ks, ds, 0.55, causal=cs)
    for a, b in zip(got, want):
        np.testing.assert_allclose(a, b, atol=1e-12)


@pytest.mark.parametrize("ext,ks,ds,cs", CASES)
def test_affine_in_the_stored_output(ext, ks, ds, cs):
    shape = (1, 2) + ext + (4,)
    q, k, v, g, e = (_rand(shape, s) for s in (91, 92, 93, 94, 95))
    sc = 0.8
    out, lse = oracle.forward(q, k, v, ks, ds, sc, causal=cs)
    base = oracle.backward_given(q, k, v, out, lse, g, ks, ds, sc, causal=cs)
    moved = oracle.backward_given(q, k, v, out + e, lse, g, ks, ds, sc, causal=cs)
    w = (g * e).sum(-1, keepdims=True)               # change of Delta per query
    pk, _ = oracle.forward(q, k, k, ks, ds, sc, causal=cs)   # sum_j P_ij k_j
    _, _, in_wq = oracle.backward(q, k, v, w * q, ks, ds, sc, causal=cs)  # sum_i P_ij w_i q_i
    np.testing.assert_allclose(moved[0] - base[0], -sc * w * pk, atol=1e-12)
    np.testing.assert_allclose(moved[1] - base[1], -sc * in_wq, atol=1e-12)
    np.testing.assert_allclose(moved[2], base[2], atol=0)


def test_logsumexp_shift_scales_every_gradient():
    ext, ks, ds = (7, 8), (3, 5), (2, 1)
    shape = (1, 2) + ext + (4,)
    q, k, v, g, o = (_rand(shape, s) for s in (101, 102, 103, 104, 105))
    _, lse = oracle.forward(q, k, v, ks, ds, 0.6)
    a = oracle.backward_given(q, k, v, o, lse, g, ks, ds, 0.6)
    b = oracle.backward_given(q, k, v, o, lse + 1.5, g, ks, ds, 0.6)
    for x, y in zip(a, b):
        np.testing.assert_allclose(y, np.exp(-1.5) * x, atol=1e-12)


@pytest.mark.parametrize("ext,ks,ds,cs", CASES)
def test_absolute_sums_bound_and_meet_the_results(ext, ks, ds, cs):
    shape = (1, 2) + ext + (4,)
    q, k, v, g = (_rand(shape, s) for s in (111, 112, 113, 114))
    sc = 0.7
    out, lse = oracle.forward(q, k, v, ks, ds, sc, causal=cs)
    dq, dk, dv, aq, ak, av = oracle.backward_given(q, k, v, out, lse, g, ks, ds, sc, causal=cs,
                                                   abs_sums=True)
    for x, a in ((dq, aq), (dk, ak), (dv, av)):
        assert (a >= np.abs(x) - 1e-12).all()
    assert (aq > np.abs(dq) + 1e-9).any() and (ak > np.abs(dk) + 1e-9).any()
    # non-negative terms: out = 0 gives Delta = 0, and q, k, v, dO >= 0 make
    # every P, dP, dA and product non-negative, so each sum is its own bound
    q, k, v, g = np.abs(q), np.abs(k), np.abs(v), np.abs(g)
    _, lse = oracle.forward(q, k, v, ks, ds, sc, causal=cs)
    dq, dk, dv, aq, ak, av = oracle.backward_given(q, k, v, np.zeros_like(q), lse, g, ks, ds, sc,
                                                   causal=cs, abs_sums=True)
    for x, a in ((dq, aq), (dk, ak), (dv, av)):
        np.testing.assert_allclose(a, x, rtol=1e-13, atol=0)
