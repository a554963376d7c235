"""GPU parity of the fused NA kernels against the fp64 oracle (needs an MI355X).

All calls go through libna.so's C ABI (paper_2403_04690_amd binding).  The
bar: neighbour sets bit-exact; outputs, logsumexp and gradients within 2e-2
max-abs for fp16/bf16 and 1e-4 for fp32 of the oracle evaluated on the same
(already rounded) inputs.  Small problems are compared element by element
(they span several tiles and ragged tails); every full-size workload is
compared element by element too, forward and backward (fused and unfused).
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests import na_bruteforce as bf

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "fp16": 2e-2, "bf16": 2e-2}
TDT = workloads.TORCH_DTYPE


@pytest.fixture(scope="module")
def na():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2403_04690_amd as lib

    lib.load_library()
    return lib


@pytest.fixture
def force(monkeypatch, na):
    """Sets forcing variables (NA_WAVE_BLOCKS, NA_FWD_WAVES, NA_BWD_SPLIT) for one test.
    The library reads them when it makes a problem's plan, so plans are dropped
    (na.tune_clear) when they are set and again once they are restored."""
    def set_(**env):
        for name, value in env.items():
            monkeypatch.setenv(name, str(value))
        na.tune_clear()
    yield set_
    monkeypatch.undo()
    na.tune_clear()


def _inputs(shape, dtype, seed, n=4):
    gen = torch.Generator().manual_seed(seed)
    return [torch.randn(shape, generator=gen).to(TDT[dtype]) for _ in range(n)]


def _dev(*ts):
    return [t.cuda() for t in ts]


def _f64(t):
    return t.detach().cpu().double().numpy()


def _maxerr(gpu, ref):
    return float(np.max(np.abs(_f64(gpu) - ref))) if ref.size else 0.0


def _log(msg):
    print(msg, flush=True)


# ---------------------------------------------------------------- index math
@pytest.mark.parametrize("ext,ks,ds", [
    ((40,), (7,), (1,)), ((37,), (4,), (3,)), ((32768,), (1023,), (4,)),
    ((56, 56), (7, 7), (1, 1)), ((128, 128), (13, 13), (2, 2)), ((10, 9), (3, 2), (3, 4)),
    ((16, 64, 64), (7, 7, 7), (1, 2, 2)), ((5, 12, 7), (5, 1, 2), (1, 6, 3)),
])
def test_debug_windows_bit_exact(na, ext, ks, ds):
    start, ilo, ihi = (t.cpu().numpy() for t in na.debug_windows(ext, ks, ds))
    off = 0
    for a, L in enumerate(ext):
        first, lo, hi, _ = oracle.axis_relation(L, ks[a], ds[a])
        np.testing.assert_array_equal(start[off:off + L], first)
        np.testing.assert_array_equal(ilo[off:off + L], lo)
        np.testing.assert_array_equal(ihi[off:off + L], hi)
        off += L


@pytest.mark.parametrize("ext,ks,ds,dtype", [
    ((150,), (7,), (2,), "fp32"), ((21, 26), (5, 3), (2, 3), "fp16"),
    ((6, 9, 10), (3, 5, 3), (2, 1, 3), "bf16"), ((70,), (9,), (1,), "fp16"),
])
def test_neighbour_support_probe(na, ext, ks, ds, dtype):
    """Q = 0 makes P uniform on N(i); one-hot V rows then expose N(i) exactly."""
    D = 32
    N = int(np.prod(ext))
    lists = bf.neighbours(ext, ks, ds)
    ell = int(np.prod(ks))
    q = torch.zeros((1, 1) + ext + (D,), dtype=TDT[dtype])
    k = _inputs(q.shape, dtype, 5, 1)[0]
    for chunk in range((N + D - 1) // D):
        v = torch.zeros(1, 1, N, D)
        for c in range(D):
            t = chunk * D + c
            if t < N:
                v[0, 0, t, c] = 1.0
        v = v.reshape(q.shape).to(TDT[dtype])
        out, lse = na.forward(*_dev(q, k, v), ks, ds)
        o = out.float().cpu().reshape(N, D).numpy()
        for i in range(N):
            want = set(t - chunk * D for t in lists[i] if chunk * D <= t < (chunk + 1) * D)
            got = set(np.nonzero(o[i])[0].tolist())
            assert got == want, (i, chunk)
        np.testing.assert_allclose(lse.cpu().numpy(), math.log(ell), atol=1e-5)


# ---------------------------------------------------------------- forward
FWD_CASES = [
    # (extents, kernel, dilation, head_dim, dtype, batch, heads)
    ((200,), (7,), (1,), 32, "fp32", 1, 2),
    ((300,), (13,), (3,), 64, "fp16", 2, 2),
    ((129,), (1,), (2,), 128, "bf16", 1, 3),
    ((257,), (64,), (4,), 64, "fp16", 1, 2),
    ((1000,), (255,), (2,), 64, "bf16", 1, 2),
    ((70,), (70,), (1,), 32, "fp16", 2, 1),
    ((37, 45), (7, 5), (2, 1), 32, "fp16", 2, 2),
    ((20, 23), (3, 3), (3, 2), 64, "bf16", 1, 3),
    ((16, 16), (16, 16), (1, 1), 64, "fp32", 1, 2),
    ((9, 50), (9, 1), (1, 3), 128, "fp16", 1, 2),
    ((33, 31), (13, 13), (2, 2), 64, "bf16", 1, 2),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), 64, "fp16", 1, 2),
    ((5, 9, 11), (5, 3, 3), (1, 3, 3), 32, "fp32", 2, 1),
    ((8, 12, 12), (7, 7, 7), (1, 1, 1), 64, "bf16", 1, 1),
    ((4, 4, 4), (4, 4, 4), (1, 1, 1), 128, "fp16", 1, 2),
    # halos of more than 64 blocks: the per-wave block tests span two 64-block chunks
    ((10, 24, 24), (7, 9, 7), (1, 1, 1), 64, "fp16", 1, 1),
    ((48, 60), (21, 33), (1, 1), 32, "bf16", 1, 1),
]


@pytest.mark.parametrize("ext,ks,ds,D,dtype,B,H", FWD_CASES)
def test_forward_small(na, ext, ks, ds, D, dtype, B, H):
    shape = (B, H) + ext + (D,)
    q, k, v = _inputs(shape, dtype, 11, 3)
    out, lse = na.forward(*_dev(q, k, v), ks, ds)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, 1.0 / math.sqrt(D))
    eo, el = _maxerr(out, ro), _maxerr(lse, rl)
    _log(f"fwd {ext} k={ks} d={ds} D={D} {dtype}: max|dO|={eo:.3g} max|dLSE|={el:.3g}")
    assert eo <= TOL[dtype] and el <= TOL[dtype]


# 1-D forwards of 16-bit types run on 8-wave workgroups when the window and
# the problem are large; the environment forces that launch shape (and the query blocks per wave) on
# small ragged, dilated and causal problems too.
EIGHT_WAVE_CASES = [
    # (extents, kernel, dilation, causal, head_dim, dtype, batch, heads, blocks per wave)
    ((300,), (13,), (3,), None, 64, "fp16", 2, 2, 1),
    ((1000,), (255,), (2,), None, 64, "bf16", 1, 2, 2),
    ((777,), (129,), (1,), (True,), 32, "fp16", 1, 2, 2),
    ((513,), (31,), (4,), None, 128, "fp16", 1, 1, 1),
    ((2100,), (1023,), (2,), None, 64, "fp16", 1, 1, 2),
    ((900,), (255,), (3,), None, 128, "bf16", 1, 2, 2),
]


@pytest.mark.parametrize("ext,ks,ds,cs,D,dtype,B,H,m", EIGHT_WAVE_CASES)
def test_forward_eight_wave_workgroups(na, force, ext, ks, ds, cs, D, dtype, B, H, m):
    force(NA_FWD_WAVES=8, NA_WAVE_BLOCKS=m)
    shape = (B, H) + ext + (D,)
    q, k, v = _inputs(shape, dtype, 13, 3)
    out, lse = na.forward(*_dev(q, k, v), ks, ds, causal=cs)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, 1.0 / math.sqrt(D), causal=cs)
    eo, el = _maxerr(out, ro), _maxerr(lse, rl)
    _log(f"fwd 8 waves {ext} k={ks} d={ds} c={cs} D={D} {dtype} m={m}: "
         f"max|dO|={eo:.3g} max|dLSE|={el:.3g}")
    assert eo <= TOL[dtype] and el <= TOL[dtype]


# Scores that grow (or shrink) steeply along the key order: each tile of keys
# passes the running reference by far more than the lazy headroom, so the
# reference is raised again and again.  fp16 with 0.4 per key (natural log
# units, 12.8 per 32-key tile) overflows fp16 P before the raise; bf16 / fp32
# with 4 per key jump by ~185 in base 2 between tiles, past the fp32 range of
# exp2; the 2-D bf16 case starts rows at a first maximum below -128 in base 2;
# the fp16 cases at 1.25 per key and the scaled random ones reach logits of
# +-60.
#
# Gradients here reach |dK| = 320 and rows are nearly one-hot, so the
# backward is held to an elementwise bound derived from the arithmetic
# (_operator_bound, _end_to_end_bound) rather than to a flat 2e-2, which the
# rounding of a stored gradient of that size alone exceeds.
U_STORE = {"fp32": 2.0 ** -24, "fp16": 2.0 ** -11, "bf16": 2.0 ** -8}  # unit roundoff


def _score_error(dtype, D, q, k, ks, ds, sc, cs=None):
    """Per-query bound on the error of a recomputed score (natural-log units), shaped
    [B, H, X.., 1].  fp16 and fp32 at D <= 64 scale Q (or K) by scale*log2(e) and round it to
    the type once, which moves the score of pair (i, j) by at most
    u * scale * sum_c |q_ic| |k_jc|; bf16 and D = 128 apply that factor in fp32.  The largest
    of those sums over j in N(i) is bounded by the logsumexp of the absolute products at a
    temperature of 1/1000 (log-sum-exp >= max)."""
    u = U_STORE[dtype] if (dtype != "bf16" and D <= 64) else 2.0 ** -24
    temp = 1000.0
    _, lse_abs = oracle.forward(np.abs(q), np.abs(k), np.abs(k), ks, ds, sc * temp, causal=cs)
    return u * np.maximum(lse_abs / temp, 0.0)[..., None] + 2.0 ** -20


def _operator_bound(dtype, D, ell, e_s, refs, abs_sums):
    """Elementwise bound on |GPU - oracle| for na_backward run on exactly the oracle's inputs
    (q, k, v, out, lse, dout): the flat tolerance, plus the rounding of the terms dA and P to
    the storage type (u relative), the score error e_s carried into every P (dQ: that query's;
    dK, dV: the largest), and the fp32 accumulations, each relative to the sum of absolute
    terms; plus the rounding of the stored gradient itself (u |ref|)."""
    u = U_STORE[dtype]
    acc = u + 2.0 ** -24 * (ell + D)
    e_max = float(e_s.max())
    rel = [acc + np.expm1(e_s), acc + math.expm1(e_max), acc + math.expm1(e_max)]
    return [TOL[dtype] + r_ * a + u * np.abs(r) for r, a, r_ in zip(refs, abs_sums, rel)]


def _end_to_end_bound(dtype, D, ell, e_s, q, k, v, g, ks, ds, sc, cs, refs, abs_sums):
    """Elementwise bound on |GPU - oracle| for the GPU forward followed by the GPU backward.
    Beyond _operator_bound, the backward then takes Delta_i = dO_i.O_i from the GPU's stored O
    and P from its stored logsumexp.  The stored O differs from the exact one by at most
    eps_O = (u + 2 u_P + 2 e_s) (P|V|) (rounding of O; rounding and score error of the
    normalised P), so Delta_i moves by at most w_i = sum_c |dO_ic| eps_O,ic; since the
    backward is affine in Delta, dQ_i moves by at most scale w_i |sum_j P_ij k_j| and dK_j by
    scale sum_i P_ij w_i |q_i|.  The stored logsumexp carries the score error too, which
    scales every P, hence every gradient term, by at most e^e_s - 1."""
    u = U_STORE[dtype]
    u_p = u if dtype != "fp32" else 2.0 ** -24
    pv, _ = oracle.forward(q, k, np.abs(v), ks, ds, sc, causal=cs)
    pk, _ = oracle.forward(q, k, k, ks, ds, sc, causal=cs)
    w = (np.abs(g) * (u + 2 * u_p + 2 * np.expm1(e_s)) * pv).sum(-1, keepdims=True)
    _, _, in_wq = oracle.backward(q, k, v, w * np.abs(q), ks, ds, sc, causal=cs)
    base = _operator_bound(dtype, D, ell, e_s, refs, abs_sums)
    e_max = math.expm1(float(e_s.max()))
    return [base[0] + sc * w * np.abs(pk) + np.expm1(e_s) * abs_sums[0],
            base[1] + sc * in_wq + e_max * abs_sums[1],
            base[2] + e_max * abs_sums[2]]


def _steep_inputs(ext, D, dtype, a, seed=21):
    """q = (a / scale) e0 and k[..., 0] = centred index along the outermost axis (1-D: the key
    index; 2-D: the row), so q.k * scale = a * index; a = None draws q, k, v, dO iid N(0, 1)
    and multiplies q by 20, giving logits of standard deviation 20 (extremes near +-60)."""
    shape = (1, 2) + ext + (D,)
    gen = torch.Generator().manual_seed(seed)
    scale = 1.0 / math.sqrt(D)
    if a is None:
        q, k, v, g = (torch.randn(shape, generator=gen, dtype=torch.float64) for _ in range(4))
        q = q * 20.0
    else:
        q = torch.zeros(shape, dtype=torch.float64)
        q[..., 0] = a / scale
        idx = torch.arange(ext[0], dtype=torch.float64) - ext[0] // 2
        k = torch.randn(shape, generator=gen, dtype=torch.float64)
        k[..., 0] = idx.view((ext[0],) + (1,) * (len(ext) - 1))
        v = torch.randn(shape, generator=gen, dtype=torch.float64)
        g = torch.randn(shape, generator=gen, dtype=torch.float64)
    return [t.to(TDT[dtype]) for t in (q, k, v, g)], scale


STEEP_CASES = [
    # (extents, kernel, head_dim, dtype, growth per key step (None: scaled random), blocks/wave)
    ((96,), (47,), 64, "fp16", 0.4, 1),
    ((96,), (47,), 64, "fp16", 0.4, 2),
    ((96,), (47,), 64, "fp16", -0.4, 2),
    ((96,), (47,), 64, "fp16", 1.25, 2),
    ((96,), (47,), 64, "fp16", -1.25, 1),
    ((96,), (47,), 64, "bf16", 4.0, 2),
    ((96,), (47,), 32, "fp32", 4.0, 1),
    ((96,), (47,), 32, "fp32", -4.0, 2),
    ((12, 40), (5, 9), 32, "bf16", 40.0, 1),
    ((12, 40), (5, 9), 64, "fp16", 2.0, 2),
    ((48, 40), (7, 9), 64, "fp16", 1.25, 2),
    ((200,), (31,), 64, "fp16", None, 2),
    ((30, 40), (7, 9), 32, "fp16", None, 1),
    ((200,), (31,), 64, "bf16", None, 1),
]


@pytest.mark.parametrize("ext,ks,D,dtype,a,m", STEEP_CASES)
def test_steep_scores_raise_the_reference(na, force, ext, ks, D, dtype, a, m):
    force(NA_WAVE_BLOCKS=m)
    (q, k, v, g), scale = _steep_inputs(ext, D, dtype, a)
    ds = (1,) * len(ext)
    ell = int(np.prod(ks))
    qd, kd, vd, gd = _dev(q, k, v, g)
    fq, fk, fv, fg = (_f64(t) for t in (q, k, v, g))
    out, lse = na.forward(qd, kd, vd, ks, ds)
    ro, rl = oracle.forward(fq, fk, fv, ks, ds, scale)
    eo, el = _maxerr(out, ro), _maxerr(lse, rl)
    _, lmax = oracle.forward(fq, fk, fv, ks, ds, scale * 1000.0)
    _log(f"fwd steep {ext} k={ks} D={D} {dtype} a={a} m={m}: max|dO|={eo:.3g} "
         f"max|dLSE|={el:.3g} max logit={float(lmax.max()) / 1000.0:.3g}")
    assert np.isfinite(_f64(out)).all() and np.isfinite(_f64(lse)).all()
    assert eo <= TOL[dtype] and el <= TOL[dtype]

    # the backward operator on exactly the oracle's stored results (out rounded to the type,
    # logsumexp to fp32), against the oracle's operator on the same values
    out_s = torch.from_numpy(ro).to(TDT[dtype])
    lse_s = torch.from_numpy(rl).float()
    refs = oracle.backward_given(fq, fk, fv, _f64(out_s), _f64(lse_s), fg, ks, ds, scale,
                                 abs_sums=True)
    got = na.backward(qd, kd, vd, out_s.cuda(), lse_s.cuda(), gd, ks, ds)
    e_s = _score_error(dtype, D, fq, fk, ks, ds, scale)
    bound = _operator_bound(dtype, D, ell, e_s, refs[:3], refs[3:])
    worst = [float((np.abs(_f64(x) - r) / b).max()) for x, r, b in zip(got, refs[:3], bound)]
    _log(f"bwd steep operator {ext} {dtype} a={a} m={m}: max err / bound dq/dk/dv = "
         f"{[f'{x:.3g}' for x in worst]}")
    for x in got:
        assert np.isfinite(_f64(x)).all()
    assert max(worst) <= 1.0

    # forward then backward on the GPU, against the oracle's plain backward
    dq, dk, dv = na.backward(qd, kd, vd, out, lse, gd, ks, ds)
    full = oracle.backward_given(fq, fk, fv, ro, rl, fg, ks, ds, scale, abs_sums=True)
    bound = _end_to_end_bound(dtype, D, ell, e_s, fq, fk, fv, fg, ks, ds, scale, None, full[:3],
                              full[3:])
    worst = [float((np.abs(_f64(x) - r) / b).max()) for x, r, b in zip((dq, dk, dv), full[:3],
                                                                         bound)]
    flat = [_maxerr(x, r) for x, r in zip((dq, dk, dv), full[:3])]
    _log(f"bwd steep end-to-end {ext} {dtype} a={a} m={m}: max err dq/dk/dv = "
         f"{[f'{x:.3g}' for x in flat]}, / bound = {[f'{x:.3g}' for x in worst]}")
    assert max(worst) <= 1.0


def test_forward_window_one_is_exact_copy(na):
    for dtype in ("fp16", "bf16", "fp32"):
        shape = (2, 2, 13, 17, 64)
        q, k, v = _inputs(shape, dtype, 12, 3)
        out, lse = na.forward(*_dev(q, k, v), (1, 1), (3, 2))
        assert torch.equal(out.cpu(), v), dtype
        ref = (q.double() * k.double()).sum(-1) / 8.0
        assert float((lse.cpu().double() - ref).abs().max()) <= TOL[dtype]


def test_forward_deterministic_and_empty(na):
    shape = (1, 2, 24, 40, 64)
    q, k, v = _dev(*_inputs(shape, "fp16", 13, 3))
    a, la = na.forward(q, k, v, (5, 7), (2, 3))
    b, lb = na.forward(q, k, v, (5, 7), (2, 3))
    assert torch.equal(a, b) and torch.equal(la, lb)
    z = torch.empty((0, 2, 24, 40, 64), dtype=torch.float16, device="cuda")
    o, l = na.forward(z, z, z, (5, 7), (2, 3))
    assert o.shape == z.shape


# Dilation at its limits (Sec. 3.4): windows that fill their whole sub-lattice
# (k * d = L), sub-lattices of unequal length (d does not divide L) whose
# shorter groups are exactly k long, dilation larger than the window, and a
# single group per axis of the other axis, in all dtypes, forward and backward.
DILATION_EDGE_CASES = [
    # (extents, kernel, dilation, causal, head_dim, dtype)
    ((12, 15), (4, 5), (3, 3), None, 32, "fp16"),
    ((10,), (3,), (3,), None, 64, "bf16"),
    ((10, 11), (3, 2), (3, 5), None, 64, "fp32"),
    ((7, 9, 10), (2, 3, 3), (3, 3, 3), None, 32, "fp16"),
    ((31, 17), (3, 4), (10, 4), (True, False), 64, "bf16"),
    ((64,), (2,), (32,), (True,), 32, "fp16"),
    ((16, 16, 16), (16, 1, 4), (1, 16, 4), None, 64, "fp16"),
]


@pytest.mark.parametrize("ext,ks,ds,cs,D,dtype", DILATION_EDGE_CASES)
def test_dilation_edge_cases(na, ext, ks, ds, cs, D, dtype):
    shape = (1, 2) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 41, 4)
    qd, kd, vd, gd = _dev(q, k, v, g)
    scale = 1.0 / math.sqrt(D)
    out, lse = na.forward(qd, kd, vd, ks, ds, causal=cs)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, scale, causal=cs)
    dq, dk, dv = na.backward(qd, kd, vd, out, lse, gd, ks, ds, causal=cs)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, scale, causal=cs)
    e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv)]
    _log(f"dilation edge {ext} k={ks} d={ds} c={cs} D={D} {dtype}: max err o/lse/dq/dk/dv = "
         f"{[f'{x:.3g}' for x in e]}")
    assert max(e) <= TOL[dtype]


# ---------------------------------------------------------------- backward
BWD_CASES = [
    ((200,), (7,), (1,), 32, "fp32", 1, 2),
    ((300,), (13,), (3,), 64, "fp16", 1, 2),
    ((257,), (64,), (4,), 64, "bf16", 1, 1),
    ((37, 45), (7, 5), (2, 1), 32, "fp16", 1, 2),
    ((20, 23), (3, 3), (3, 2), 64, "bf16", 1, 2),
    ((16, 16), (16, 16), (1, 1), 64, "fp32", 1, 1),
    ((33, 31), (13, 13), (2, 2), 64, "bf16", 1, 1),
    ((9, 50), (9, 1), (1, 3), 128, "fp16", 1, 1),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), 64, "fp16", 1, 1),
    ((5, 9, 11), (5, 3, 3), (1, 3, 3), 32, "fp32", 1, 2),
    ((8, 12, 12), (7, 7, 7), (1, 1, 1), 128, "bf16", 1, 1),
    # query boxes of border key tiles wider than the interior T + k - 1
    # (keys within k - 1 of the start are attended from query 0): 3 blocks
    # per row where the interior needs 2
    ((5, 40), (3, 17), (1, 1), 32, "fp16", 1, 1),
    ((3, 4, 64), (3, 3, 25), (1, 1, 1), 32, "bf16", 1, 1),
    ((4, 81), (3, 9), (1, 2), 64, "fp16", 1, 1),
    # halos and query boxes of more than 64 blocks (two 64-block test chunks)
    ((10, 24, 24), (7, 9, 7), (1, 1, 1), 64, "fp16", 1, 1),
    ((48, 60), (21, 33), (1, 1), 32, "bf16", 1, 1),
]


@pytest.mark.parametrize("ext,ks,ds,D,dtype,B,H", BWD_CASES)
def test_backward_small(na, ext, ks, ds, D, dtype, B, H):
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 21, 4)
    dq_, dk_, dv_, dg_ = _dev(q, k, v, g)
    out, lse = na.forward(dq_, dk_, dv_, ks, ds)
    dq, dk, dv = na.backward(dq_, dk_, dv_, out, lse, dg_, ks, ds)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, 1.0 / math.sqrt(D))
    e = [_maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv)]
    _log(f"bwd {ext} k={ks} d={ds} D={D} {dtype}: max err dq/dk/dv = {e}")
    assert max(e) <= TOL[dtype]


# The backward runs as one launch of both roles, or split into a Delta pre-pass, a dK/dV launch
# and a dQ launch (large 3-D problems with two blocks per wave by default); the environment
# forces each form on problems the other would take.
SPLIT_CASES = [
    # (extents, kernel, dilation, causal, head_dim, dtype, blocks per wave, split)
    ((300,), (13,), (3,), None, 64, "fp16", 2, 1),
    ((257,), (64,), (4,), (True,), 64, "bf16", 1, 1),
    ((1500,), (600,), (2,), None, 64, "fp16", 2, 1),  # the 1-D split of long windows
    ((1500,), (600,), (2,), None, 32, "bf16", 2, 1),
    ((37, 45), (7, 5), (2, 1), None, 32, "fp16", 2, 1),
    ((33, 31), (13, 13), (2, 2), (True, False), 64, "bf16", 1, 1),
    ((5, 40), (3, 17), (1, 1), None, 32, "fp16", 1, 1),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), None, 64, "fp16", 2, 1),
    ((8, 12, 12), (7, 7, 7), (1, 1, 1), (True, False, False), 32, "bf16", 2, 1),
    ((3, 4, 64), (3, 3, 25), (1, 1, 1), None, 64, "fp16", 1, 1),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), None, 64, "fp16", 2, 0),
    ((8, 12, 12), (7, 7, 7), (1, 1, 1), (True, False, False), 32, "bf16", 2, 0),
    ((10, 24, 24), (7, 9, 7), (1, 1, 1), None, 64, "fp16", 2, 1),  # boxes of > 64 blocks
]


@pytest.mark.parametrize("ext,ks,ds,cs,D,dtype,m,split", SPLIT_CASES)
def test_backward_split_and_single_launch(na, force, ext, ks, ds, cs, D, dtype, m, split):
    force(NA_WAVE_BLOCKS=m, NA_BWD_SPLIT=split)
    shape = (1, 2) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 24, 4)
    qd, kd, vd, gd = _dev(q, k, v, g)
    sc = 1.0 / math.sqrt(D)
    out, lse = na.forward(qd, kd, vd, ks, ds, causal=cs)
    dq, dk, dv = na.backward(qd, kd, vd, out, lse, gd, ks, ds, causal=cs)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc, causal=cs)
    e = [_maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv)]
    _log(f"bwd {'split' if split else 'single launch'} {ext} k={ks} d={ds} c={cs} D={D} {dtype} "
         f"m={m}: max err dq/dk/dv = {[f'{x:.3g}' for x in e]}")
    assert max(e) <= TOL[dtype]
    again = na.backward(qd, kd, vd, out, lse, gd, ks, ds, causal=cs)
    for a, b in zip((dq, dk, dv), again):
        assert torch.equal(a, b)


def test_backward_deterministic(na):
    shape = (1, 2, 30, 27, 64)
    q, k, v, g = _dev(*_inputs(shape, "bf16", 22, 4))
    out, lse = na.forward(q, k, v, (7, 5), (2, 3))
    a = na.backward(q, k, v, out, lse, g, (7, 5), (2, 3))
    b = na.backward(q, k, v, out, lse, g, (7, 5), (2, 3))
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_autograd_function_matches_explicit_calls(na):
    shape = (1, 2, 19, 64)
    q, k, v, g = _dev(*_inputs(shape, "fp32", 23, 4))
    qq, kk, vv = (t.clone().requires_grad_(True) for t in (q, k, v))
    o = na.na_attention(qq, kk, vv, 5, 2)
    o.backward(g)
    out, lse = na.forward(q, k, v, 5, 2)
    dq, dk, dv = na.backward(q, k, v, out, lse, g, 5, 2)
    assert torch.equal(o.detach(), out)
    for a, b in ((qq.grad, dq), (kk.grad, dk), (vv.grad, dv)):
        assert torch.equal(a, b)


# ---------------------------------------------------------------- full-size workloads
# Every workload at full size, in the launch configuration bench.py times, compared element by
# element against the oracle on the whole tensors (O, LSE, dQ, dK, dV); the unfused baseline
# (na_unfused_*) is compared against the same oracle results.
@pytest.mark.parametrize("name", workloads.CONFIG_ORDER)
def test_full_workload_forward(na, name):
    p = workloads.CONFIGS[name]
    _log(f"[full fwd] {p.describe()}")
    x = workloads.make_inputs(p, seed=0, with_grad=False)
    cz = p.causal_axes
    out, lse = na.forward(*_dev(x["q"], x["k"], x["v"]), p.kernel_size, p.dilation,
                          p.softmax_scale, causal=cz)
    torch.cuda.synchronize()
    # the unfused baseline (separate PN, softmax and NN launches) on the same inputs
    uo, ul, _ = na.unfused_forward(*_dev(x["q"], x["k"], x["v"]), p.kernel_size, p.dilation,
                                   p.softmax_scale, causal=cz)
    torch.cuda.synchronize()
    qd, kd, vd = (_f64(x[n]) for n in ("q", "k", "v"))
    ro, rl = oracle.forward(qd, kd, vd, p.kernel_size, p.dilation, p.softmax_scale, causal=cz)
    eo, el = _maxerr(out, ro), _maxerr(lse, rl)
    uo_e, ul_e = _maxerr(uo, ro), _maxerr(ul, rl)
    _log(f"[full fwd] {name}: {ro.size} outputs, {rl.size} logsumexps: max|dO|={eo:.3g} "
         f"max|dLSE|={el:.3g}; unfused max|dO|={uo_e:.3g} max|dLSE|={ul_e:.3g}")
    assert eo <= TOL[p.dtype] and el <= TOL[p.dtype]
    assert uo_e <= TOL[p.dtype] and ul_e <= TOL[p.dtype]


@pytest.mark.parametrize("name", workloads.CONFIG_ORDER)
def test_full_workload_backward(na, name):
    """Every workload's backward at full size (bench.py times the backward of any of them)."""
    p = workloads.CONFIGS[name]
    _log(f"[full bwd] {p.describe()}")
    x = workloads.make_inputs(p, seed=0, with_grad=True)
    q, k, v, g = _dev(x["q"], x["k"], x["v"], x["dout"])
    cz = p.causal_axes
    out, lse = na.forward(q, k, v, p.kernel_size, p.dilation, p.softmax_scale, causal=cz)
    dq, dk, dv = na.backward(q, k, v, out, lse, g, p.kernel_size, p.dilation, p.softmax_scale,
                             causal=cz)
    # the unfused baseline: PN, softmax backward, NN and two IN launches
    _, _, probs = na.unfused_forward(q, k, v, p.kernel_size, p.dilation, p.softmax_scale,
                                     causal=cz)
    ug = na.unfused_backward(q, k, v, probs, g, p.kernel_size, p.dilation, p.softmax_scale,
                             causal=cz)
    torch.cuda.synchronize()
    del q, k, v, g, out, lse, probs
    refs = oracle.backward(*(_f64(x[n]) for n in ("q", "k", "v", "dout")), p.kernel_size,
                           p.dilation, p.softmax_scale, causal=cz)
    e = [_maxerr(a, r) for a, r in zip((dq, dk, dv), refs)]
    ue = [_maxerr(a, r) for a, r in zip(ug, refs)]
    _log(f"[full bwd] {name}: 3 x {refs[0].size} gradients: max err dq/dk/dv = "
         f"{[f'{x:.3g}' for x in e]}; unfused {[f'{x:.3g}' for x in ue]}")
    assert max(e) <= TOL[p.dtype]
    assert max(ue) <= TOL[p.dtype]


# ---------------------------------------------------------------- causal axes
CAUSAL_WINDOWS = [
    ((40,), (7,), (1,), (1,)), ((37,), (4,), (3,), (1,)), ((16, 64, 64), (7, 7, 7), (1, 2, 2), (1, 0, 0)),
    ((10, 9), (3, 2), (3, 4), (1, 1)),
]


@pytest.mark.parametrize("ext,ks,ds,cs", CAUSAL_WINDOWS)
def test_causal_debug_windows_bit_exact(na, ext, ks, ds, cs):
    start, ilo, ihi = (t.cpu().numpy() for t in na.debug_windows(ext, ks, ds, causal=cs))
    off = 0
    for a, L in enumerate(ext):
        first, lo, hi, _ = oracle.axis_relation(L, ks[a], ds[a], causal=bool(cs[a]))
        np.testing.assert_array_equal(start[off:off + L], first)
        np.testing.assert_array_equal(ilo[off:off + L], lo)
        np.testing.assert_array_equal(ihi[off:off + L], hi)
        off += L


@pytest.mark.parametrize("ext,ks,ds,cs,dtype", [
    ((70,), (9,), (1,), (1,), "fp16"), ((21, 26), (5, 3), (2, 3), (1, 0), "fp16"),
    ((6, 9, 10), (3, 5, 3), (2, 1, 3), (1, 0, 1), "bf16"), ((60,), (7,), (2,), (1,), "fp32"),
])
def test_causal_neighbour_support_probe(na, ext, ks, ds, cs, dtype):
    """Q = 0: P uniform on N(i), so one-hot V rows expose the causal N(i) exactly."""
    D = 32
    N = int(np.prod(ext))
    lists = bf.neighbours(ext, ks, ds, [bool(c) for c in cs])
    q = torch.zeros((1, 1) + ext + (D,), dtype=TDT[dtype])
    k = _inputs(q.shape, dtype, 5, 1)[0]
    for chunk in range((N + D - 1) // D):
        v = torch.zeros(1, 1, N, D)
        for c in range(D):
            if chunk * D + c < N:
                v[0, 0, chunk * D + c, c] = 1.0
        v = v.reshape(q.shape).to(TDT[dtype])
        out, lse = na.forward(*_dev(q, k, v), ks, ds, causal=cs)
        o = out.float().cpu().reshape(N, D).numpy()
        for i in range(N):
            want = set(t - chunk * D for t in lists[i] if chunk * D <= t < (chunk + 1) * D)
            assert set(np.nonzero(o[i])[0].tolist()) == want, (i, chunk)
        sizes = np.array([math.log(len(r)) for r in lists]).reshape(lse.shape[2:])
        np.testing.assert_allclose(lse.cpu().numpy()[0, 0], sizes, atol=1e-5)


CAUSAL_CASES = [
    # (extents, kernel, dilation, causal, head_dim, dtype, batch, heads)
    ((200,), (7,), (1,), (1,), 32, "fp32", 1, 2),
    ((300,), (13,), (3,), (1,), 64, "fp16", 1, 2),
    ((1000,), (255,), (2,), (1,), 64, "bf16", 1, 1),
    ((37, 45), (7, 5), (2, 1), (1, 0), 32, "fp16", 1, 2),
    ((20, 23), (3, 3), (3, 2), (0, 1), 64, "bf16", 1, 2),
    ((33, 31), (13, 13), (2, 2), (1, 1), 64, "bf16", 1, 1),
    ((9, 50), (9, 25), (1, 2), (0, 1), 128, "fp16", 1, 1),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), (1, 0, 0), 64, "fp16", 1, 1),
    ((8, 12, 12), (7, 7, 7), (1, 1, 1), (1, 0, 0), 32, "fp16", 1, 2),
    ((5, 9, 11), (5, 3, 3), (1, 3, 3), (1, 1, 1), 32, "fp32", 1, 1),
]


@pytest.mark.parametrize("ext,ks,ds,cs,D,dtype,B,H", CAUSAL_CASES)
def test_causal_forward_and_backward_small(na, ext, ks, ds, cs, D, dtype, B, H):
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 31, 4)
    dq_, dk_, dv_, dg_ = _dev(q, k, v, g)
    out, lse = na.forward(dq_, dk_, dv_, ks, ds, causal=cs)
    dq, dk, dv = na.backward(dq_, dk_, dv_, out, lse, dg_, ks, ds, causal=cs)
    sc = 1.0 / math.sqrt(D)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc, causal=cs)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc, causal=cs)
    e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv)]
    _log(f"causal {ext} k={ks} d={ds} c={cs} D={D} {dtype}: max err o/lse/dq/dk/dv = {e}")
    assert max(e) <= TOL[dtype]


# ---------------------------------------------------------------- maximum sizes
def _gpu_inputs(shape, dtype, seed, n):
    """Seeded synthetic inputs drawn on the GPU (the tensors are too large to stage from the host)."""
    gen = torch.Generator(device="cuda").manual_seed(seed)
    return [torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32).to(TDT[dtype])
            for _ in range(n)]


def test_max_grid_many_slices(na):
    """65,536 (batch, head) slices, 2 GiB per tensor: 64-bit slice offsets and a large grid.
    Each slice is an independent problem, so sampled slices are checked alone."""
    B, H, L, D, ks, ds = 256, 256, 256, 64, (7,), (2,)
    q, k, v, g = _gpu_inputs((B, H, L, D), "fp16", 71, 4)
    out, lse = na.forward(q, k, v, ks, ds)
    dq, dk, dv = na.backward(q, k, v, out, lse, g, ks, ds)
    torch.cuda.synchronize()
    sc = 1.0 / math.sqrt(D)
    for b, h in [(0, 0), (B - 1, H - 1), (17, 200), (128, 3), (255, 0)]:
        sl = lambda t: _f64(t[b:b + 1, h:h + 1])
        ro, rl = oracle.forward(sl(q), sl(k), sl(v), ks, ds, sc)
        rq, rk, rv = oracle.backward(sl(q), sl(k), sl(v), sl(g), ks, ds, sc)
        e = [float(np.max(np.abs(sl(a) - r))) for a, r in
             ((out, ro), (lse, rl), (dq, rq), (dk, rk), (dv, rv))]
        _log(f"max grid slice ({b},{h}): max err o/lse/dq/dk/dv = {e}")
        assert max(e) <= TOL["fp16"]
    del q, k, v, g, out, lse, dq, dk, dv
    torch.cuda.empty_cache()


def test_max_tokens_times_head_dim(na):
    """One 1-D slice with N * D = 2^30 (the 32-bit token-offset limit is 2^31): the rows of
    sampled queries and keys are checked on sub-sequences large enough that their windows and
    inverse neighbourhoods are those of the full sequence (anchored at the true borders)."""
    L, D, kk = 1 << 24, 64, 9
    q, k, v, g = _gpu_inputs((1, 1, L, D), "fp16", 72, 4)
    out, lse = na.forward(q, k, v, (kk,), (1,))
    dq, dk, dv = na.backward(q, k, v, out, lse, g, (kk,), (1,))
    torch.cuda.synchronize()
    sc = 1.0 / math.sqrt(D)
    margin = 3 * kk
    for x in [0, 3, 4099, L // 2 + 1, L - 5, L - 1]:
        lo, hi = max(0, x - margin), min(L, x + margin + 1)
        sub = lambda t: _f64(t[:, :, lo:hi])
        ro, rl = oracle.forward(sub(q), sub(k), sub(v), (kk,), (1,), sc)
        rq, rk, rv = oracle.backward(sub(q), sub(k), sub(v), sub(g), (kk,), (1,), sc)
        i = x - lo
        at = lambda t: _f64(t[0, 0, x])
        e = [float(np.max(np.abs(at(out) - ro[0, 0, i]))), abs(float(lse[0, 0, x]) - rl[0, 0, i]),
             float(np.max(np.abs(at(dq) - rq[0, 0, i]))), float(np.max(np.abs(at(dk) - rk[0, 0, i]))),
             float(np.max(np.abs(at(dv) - rv[0, 0, i])))]
        _log(f"max N*D row {x}: max err o/lse/dq/dk/dv = {e}")
        assert max(e) <= TOL["fp16"]
    del q, k, v, g, out, lse, dq, dk, dv
    torch.cuda.empty_cache()


# ---------------------------------------------------------------- tilings and the tuner
TILING_CASES = [
    # (extents, kernel, dilation, causal, head_dim, dtype, batch, heads)
    ((37, 45), (7, 5), (2, 1), None, 32, "fp16", 2, 2),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), None, 64, "fp16", 1, 2),
    ((300,), (13,), (3,), None, 64, "bf16", 2, 2),
    ((17, 33), (5, 9), (1, 2), (True, False), 64, "bf16", 1, 2),
    ((5, 9, 11), (5, 3, 3), (1, 3, 3), None, 32, "fp32", 2, 1),
    # head dim 128: two-block tilings of the 16-bit kernels, and the 8-wave 1-D forwards
    ((9, 40), (5, 7), (1, 2), None, 128, "fp16", 1, 2),
    ((300,), (31,), (2,), None, 128, "bf16", 1, 2),
    ((6, 12, 20), (3, 5, 5), (1, 2, 1), None, 128, "fp16", 1, 1),
    # head dim 128 with long windows: many of the halved one-block stages (2 blocks, 4 with 8 waves)
    ((1300,), (511,), (2,), None, 128, "fp16", 1, 1),
    ((40, 48), (13, 21), (1, 1), None, 128, "bf16", 1, 1),
]


@pytest.mark.parametrize("ext,ks,ds,cs,D,dtype,B,H", TILING_CASES)
def test_every_candidate_tiling_matches_the_oracle(na, ext, ks, ds, cs, D, dtype, B, H):
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 41, 4)
    dq_, dk_, dv_, dg_ = _dev(q, k, v, g)
    sc = 1.0 / math.sqrt(D)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc, causal=cs)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc, causal=cs)
    fwd_c = na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=True)
    bwd_c = na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=False)
    worst = 0.0
    for t in fwd_c:
        out, lse = na.forward(dq_, dk_, dv_, ks, ds, causal=cs, tiling=t)
        e = max(_maxerr(out, ro), _maxerr(lse, rl))
        assert e <= TOL[dtype], (t, e)
        worst = max(worst, e)
    out, lse = na.forward(dq_, dk_, dv_, ks, ds, causal=cs)
    for t in bwd_c:
        dq, dk, dv = na.backward(dq_, dk_, dv_, out, lse, dg_, ks, ds, causal=cs, tiling=t)
        e = max(_maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv))
        assert e <= TOL[dtype], (t, e)
        worst = max(worst, e)
    _log(f"tilings {ext} k={ks} d={ds} c={cs} D={D} {dtype}: {len(fwd_c)} forward and "
         f"{len(bwd_c)} backward tilings, worst max err {worst:.3g}")


# Head dim 128 with two query blocks per wave: the heuristic picks it for the forward of large
# 16-bit problems (at least 1024 workgroups remain); the environment forces it for the
# backward and the 8-wave 1-D forward too.
D128_CASES = [
    # (extents, kernel, dilation, dtype, batch, heads, forced blocks per wave or None, 8 waves)
    ((4096,), (63,), (1,), "fp16", 1, 32, None, False),
    ((16, 32, 32), (7, 7, 7), (1, 1, 1), "bf16", 1, 8, None, False),
    ((700,), (45,), (3,), "bf16", 1, 2, 2, False),
    ((37, 29), (7, 5), (2, 1), "fp16", 1, 2, 2, False),
    ((6, 13, 22), (3, 5, 7), (1, 1, 2), "bf16", 1, 1, 2, False),
    ((1300,), (511,), (2,), "fp16", 1, 1, 2, True),
]


@pytest.mark.parametrize("ext,ks,ds,dtype,B,H,m,eight", D128_CASES)
def test_head_dim_128_two_blocks_per_wave(na, force, ext, ks, ds, dtype, B, H, m, eight):
    D = 128
    if m is not None:
        force(NA_WAVE_BLOCKS=m)
    if eight:
        force(NA_FWD_WAVES=8)
    t = na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=True)
    assert t.blocks_per_wave == 2 and (not eight or t.waves[0] == 8), t
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 45, 4)
    qd, kd, vd, gd = _dev(q, k, v, g)
    sc = 1.0 / math.sqrt(D)
    out, lse = na.forward(qd, kd, vd, ks, ds)
    dq, dk, dv = na.backward(qd, kd, vd, out, lse, gd, ks, ds)
    tb = na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=False)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc)
    e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv)]
    _log(f"D=128 {ext} k={ks} d={ds} {dtype} fwd tiling {t} bwd tiling {tb}: "
         f"max err o/lse/dq/dk/dv = {[f'{x:.3g}' for x in e]}")
    assert max(e) <= TOL[dtype]


def test_tune_records_the_fastest_tilings_and_keeps_parity(na):
    ext, ks, ds, D, dtype, B, H = (40, 48), (7, 7), (1, 1), 32, "fp16", 2, 4
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 43, 4)
    dq_, dk_, dv_, dg_ = _dev(q, k, v, g)
    sc = 1.0 / math.sqrt(D)
    na.tune_clear()
    heur_f = na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=True)
    bf, bb, times = na.tune(dq_, dk_, dv_, dg_, ks, ds, repeats=3)
    try:
        assert bf in na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=True)
        assert bb in na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=False)
        assert na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=True) == bf
        assert na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=False) == bb
        assert 0 < times[0] <= times[2] and 0 < times[1] <= times[3]
        ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc)
        rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc)
        out, lse = na.forward(dq_, dk_, dv_, ks, ds)  # the tuned tiling
        dq, dk, dv = na.backward(dq_, dk_, dv_, out, lse, dg_, ks, ds)
        e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk),
             _maxerr(dv, rv)]
        _log(f"tuned {bf} / {bb}, ms {times}: max err {e}")
        assert max(e) <= TOL[dtype]
    finally:
        na.tune_clear()
    assert na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=True) == heur_f


def test_thorough_tune_times_every_candidate_and_keeps_parity(na):
    """A 3-D problem with more candidate tilings than na_tune times by default: the thorough
    mode may pick any of them, and the tuned launches match the oracle."""
    ext, ks, ds, D, dtype, B, H = (16, 32, 32), (7, 7, 7), (1, 1, 1), 64, "fp16", 1, 2
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 44, 4)
    dq_, dk_, dv_, dg_ = _dev(q, k, v, g)
    sc = 1.0 / math.sqrt(D)
    fc = na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=True)
    assert len(fc) > 64
    na.tune_clear()
    try:
        bf, bb, times = na.tune(dq_, dk_, dv_, dg_, ks, ds, repeats=2, thorough=True)
        assert bf in fc
        assert bb in na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=False)
        assert 0 < times[0] <= times[2] and 0 < times[1] <= times[3]
        out, lse = na.forward(dq_, dk_, dv_, ks, ds)
        dq, dk, dv = na.backward(dq_, dk_, dv_, out, lse, dg_, ks, ds)
        ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc)
        rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc)
        e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk),
             _maxerr(dv, rv)]
        _log(f"thorough tune of {len(fc)} forward tilings: {bf} / {bb}, ms {times}: "
             f"max err {[f'{x:.3g}' for x in e]}")
        assert max(e) <= TOL[dtype]
    finally:
        na.tune_clear()


def test_tune_on_first_use(na):
    """With tuning on first use, the first forward and backward of a problem tune it on the
    call's own buffers and return the chosen tiling's results; later calls run that tiling."""
    ext, ks, ds, D, dtype, B, H = (40, 44), (9, 7), (2, 1), 64, "bf16", 1, 3
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 46, 4)
    dq_, dk_, dv_, dg_ = _dev(q, k, v, g)
    sc = 1.0 / math.sqrt(D)
    before = na.autotune()
    na.tune_clear()
    na.set_autotune(1)
    try:
        out, lse = na.forward(dq_, dk_, dv_, ks, ds)
        dq, dk, dv = na.backward(dq_, dk_, dv_, out, lse, dg_, ks, ds)
        tf = na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=True)
        tb = na.current_tiling(ext, ks, ds, B, H, D, TDT[dtype], forward=False)
        assert tf in na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=True)
        assert tb in na.candidate_tilings(ext, ks, ds, B, H, D, TDT[dtype], forward=False)
        out2, lse2 = na.forward(dq_, dk_, dv_, ks, ds)  # cached: no tuning, same tiling
        dq2, dk2, dv2 = na.backward(dq_, dk_, dv_, out, lse, dg_, ks, ds)
        for a, b in ((out, out2), (lse, lse2), (dq, dq2), (dk, dk2), (dv, dv2)):
            assert torch.equal(a, b)
        ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc)
        rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc)
        e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk),
             _maxerr(dv, rv)]
        _log(f"tuned on first use: {tf} / {tb}: max err {[f'{x:.3g}' for x in e]}")
        assert max(e) <= TOL[dtype]
    finally:
        na.set_autotune(before)
        na.tune_clear()


def test_graph_capture_replays_match_eager(na):
    """Forward and backward captured in one HIP graph replay the eager results bit for bit,
    replay after replay, with eager work on the same buffers in between."""
    ext, ks, ds, D, dtype, B, H = (24, 40), (7, 5), (1, 2), 32, "fp16", 2, 2
    shape = (B, H) + ext + (D,)
    q, k, v, g = _dev(*_inputs(shape, dtype, 47, 4))
    out, lse = torch.empty_like(q), torch.empty(q.shape[:-1], dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)

    def step():
        na.forward(q, k, v, ks, ds, out=out, lse=lse)
        na.backward(q, k, v, out, lse, g, ks, ds, dq=dq, dk=dk, dv=dv)

    step()
    torch.cuda.synchronize()
    want = [t.clone() for t in (out, lse, dq, dk, dv)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        step()  # warm-up on the capture stream
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=s):
            step()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (out, lse, dq, dk, dv):
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for name, got, ref in zip(("out", "lse", "dq", "dk", "dv"), (out, lse, dq, dk, dv), want):
            assert torch.equal(got, ref), (rep, name)
        step()  # eager work between replays
        torch.cuda.synchronize()


# ---------------------------------------------------------------- per-thread plans
PLAN_PROBLEMS = [
    # (extents, kernel, dilation, causal, head_dim, dtype): more problems than a thread keeps plans
    ((64,), (7,), (1,), None, 32, "fp16"), ((90,), (9,), (2,), (True,), 64, "bf16"),
    ((50,), (5,), (3,), None, 32, "fp32"), ((12, 14), (3, 5), (1, 1), None, 32, "fp16"),
    ((12, 14), (3, 5), (1, 1), (True, False), 32, "fp16"), ((20, 9), (5, 3), (2, 1), None, 64, "bf16"),
    ((6, 7, 8), (3, 3, 3), (1, 1, 2), None, 32, "fp16"), ((6, 7, 8), (3, 3, 3), (1, 1, 2), None, 64, "fp16"),
    ((33,), (7,), (1,), None, 128, "bf16"), ((10, 10), (10, 10), (1, 1), None, 32, "fp16"),
]


def _plan_case(na, i, seed):
    ext, ks, ds, cs, D, dtype = PLAN_PROBLEMS[i]
    shape = (1, 2) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, seed, 4)
    qd, kd, vd, gd = _dev(q, k, v, g)
    out, lse = na.forward(qd, kd, vd, ks, ds, causal=cs)
    dq, dk, dv = na.backward(qd, kd, vd, out, lse, gd, ks, ds, causal=cs)
    torch.cuda.synchronize()
    sc = 1.0 / math.sqrt(D)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc, causal=cs)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc, causal=cs)
    e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv)]
    return max(e) <= TOL[dtype], e


def test_plans_of_many_problems_and_threads(na):
    """Each thread keeps the last few problems' plans: cycling through more problems than
    that, twice (plans evicted, made again and reused, on fresh inputs), from one thread and
    then from two at once, every result still matches the oracle."""
    import threading

    na.tune_clear()
    for rnd in range(2):
        for i in range(len(PLAN_PROBLEMS)):
            ok, e = _plan_case(na, i, 60 + rnd)
            _log(f"plans round {rnd} problem {i}: max err {max(e):.3g}")
            assert ok, (rnd, i, e)
    results, errors = {}, []

    def worker(tid):
        try:
            for rnd in range(2):
                for i in range(tid, len(PLAN_PROBLEMS), 2):
                    results[(tid, rnd, i)] = _plan_case(na, i, 70 + tid + rnd)
        except Exception as ex:  # reported below, in the test's thread
            errors.append(repr(ex))

    threads = [threading.Thread(target=worker, args=(t,)) for t in (0, 1)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    assert len(results) == 2 * len(PLAN_PROBLEMS)
    for key, (ok, e) in results.items():
        assert ok, (key, e)
    # a plan made before na.tune_clear is not used after it (same result either way)
    ok, _ = _plan_case(na, 0, 80)
    na.tune_clear()
    ok2, _ = _plan_case(na, 0, 80)
    assert ok and ok2


# ---------------------------------------------------------------- random problems
def _random_problems(n, seed):
    """Seeded random problems of every rank: extents, windows (odd and even), dilations,
    causal axes, head dims and types, kept small enough for the oracle."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        rank = int(rng.integers(1, 4))
        budget = {1: 400, 2: 900, 3: 1200}[rank]
        ext, ks, ds, cs = [], [], [], []
        for _ in range(rank):
            L = int(rng.integers(2, {1: 400, 2: 40, 3: 14}[rank]))
            d = int(rng.integers(1, min(4, L) + 1))
            k = int(rng.integers(1, L // d + 1))
            ext.append(L), ds.append(d), ks.append(k), cs.append(bool(rng.random() < 0.25))
        if int(np.prod(ext)) > budget:
            continue
        D = int(rng.choice([32, 64, 128]))
        dtype = str(rng.choice(["fp16", "bf16", "fp32"]))
        B, H = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        out.append((tuple(ext), tuple(ks), tuple(ds), tuple(cs) if any(cs) else None, D, dtype,
                    B, H))
    return out


def _mid_problems(n, seed):
    """Seeded random 2-D / 3-D problems of up to 4608 / 7000 tokens with windows of at least 40
    keys, so that many workgroup halos hold more than 64 blocks (several 64-block test chunks)."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        rank = int(rng.integers(2, 4))
        ext, ks, ds, cs = [], [], [], []
        for _ in range(rank):
            L = int(rng.integers(8, {2: 72, 3: 26}[rank]))
            d = int(rng.integers(1, 3))
            k = int(rng.integers(1, L // d + 1))
            ext.append(L), ds.append(d), ks.append(k), cs.append(bool(rng.random() < 0.2))
        if int(np.prod(ext)) > {2: 4608, 3: 7000}[rank] or int(np.prod(ks)) < 40:
            continue
        D = int(rng.choice([32, 64]))
        dtype = str(rng.choice(["fp16", "bf16"]))
        out.append((tuple(ext), tuple(ks), tuple(ds), tuple(cs) if any(cs) else None, D, dtype,
                    1, 2))
    return out


def _check_random_problem(na, tag, problem, seed):
    """Forward within the flat tolerance.  The backward within the bound derived from its
    arithmetic (_end_to_end_bound: the flat tolerance plus roundings relative to the terms'
    magnitudes), since small windows give gradients large enough that storing them in bf16
    alone moves them by more than 2e-2 (|dQ| in [4, 8) has a half-ulp of 1/64)."""
    ext, ks, ds, cs, D, dtype, B, H = problem
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, seed, 4)
    qd, kd, vd, gd = _dev(q, k, v, g)
    fq, fk, fv, fg = (_f64(t) for t in (q, k, v, g))
    sc = 1.0 / math.sqrt(D)
    out, lse = na.forward(qd, kd, vd, ks, ds, causal=cs)
    dq, dk, dv = na.backward(qd, kd, vd, out, lse, gd, ks, ds, causal=cs)
    ro, rl = oracle.forward(fq, fk, fv, ks, ds, sc, causal=cs)
    full = oracle.backward_given(fq, fk, fv, ro, rl, fg, ks, ds, sc, causal=cs, abs_sums=True)
    ef = [_maxerr(out, ro), _maxerr(lse, rl)]
    eb = [_maxerr(x, r) for x, r in zip((dq, dk, dv), full[:3])]
    e_s = _score_error(dtype, D, fq, fk, ks, ds, sc, cs)
    bound = _end_to_end_bound(dtype, D, int(np.prod(ks)), e_s, fq, fk, fv, fg, ks, ds, sc, cs,
                              full[:3], full[3:])
    worst = [float((np.abs(_f64(x) - r) / b).max()) for x, r, b in zip((dq, dk, dv), full[:3],
                                                                         bound)]
    _log(f"{tag}: {ext} k={ks} d={ds} c={cs} D={D} {dtype} B={B} H={H}: "
         f"max err o/lse = {[f'{x:.3g}' for x in ef]}, dq/dk/dv = {[f'{x:.3g}' for x in eb]} "
         f"(/ bound {[f'{x:.3g}' for x in worst]}, max |ref| "
         f"{[f'{float(np.abs(r).max()):.3g}' for r in full[:3]]})")
    assert max(ef) <= TOL[dtype]
    assert max(worst) <= 1.0


# Case counts of the two random families; a longer sweep raises them, e.g.
# NA_TEST_RANDOM_PROBLEMS=600 NA_TEST_MID_PROBLEMS=200 pytest -m gpu -k random_problems
N_RANDOM = int(os.environ.get("NA_TEST_RANDOM_PROBLEMS", "24"))
N_MID = int(os.environ.get("NA_TEST_MID_PROBLEMS", "12"))


@pytest.mark.parametrize("case", range(N_RANDOM))
def test_random_problems_match_the_oracle(na, case):
    _check_random_problem(na, f"random {case}", _random_problems(N_RANDOM, 2026)[case], 90 + case)


@pytest.mark.parametrize("split", [0, 1])
@pytest.mark.parametrize("case", range(N_MID))
def test_mid_size_random_problems_match_the_oracle(na, force, case, split):
    """Larger halos than the small random problems, under both backward forms."""
    force(NA_BWD_SPLIT=split)
    _check_random_problem(na, f"mid {case} split={split}", _mid_problems(N_MID, 4243)[case],
                          300 + case)
