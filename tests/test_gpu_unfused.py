"""GPU parity of the unfused NA operators (na_unfused_* in include/na.h) against the oracle.

The unfused baseline computes NA as separate launches that store the l-wide attention weights
(PN, softmax, NN; softmax backward, NN and IN for the gradients, Sec. 3.1).  Checked through the
C ABI:
  * PN writes each query's scores in the documented layout: at non-causal problems entry e of
    row i is scale * q_i . k_j for the e-th neighbour j of the oracle's list (row-major over the
    per-axis windows); with causal axes the finite entries are exactly the oracle's neighbours;
  * the softmax rows sum to 1 and its logsumexp and the forward output match the oracle;
  * the backward (dQ, dK, dV) matches the oracle's;
  * the full-size workloads are compared in test_gpu_parity.py (shared oracle results).
Bar: 2e-2 max-abs for fp16/bf16, 1e-4 for fp32.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads

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


def _inputs(shape, dtype, seed, n=4):
    gen = torch.Generator().manual_seed(seed)
    return [torch.randn(shape, generator=gen).to(TDT[dtype]) for _ in range(n)]


def _f64(t):
    return t.detach().cpu().double().numpy()


def _maxerr(gpu, ref):
    return float(np.max(np.abs(_f64(gpu) - ref))) if ref.size else 0.0


def _log(msg):
    print(msg, flush=True)


CASES = [
    # (extents, kernel, dilation, causal, head_dim, dtype, batch, heads)
    ((200,), (7,), (1,), None, 32, "fp32", 1, 2),
    ((300,), (13,), (3,), None, 64, "fp16", 2, 2),
    ((257,), (64,), (4,), None, 128, "bf16", 1, 2),
    ((37, 45), (7, 5), (2, 1), None, 32, "fp16", 1, 2),
    ((20, 23), (3, 3), (3, 2), None, 64, "bf16", 1, 3),
    ((16, 16), (16, 16), (1, 1), None, 64, "fp32", 1, 1),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), None, 64, "fp16", 1, 2),
    ((5, 9, 11), (5, 3, 3), (1, 3, 3), None, 32, "fp32", 2, 1),
    ((8, 12, 12), (7, 7, 7), (1, 1, 1), None, 128, "bf16", 1, 1),
    ((300,), (13,), (3,), (True,), 64, "fp16", 1, 2),
    ((37, 45), (7, 5), (2, 1), (True, False), 32, "bf16", 1, 2),
    ((6, 20, 22), (3, 7, 5), (1, 2, 2), (True, False, False), 64, "fp16", 1, 1),
    ((5, 9, 11), (5, 3, 3), (1, 3, 3), (True, True, True), 32, "fp32", 1, 1),
]


@pytest.mark.parametrize("ext,ks,ds,cs,D,dtype,B,H", CASES)
def test_unfused_pn_writes_the_neighbour_scores(na, ext, ks, ds, cs, D, dtype, B, H):
    shape = (B, H) + ext + (D,)
    q, k = _inputs(shape, dtype, 51, 2)
    sc = 1.0 / math.sqrt(D)
    w = na.unfused_pn(q.cuda(), k.cuda(), ks, ds, sc, causal=cs)
    got = _f64(w).reshape(B * H, -1, w.shape[-1])
    nb = oracle.neighbors(ext, ks, ds, causal=cs)
    qf, kf = _f64(q).reshape(B * H, -1, D), _f64(k).reshape(B * H, -1, D)
    worst = 0.0
    for s in range(B * H):
        for i in range(nb.shape[0]):
            js = nb[i][nb[i] >= 0]
            want = sc * kf[s, js] @ qf[s, i]
            row = got[s, i]
            if cs is None:
                worst = max(worst, float(np.max(np.abs(row - want))))
            else:
                fin = row[np.isfinite(row)]
                assert fin.size == js.size and np.all(row[~np.isfinite(row)] == -np.inf)
                worst = max(worst, float(np.max(np.abs(np.sort(fin) - np.sort(want)))))
    _log(f"unfused PN {ext} k={ks} d={ds} c={cs} D={D} {dtype}: max err {worst:.3g}")
    # the scores are stored in the inputs' type: their own rounding is relative to |score|
    u = {"fp32": 2.0 ** -24, "fp16": 2.0 ** -11, "bf16": 2.0 ** -8}[dtype]
    bound = TOL[dtype] + u * float(np.max(np.abs(got[np.isfinite(got)])))
    assert worst <= bound


@pytest.mark.parametrize("ext,ks,ds,cs,D,dtype,B,H", CASES)
def test_unfused_forward_and_backward_match_the_oracle(na, ext, ks, ds, cs, D, dtype, B, H):
    shape = (B, H) + ext + (D,)
    q, k, v, g = _inputs(shape, dtype, 52, 4)
    qd, kd, vd, gd = (t.cuda() for t in (q, k, v, g))
    sc = 1.0 / math.sqrt(D)
    out, lse, p = na.unfused_forward(qd, kd, vd, ks, ds, sc, causal=cs)
    dq, dk, dv = na.unfused_backward(qd, kd, vd, p, gd, ks, ds, sc, causal=cs)
    torch.cuda.synchronize()
    sums = p.double().sum(-1)
    ro, rl = oracle.forward(_f64(q), _f64(k), _f64(v), ks, ds, sc, causal=cs)
    rq, rk, rv = oracle.backward(_f64(q), _f64(k), _f64(v), _f64(g), ks, ds, sc, causal=cs)
    e = [_maxerr(out, ro), _maxerr(lse, rl), _maxerr(dq, rq), _maxerr(dk, rk), _maxerr(dv, rv)]
    es = float((sums - 1.0).abs().max())
    _log(f"unfused {ext} k={ks} d={ds} c={cs} D={D} {dtype}: max err o/lse/dq/dk/dv = "
         f"{[f'{x:.3g}' for x in e]}, max |row sum - 1| = {es:.3g}")
    # each stored probability carries one rounding to the type (relative u), the row sum
    # fp32 additions
    u = {"fp32": 2.0 ** -24, "fp16": 2.0 ** -11, "bf16": 2.0 ** -8}[dtype]
    assert es <= u + p.shape[-1] * 2.0 ** -23
    assert max(e) <= TOL[dtype]


def test_unfused_operators_reject_bad_arguments(na):
    q = torch.zeros((1, 1, 20, 32), dtype=torch.float16, device="cuda")
    with pytest.raises(ValueError):
        na.unfused_pn(q, q, (5,), 1, 1.0, weights=torch.empty((1, 1, 20, 4), dtype=q.dtype,
                                                               device="cuda"))
    with pytest.raises(na.NAError):
        na.unfused_pn(q, q, (7,), (3,), 1.0)  # 7 * 3 > 20
    w = na.unfused_pn(q, q, (5,), 1, 1.0)
    lib = na.load_library()
    import ctypes
    rank, ext, ks, ds, cs = na._problem_arrays((20,), (5,), 1)
    st = lib.na_unfused_nn(rank, ext, ks, ds, cs, 1, 1, 32, 1, 1.0, w.data_ptr(), None,
                           q.data_ptr(), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 1  # NA_ERR_NULL
    st = lib.na_unfused_in(rank, ext, ks, ds, cs, 1, 1, 32, 1, 1.0, w.data_ptr() + 2,
                           q.data_ptr(), q.data_ptr(), None)
    assert st == 9  # NA_ERR_ALIGNMENT
