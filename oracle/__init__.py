"""Plain fp64 CPU oracle for neighborhood attention -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product path (the HIP library and its Python binding) never
imports, links or runs anything here, and this package never touches the
product: the two share no code.

The arithmetic lives in ``na_ref.c`` (built into ``libna_ref.so`` by
``oracle/build.py``); this module only marshals numpy arrays through ctypes.
Every function follows the plain definition of neighborhood attention
(Sec. 1-2 and Fig. "neighborhoodattention" of Faster Neighborhood Attention,
dilation as sub-lattice partitioning in Sec. 3.4, attention as in Eq. 1, the
backward as the PN/NN/IN operators of Sec. 3.1).  ``causal`` (optional, one
flag per axis) marks axes along which a query never attends to tokens of
larger coordinate (causal masking, Sec. 3.4): its window there is the k
nearest same-group positions not after it, [max(0, p - k + 1), p].
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# NA_REF_LIBRARY selects another build of the same source (the sanitizer build)
_LIB_PATH = os.environ.get("NA_REF_LIBRARY") or os.path.join(_HERE, "libna_ref.so")
_lib = None

_STATUS = {
    0: "ok",
    2: "rank must be 1, 2 or 3",
    3: "every extent must be >= 1",
    4: "kernel size must be >= 1 (and <= 4096 in the oracle)",
    5: "dilation must be >= 1",
    6: "kernel_size * dilation exceeds the extent",
    13: "allocation failed",
}

_i64p = ctypes.POINTER(ctypes.c_int64)
_i32p = ctypes.POINTER(ctypes.c_int32)
_f64p = ctypes.POINTER(ctypes.c_double)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.na_ref_num_threads.restype = ctypes.c_int
    lib.na_ref_set_num_threads.argtypes = [ctypes.c_int]
    lib.na_ref_set_num_threads.restype = None
    lib.na_ref_neighbors.argtypes = [ctypes.c_int, _i64p, _i32p, _i32p, _i32p, _i64p]
    lib.na_ref_axis_relation.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32, _i64p, _i64p, _i64p, _i64p]
    prob = [ctypes.c_int, _i64p, _i32p, _i32p, _i32p, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_double]
    lib.na_ref_forward.argtypes = prob + [_f64p] * 5
    lib.na_ref_forward_rows.argtypes = prob + [_f64p] * 3 + [ctypes.c_int64, _i64p, _f64p, _f64p]
    lib.na_ref_backward.argtypes = prob + [_f64p] * 7
    lib.na_ref_backward_given.argtypes = prob + [_f64p] * 12
    lib.na_ref_backward_rows.argtypes = prob + [_f64p] * 4 + [
        ctypes.c_int64, _i64p, _f64p, ctypes.c_int64, _i64p, _f64p, _f64p]
    for name in ("na_ref_neighbors", "na_ref_axis_relation", "na_ref_forward",
                 "na_ref_forward_rows", "na_ref_backward", "na_ref_backward_given",
                 "na_ref_backward_rows"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status):
    if status != 0:
        raise ValueError("oracle: " + _STATUS.get(status, "status %d" % status))


def _ptr(a, t):
    return a.ctypes.data_as(t)


def _problem(extents, kernel_size, dilation, causal=None):
    rank = len(extents)
    ks = list(kernel_size) if hasattr(kernel_size, "__len__") else [kernel_size] * rank
    ds = list(dilation) if hasattr(dilation, "__len__") else [dilation] * rank
    cs = [0] * rank if causal is None else (
        [int(bool(c)) for c in causal] if hasattr(causal, "__len__") else [int(bool(causal))] * rank)
    if len(ks) != rank or len(ds) != rank or len(cs) != rank:
        raise ValueError("oracle: kernel_size, dilation and causal need one entry per axis")
    L = np.ascontiguousarray(extents, dtype=np.int64)
    K = np.ascontiguousarray(ks, dtype=np.int32)
    Dl = np.ascontiguousarray(ds, dtype=np.int32)
    C = np.ascontiguousarray(cs, dtype=np.int32)
    return rank, L, K, Dl, C


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def num_threads():
    return int(_load().na_ref_num_threads())


def set_num_threads(n):
    """Threads used by later calls (the results do not depend on it)."""
    _load().na_ref_set_num_threads(int(n))


def neighbors(extents, kernel_size, dilation, causal=None):
    """Explicit neighbour lists: int64 [N, prod k], flat token indices, rows padded with -1
    (only causal axes make a neighbourhood smaller than prod k)."""
    lib = _load()
    rank, L, K, Dl, C = _problem(extents, kernel_size, dilation, causal)
    N = int(np.prod(L))
    ell = int(np.prod(K))
    idx = np.zeros((N, ell), dtype=np.int64)
    _check(lib.na_ref_neighbors(rank, _ptr(L, _i64p), _ptr(K, _i32p), _ptr(Dl, _i32p),
                                _ptr(C, _i32p), _ptr(idx, _i64p)))
    return idx


def axis_relation(length, kernel_size, dilation, causal=False):
    """Per-axis brute-force summary: (first, inv_lo, inv_hi, inv_count), each int64 [length]."""
    lib = _load()
    out = [np.zeros(length, dtype=np.int64) for _ in range(4)]
    _check(lib.na_ref_axis_relation(int(length), int(kernel_size), int(dilation), int(bool(causal)),
                                    *[_ptr(o, _i64p) for o in out]))
    return tuple(out)


def forward(q, k, v, kernel_size, dilation, scale, causal=None):
    """q, k, v: [B, H, X_1..X_r, D] arrays.  Returns (out [B,H,X..,D], lse [B,H,X..]) in fp64."""
    lib = _load()
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    extents = q.shape[2:-1]
    rank, L, K, Dl, C = _problem(extents, kernel_size, dilation, causal)
    out = np.zeros_like(q)
    lse = np.zeros(q.shape[:-1], dtype=np.float64)
    _check(lib.na_ref_forward(rank, _ptr(L, _i64p), _ptr(K, _i32p), _ptr(Dl, _i32p),
                              _ptr(C, _i32p), B, H, D, float(scale), _ptr(q, _f64p), _ptr(k, _f64p), _ptr(v, _f64p),
                              _ptr(out, _f64p), _ptr(lse, _f64p)))
    return out, lse


def forward_rows(q, k, v, kernel_size, dilation, scale, rows, causal=None):
    """Forward for selected flat query rows (indices into [B*H*N]).  Returns (out [n, D], lse [n])."""
    lib = _load()
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    rank, L, K, Dl, C = _problem(q.shape[2:-1], kernel_size, dilation, causal)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, D), dtype=np.float64)
    lse = np.zeros(rows.size, dtype=np.float64)
    _check(lib.na_ref_forward_rows(rank, _ptr(L, _i64p), _ptr(K, _i32p), _ptr(Dl, _i32p),
                                   _ptr(C, _i32p), B, H, D, float(scale), _ptr(q, _f64p), _ptr(k, _f64p), _ptr(v, _f64p),
                                   rows.size, _ptr(rows, _i64p), _ptr(out, _f64p),
                                   _ptr(lse, _f64p)))
    return out, lse


def backward(q, k, v, dout, kernel_size, dilation, scale, causal=None):
    """Returns (dq, dk, dv) in fp64, each shaped like q."""
    lib = _load()
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    rank, L, K, Dl, C = _problem(q.shape[2:-1], kernel_size, dilation, causal)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(q), np.zeros_like(q)
    _check(lib.na_ref_backward(rank, _ptr(L, _i64p), _ptr(K, _i32p), _ptr(Dl, _i32p),
                               _ptr(C, _i32p), B, H, D, float(scale), _ptr(q, _f64p), _ptr(k, _f64p), _ptr(v, _f64p),
                               _ptr(dout, _f64p), _ptr(dq, _f64p), _ptr(dk, _f64p),
                               _ptr(dv, _f64p)))
    return dq, dk, dv


def backward_given(q, k, v, out, lse, dout, kernel_size, dilation, scale, causal=None,
                   abs_sums=False):
    """The backward operator from stored forward results: P rebuilt from ``lse``, Delta from
    ``out`` (as the library's na_backward takes them).  Returns (dq, dk, dv) in fp64, and with
    ``abs_sums`` also (dq_abs, dk_abs, dv_abs): the same sums over absolute values of their
    terms, the magnitude a rounding of the terms is relative to."""
    lib = _load()
    q, k, v, out, lse, dout = (_f64(a) for a in (q, k, v, out, lse, dout))
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    rank, L, K, Dl, C = _problem(q.shape[2:-1], kernel_size, dilation, causal)
    if out.shape != q.shape or dout.shape != q.shape or lse.shape != q.shape[:-1]:
        raise ValueError("oracle: out and dout must be shaped like q, lse like q[..., 0]")
    res = [np.zeros_like(q) for _ in range(6 if abs_sums else 3)]
    ptrs = [_ptr(r, _f64p) for r in res] + ([None] * 3 if not abs_sums else [])
    _check(lib.na_ref_backward_given(rank, _ptr(L, _i64p), _ptr(K, _i32p), _ptr(Dl, _i32p),
                                     _ptr(C, _i32p), B, H, D, float(scale), _ptr(q, _f64p),
                                     _ptr(k, _f64p), _ptr(v, _f64p), _ptr(out, _f64p),
                                     _ptr(lse, _f64p), _ptr(dout, _f64p), *ptrs))
    return tuple(res)


def backward_rows(q, k, v, dout, kernel_size, dilation, scale, qrows, krows, causal=None):
    """dQ at selected flat query rows and dK, dV at selected flat key rows."""
    lib = _load()
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    rank, L, K, Dl, C = _problem(q.shape[2:-1], kernel_size, dilation, causal)
    qrows = np.ascontiguousarray(qrows, dtype=np.int64)
    krows = np.ascontiguousarray(krows, dtype=np.int64)
    dq = np.zeros((qrows.size, D), dtype=np.float64)
    dk = np.zeros((krows.size, D), dtype=np.float64)
    dv = np.zeros((krows.size, D), dtype=np.float64)
    _check(lib.na_ref_backward_rows(rank, _ptr(L, _i64p), _ptr(K, _i32p), _ptr(Dl, _i32p), _ptr(C, _i32p),
                                    B, H, D, float(scale), _ptr(q, _f64p), _ptr(k, _f64p),
                                    _ptr(v, _f64p), _ptr(dout, _f64p), qrows.size,
                                    _ptr(qrows, _i64p), _ptr(dq, _f64p), krows.size,
                                    _ptr(krows, _i64p), _ptr(dk, _f64p), _ptr(dv, _f64p)))
    return dq, dk, dv
