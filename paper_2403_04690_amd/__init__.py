"""Fused neighborhood attention for MI355X (gfx950): Python binding of libna.so.

Every computation runs in the HIP kernels of ``libna.so``; this module only
checks tensor arguments and passes device pointers, sizes and the current
stream through the C ABI declared in ``include/na.h``.  PyTorch supplies
device memory and streams.  If the library is missing, every call raises.

Neighborhood attention (Faster Neighborhood Attention, arXiv 2403.04690):
each query attends to its k_a nearest same-group tokens along every axis a
(window centred where possible, shifted at borders, never truncated), with
dilation d_a splitting each axis into d_a interleaved sub-lattices.  Axes can
be causal (``causal``, one flag per axis): there a query attends only to the
k nearest positions not after it.
"""
import ctypes
import functools
import math
import os

import torch

__all__ = ["NAError", "forward", "backward", "na_attention", "debug_windows", "validate",
           "library_path", "load_library", "DTYPES", "Tiling", "candidate_tilings",
           "current_tiling", "tune", "tune_clear", "set_autotune", "autotune", "unfused_pn",
           "unfused_softmax", "unfused_nn", "unfused_in", "unfused_softmax_backward",
           "unfused_forward", "unfused_backward"]

_PKG = os.path.dirname(os.path.abspath(__file__))
# NA_LIBRARY may point at another build of the same library (A/B comparisons
# of kernel variants); by default the in-tree build is used.
_LIB_PATH = os.environ.get("NA_LIBRARY") or os.path.join(_PKG, "libna.so")
_lib = None
# the optional argument-marshalling extension (csrc/na_pyext.c) and the addresses of the
# two functions it calls; without it the calls go through ctypes
_fast = None
_fast_fn = {}

DTYPES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}

_i64p = ctypes.POINTER(ctypes.c_int64)
_i32p = ctypes.POINTER(ctypes.c_int32)
_vp = ctypes.c_void_p


class _NaTiling(ctypes.Structure):
    _fields_ = [("blocks_per_wave", ctypes.c_int32), ("wave_tile", ctypes.c_int32 * 3),
                ("waves", ctypes.c_int32 * 3)]


class Tiling(tuple):
    """(blocks_per_wave, wave_tile[3], waves[3]) of a launch (na_tiling in na.h)."""

    def __new__(cls, blocks_per_wave, wave_tile, waves):
        return super().__new__(cls, (int(blocks_per_wave), tuple(int(x) for x in wave_tile),
                                     tuple(int(x) for x in waves)))

    blocks_per_wave = property(lambda self: self[0])
    wave_tile = property(lambda self: self[1])
    waves = property(lambda self: self[2])

    def _c(self):
        return _NaTiling(self[0], (ctypes.c_int32 * 3)(*self[1]), (ctypes.c_int32 * 3)(*self[2]))

    @staticmethod
    def _from_c(t):
        return Tiling(t.blocks_per_wave, tuple(t.wave_tile), tuple(t.waves))


class NAError(RuntimeError):
    """A non-OK status returned by libna.so."""

    def __init__(self, status, text):
        super().__init__(f"libna: {text} (status {status})")
        self.status = status


def library_path():
    return _LIB_PATH


def load_library():
    """Load libna.so (built by paper_2403_04690_amd/build.py); raise if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"libna.so not found at {_LIB_PATH}: build it first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(_LIB_PATH)
    prob = [ctypes.c_int, _i64p, _i32p, _i32p, _i32p, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_int, ctypes.c_float]
    lib.na_status_string.argtypes = [ctypes.c_int]
    lib.na_status_string.restype = ctypes.c_char_p
    lib.na_version.restype = ctypes.c_int
    lib.na_validate.argtypes = prob
    lib.na_validate.restype = ctypes.c_int
    lib.na_forward.argtypes = prob + [_vp] * 6
    lib.na_forward.restype = ctypes.c_int
    lib.na_backward.argtypes = prob + [_vp] * 10
    lib.na_backward.restype = ctypes.c_int
    lib.na_debug_windows.argtypes = [ctypes.c_int, _i64p, _i32p, _i32p, _i32p, _vp, _vp, _vp, _vp]
    lib.na_debug_windows.restype = ctypes.c_int
    tp = ctypes.POINTER(_NaTiling)
    lib.na_candidate_tilings.argtypes = [ctypes.c_int, _i64p, _i32p, _i32p, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                         ctypes.c_int, tp, ctypes.c_int]
    lib.na_candidate_tilings.restype = ctypes.c_int
    lib.na_current_tiling.argtypes = prob[:-1] + [ctypes.c_int, tp]
    lib.na_current_tiling.restype = ctypes.c_int
    lib.na_forward_tiled.argtypes = prob + [tp] + [_vp] * 6
    lib.na_forward_tiled.restype = ctypes.c_int
    lib.na_backward_tiled.argtypes = prob + [tp] + [_vp] * 10
    lib.na_backward_tiled.restype = ctypes.c_int
    lib.na_tune.argtypes = prob + [_vp] * 9 + [ctypes.c_int, ctypes.c_int, _vp, tp, tp,
                                               ctypes.POINTER(ctypes.c_float)]
    lib.na_tune.restype = ctypes.c_int
    lib.na_tune_clear.argtypes = []
    lib.na_tune_clear.restype = None
    lib.na_set_autotune.argtypes = [ctypes.c_int]
    lib.na_set_autotune.restype = None
    lib.na_autotune.argtypes = []
    lib.na_autotune.restype = ctypes.c_int
    for name in ("na_unfused_pn", "na_unfused_nn", "na_unfused_in"):
        getattr(lib, name).argtypes = prob + [_vp] * 4
        getattr(lib, name).restype = ctypes.c_int
    for name in ("na_unfused_softmax", "na_unfused_softmax_backward"):
        getattr(lib, name).argtypes = prob[:-1] + [_vp] * 3
        getattr(lib, name).restype = ctypes.c_int
    _load_fast(lib)
    _lib = lib
    return lib


def _load_fast(lib):
    """Use _na_fast (built beside libna.so) for na_forward / na_backward when it is there."""
    global _fast
    try:
        from . import _na_fast
    except ImportError:
        _fast = None
        return
    _fast_fn["fwd"] = ctypes.cast(lib.na_forward, ctypes.c_void_p).value
    _fast_fn["bwd"] = ctypes.cast(lib.na_backward, ctypes.c_void_p).value
    _fast_fn["lib"] = lib
    _fast = _na_fast


def _fast_for(lib):
    """The function addresses for `lib` (re-read when another build has been swapped in)."""
    if _fast_fn.get("lib") is not lib:
        _load_fast(lib)
    return _fast_fn


def _check(status):
    if status != 0:
        text = load_library().na_status_string(status).decode()
        raise NAError(status, text)


def _per_axis(value, rank, name):
    vals = list(value) if isinstance(value, (list, tuple)) else [int(value)] * rank
    if len(vals) != rank:
        raise ValueError(f"{name} needs {rank} entries, got {len(vals)}")
    return vals


@functools.lru_cache(maxsize=256)
def _problem_arrays_of(extents, kernel_size, dilation, causal):
    """(rank, extents, kernel_size, dilation, causal-or-None as ctypes arrays, and their
    addresses); the tuple keeps the arrays alive while a caller uses the addresses."""
    rank = len(extents)
    ext = (ctypes.c_int64 * rank)(*[int(e) for e in extents])
    ks = (ctypes.c_int32 * rank)(*_per_axis(kernel_size, rank, "kernel_size"))
    ds = (ctypes.c_int32 * rank)(*_per_axis(dilation, rank, "dilation"))
    cs = None if causal is None else (ctypes.c_int32 * rank)(
        *[int(bool(c)) for c in _per_axis(causal, rank, "causal")])
    addrs = (ctypes.addressof(ext), ctypes.addressof(ks), ctypes.addressof(ds),
             0 if cs is None else ctypes.addressof(cs))
    return rank, ext, ks, ds, cs, addrs


def _hashable(value):
    return tuple(value) if isinstance(value, (list, tuple)) else value


def _problem(extents, kernel_size, dilation, causal=None):
    return _problem_arrays_of(tuple(extents), _hashable(kernel_size), _hashable(dilation),
                              None if causal is None else _hashable(causal))


def _problem_arrays(extents, kernel_size, dilation, causal=None):
    """The problem as ctypes arrays (read only by the library; cached per problem)."""
    return _problem(extents, kernel_size, dilation, causal)[:5]


# the current stream's handle without building a Stream object (where torch has it)
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(device):
    if _raw_stream is not None:
        return _raw_stream(device.index)
    return torch.cuda.current_stream(device).cuda_stream


def _check_tensors(ref, *others):
    if ref.dim() < 4:
        raise ValueError("expected [batch, heads, X_1..X_r, head_dim] with 1 <= r <= 3")
    if ref.dtype not in DTYPES:
        raise TypeError(f"unsupported dtype {ref.dtype}")
    for t in (ref,) + others:
        if not t.is_cuda:
            raise ValueError("tensors must live on a GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    for t in others:
        if t.dtype != ref.dtype or t.shape != ref.shape or t.device != ref.device:
            raise ValueError("q, k, v (and grads) must share dtype, shape and device")


def validate(extents, kernel_size, dilation, batch, heads, head_dim, dtype, scale, causal=None):
    """Host-only validation through na_validate; raises NAError on a bad problem."""
    lib = load_library()
    rank, ext, ks, ds, cs = _problem_arrays(extents, kernel_size, dilation, causal)
    _check(lib.na_validate(rank, ext, ks, ds, cs, batch, heads, head_dim, DTYPES[dtype], scale))


def candidate_tilings(extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                      forward=True):
    """Every candidate tiling (the heuristic one first), host only; na_tune times the first
    NA_TUNE_DEFAULT_CANDIDATES (64) of them, or all when thorough."""
    lib = load_library()
    rank, ext, ks, ds, _ = _problem_arrays(extents, kernel_size, dilation)
    n = lib.na_candidate_tilings(rank, ext, ks, ds, batch, heads, head_dim, DTYPES[dtype],
                                 int(bool(forward)), None, 0)
    if n < 0:
        _check(-n)
    buf = (_NaTiling * max(n, 1))()
    lib.na_candidate_tilings(rank, ext, ks, ds, batch, heads, head_dim, DTYPES[dtype],
                             int(bool(forward)), buf, n)
    return [Tiling._from_c(buf[i]) for i in range(n)]


def current_tiling(extents, kernel_size, dilation, batch, heads, head_dim, dtype, forward=True,
                   causal=None):
    """The tiling na_forward (or na_backward) uses now for this problem, host only."""
    lib = load_library()
    rank, ext, ks, ds, cs = _problem_arrays(extents, kernel_size, dilation, causal)
    t = _NaTiling()
    _check(lib.na_current_tiling(rank, ext, ks, ds, cs, batch, heads, head_dim, DTYPES[dtype],
                                 int(bool(forward)), ctypes.byref(t)))
    return Tiling._from_c(t)


def tune(q, k, v, dout, kernel_size, dilation=1, scale=None, causal=None, repeats=5,
         out=None, lse=None, dq=None, dk=None, dv=None, thorough=False):
    """Auto-tune the tilings of this problem (na_tune): times the candidate forward and
    backward tilings (the first 64, or all with thorough=True), caches the fastest for later
    calls and returns (best_forward, best_backward, times_ms) with times_ms = [best fwd,
    best bwd, heuristic fwd, heuristic bwd].  Synchronises the current stream."""
    lib = load_library()
    _check_tensors(q, k, v, dout)
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    rank, ext, ks, ds, cs = _problem_arrays(tuple(q.shape[2:-1]), kernel_size, dilation, causal)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(q.shape[:-1], dtype=torch.float32, device=q.device) if lse is None else lse
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    _check_tensors(q, out, dq, dk, dv)
    bf, bb = _NaTiling(), _NaTiling()
    times = (ctypes.c_float * 4)()
    _check(lib.na_tune(rank, ext, ks, ds, cs, B, H, D, DTYPES[q.dtype], float(scale),
                       q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                       dout.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                       int(repeats), 1 if thorough else 0, _stream(q.device), ctypes.byref(bf),
                       ctypes.byref(bb), times))
    return Tiling._from_c(bf), Tiling._from_c(bb), list(times)


def tune_clear():
    """Forget every tiling na_tune recorded."""
    load_library().na_tune_clear()


def set_autotune(mode):
    """Tune on first use (na_set_autotune): 1 makes forward/backward tune a problem whose
    tiling is not cached yet on the call's own buffers (3 launches per candidate), 2 does so
    over every candidate, 0 turns it off."""
    load_library().na_set_autotune(int(mode))


def autotune():
    """The tune-on-first-use mode in force (0, 1 or 2)."""
    return int(load_library().na_autotune())


def forward(q, k, v, kernel_size, dilation=1, scale=None, out=None, lse=None, causal=None,
            tiling=None):
    """Fused NA forward.  Returns (out, logsumexp); logsumexp is fp32 [B, H, X..].
    tiling: an explicit Tiling (na_forward_tiled); None uses the cached or heuristic one."""
    lib = load_library()
    _check_tensors(q, k, v)
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    extents = tuple(q.shape[2:-1])
    prob = _problem(extents, kernel_size, dilation, causal)
    rank, ext, ks, ds, cs, addrs = prob
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty(q.shape[:-1], dtype=torch.float32, device=q.device)
    _check_tensors(q, out)
    if lse.dtype != torch.float32 or lse.shape != q.shape[:-1] or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous fp32 tensor of shape q.shape[:-1]")
    args = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
            _stream(q.device))
    if tiling is None and _fast is not None:
        _check(_fast.forward(_fast_for(lib)["fwd"], rank, *addrs, B, H, D, DTYPES[q.dtype],
                             float(scale), *args))
    elif tiling is None:
        _check(lib.na_forward(rank, ext, ks, ds, cs, B, H, D, DTYPES[q.dtype], float(scale), *args))
    else:
        _check(lib.na_forward_tiled(rank, ext, ks, ds, cs, B, H, D, DTYPES[q.dtype], float(scale),
                                    ctypes.byref(Tiling(*tiling)._c()), *args))
    return out, lse


def backward(q, k, v, out, lse, dout, kernel_size, dilation=1, scale=None, dq=None, dk=None,
             dv=None, causal=None, tiling=None):
    """Fused NA backward.  Returns (dq, dk, dv).
    tiling: an explicit Tiling (na_backward_tiled); None uses the cached or heuristic one."""
    lib = load_library()
    _check_tensors(q, k, v, out, dout)
    B, H, D = q.shape[0], q.shape[1], q.shape[-1]
    extents = tuple(q.shape[2:-1])
    prob = _problem(extents, kernel_size, dilation, causal)
    rank, ext, ks, ds, cs, addrs = prob
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if lse.dtype != torch.float32 or lse.shape != q.shape[:-1] or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous fp32 tensor of shape q.shape[:-1]")
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    _check_tensors(q, dq, dk, dv)
    args = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
            dout.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), _stream(q.device))
    if tiling is None and _fast is not None:
        _check(_fast.backward(_fast_for(lib)["bwd"], rank, *addrs, B, H, D, DTYPES[q.dtype],
                              float(scale), *args))
    elif tiling is None:
        _check(lib.na_backward(rank, ext, ks, ds, cs, B, H, D, DTYPES[q.dtype], float(scale),
                               *args))
    else:
        _check(lib.na_backward_tiled(rank, ext, ks, ds, cs, B, H, D, DTYPES[q.dtype],
                                     float(scale), ctypes.byref(Tiling(*tiling)._c()), *args))
    return dq, dk, dv


def debug_windows(extents, kernel_size, dilation, device="cuda", causal=None):
    """Per-axis window starts and inverse ranges computed on the device (int32, concatenated)."""
    lib = load_library()
    rank, ext, ks, ds, cs = _problem_arrays(extents, kernel_size, dilation, causal)
    total = int(sum(extents))
    start = torch.empty(total, dtype=torch.int32, device=device)
    ilo = torch.empty_like(start)
    ihi = torch.empty_like(start)
    _check(lib.na_debug_windows(rank, ext, ks, ds, cs, start.data_ptr(), ilo.data_ptr(),
                                ihi.data_ptr(), _stream(start.device)))
    return start, ilo, ihi


class _NAFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, kernel_size, dilation, scale, causal):
        out, lse = forward(q, k, v, kernel_size, dilation, scale, causal=causal)
        ctx.save_for_backward(q, k, v, out, lse)
        ctx.cfg = (kernel_size, dilation, scale, causal)
        return out

    @staticmethod
    def backward(ctx, dout):
        q, k, v, out, lse = ctx.saved_tensors
        kernel_size, dilation, scale, causal = ctx.cfg
        dq, dk, dv = backward(q, k, v, out, lse, dout.contiguous(), kernel_size, dilation, scale,
                              causal=causal)
        return dq, dk, dv, None, None, None, None


def na_attention(q, k, v, kernel_size, dilation=1, scale=None, causal=None):
    """Autograd-aware fused neighborhood attention on [B, H, X_1..X_r, D] tensors."""
    return _NAFunction.apply(q, k, v, kernel_size, dilation, scale, causal)


# ---------------------------------------------------------------- unfused operators
# The baseline of separate PN / softmax / NN / IN launches (na_unfused_* in na.h) that
# read and write the l-wide attention weights [B, H, X.., l] in global memory.

def _window(kernel_size, rank):
    return int(math.prod(_per_axis(kernel_size, rank, "kernel_size")))


def _weights_like(x, kernel_size):
    return torch.empty(tuple(x.shape[:-1]) + (_window(kernel_size, x.dim() - 3),), dtype=x.dtype,
                       device=x.device)


def _check_weights(w, ref, kernel_size):
    want = tuple(ref.shape[:-1]) + (_window(kernel_size, ref.dim() - 3),)
    if tuple(w.shape) != want or w.dtype != ref.dtype or not w.is_contiguous() or not w.is_cuda:
        raise ValueError(f"weights must be a contiguous {ref.dtype} GPU tensor of shape {want}")


def _uargs(ref, kernel_size, dilation, causal):
    B, H, D = ref.shape[0], ref.shape[1], ref.shape[-1]
    rank, ext, ks, ds, cs = _problem_arrays(tuple(ref.shape[2:-1]), kernel_size, dilation, causal)
    return (rank, ext, ks, ds, cs, B, H, D, DTYPES[ref.dtype])


def unfused_pn(a, b, kernel_size, dilation=1, scale=1.0, causal=None, weights=None):
    """PN: weights[i, e] = scale * a_i . b_j(i,e) (-inf where e is not a neighbour)."""
    lib = load_library()
    _check_tensors(a, b)
    w = _weights_like(a, kernel_size) if weights is None else weights
    _check_weights(w, a, kernel_size)
    _check(lib.na_unfused_pn(*_uargs(a, kernel_size, dilation, causal), float(scale),
                             a.data_ptr(), b.data_ptr(), w.data_ptr(), _stream(a.device)))
    return w


def unfused_softmax(weights, head_dim, kernel_size, dilation=1, causal=None, lse=None):
    """Row softmax of the weights in place; returns (probs, logsumexp [B, H, X..] fp32)."""
    lib = load_library()
    ref = torch.empty(tuple(weights.shape[:-1]) + (head_dim,), dtype=weights.dtype, device="meta")
    _check_weights(weights, ref, kernel_size)
    if lse is None:
        lse = torch.empty(weights.shape[:-1], dtype=torch.float32, device=weights.device)
    rank, ext, ks, ds, cs = _problem_arrays(tuple(weights.shape[2:-1]), kernel_size, dilation,
                                            causal)
    _check(lib.na_unfused_softmax(rank, ext, ks, ds, cs, weights.shape[0], weights.shape[1],
                                  head_dim, DTYPES[weights.dtype], weights.data_ptr(),
                                  lse.data_ptr(), _stream(weights.device)))
    return weights, lse


def unfused_nn(weights, b, kernel_size, dilation=1, scale=1.0, causal=None, out=None):
    """NN: out_i = scale * sum_e weights[i, e] b_j(i,e)."""
    lib = load_library()
    _check_tensors(b)
    _check_weights(weights, b, kernel_size)
    out = torch.empty_like(b) if out is None else out
    _check_tensors(b, out)
    _check(lib.na_unfused_nn(*_uargs(b, kernel_size, dilation, causal), float(scale),
                             weights.data_ptr(), b.data_ptr(), out.data_ptr(), _stream(b.device)))
    return out


def unfused_in(weights, b, kernel_size, dilation=1, scale=1.0, causal=None, out=None):
    """IN: out_j = scale * sum over the queries i whose window holds j of weights[i, e(i,j)] b_i."""
    lib = load_library()
    _check_tensors(b)
    _check_weights(weights, b, kernel_size)
    out = torch.empty_like(b) if out is None else out
    _check_tensors(b, out)
    _check(lib.na_unfused_in(*_uargs(b, kernel_size, dilation, causal), float(scale),
                             weights.data_ptr(), b.data_ptr(), out.data_ptr(), _stream(b.device)))
    return out


def unfused_softmax_backward(probs, grad, head_dim, kernel_size, dilation=1, causal=None):
    """In place on grad (dP in, dA out): dA = P * (dP - sum_e P dP) per row."""
    lib = load_library()
    if grad.shape != probs.shape or grad.dtype != probs.dtype or not grad.is_contiguous():
        raise ValueError("probs and grad must be contiguous tensors of one shape and dtype")
    rank, ext, ks, ds, cs = _problem_arrays(tuple(probs.shape[2:-1]), kernel_size, dilation,
                                            causal)
    if probs.shape[-1] != _window(kernel_size, rank):
        raise ValueError("the last axis of probs must hold prod(kernel_size) weights")
    _check(lib.na_unfused_softmax_backward(rank, ext, ks, ds, cs, probs.shape[0], probs.shape[1],
                                           head_dim, DTYPES[probs.dtype], probs.data_ptr(),
                                           grad.data_ptr(), _stream(probs.device)))
    return grad


def unfused_forward(q, k, v, kernel_size, dilation=1, scale=None, causal=None, weights=None):
    """Unfused NA forward: PN, softmax, NN as three launches.  Returns (out, lse, probs)."""
    D = q.shape[-1]
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    w = unfused_pn(q, k, kernel_size, dilation, scale, causal, weights)
    p, lse = unfused_softmax(w, D, kernel_size, dilation, causal)
    out = unfused_nn(p, v, kernel_size, dilation, 1.0, causal)
    return out, lse, p


def unfused_backward(q, k, v, probs, dout, kernel_size, dilation=1, scale=None, causal=None,
                     grad_weights=None):
    """Unfused NA backward from the forward's probabilities: PN, softmax backward, NN and two
    IN launches.  Returns (dq, dk, dv)."""
    D = q.shape[-1]
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    dp = unfused_pn(dout, v, kernel_size, dilation, 1.0, causal, grad_weights)
    da = unfused_softmax_backward(probs, dp, D, kernel_size, dilation, causal)
    dq = unfused_nn(da, k, kernel_size, dilation, scale, causal)
    dk = unfused_in(da, q, kernel_size, dilation, scale, causal)
    dv = unfused_in(probs, dout, kernel_size, dilation, 1.0, causal)
    return dq, dk, dv
