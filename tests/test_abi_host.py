"""Host-side checks of the C ABI (no GPU needed, no kernel launched).

  * libna.so loads and exports every function include/na.h declares;
  * na_validate and the entry points return each documented error status
    before touching the device (bad rank, extents, window, dilation, head
    dim, dtype, scale, NULL or misaligned pointers);
  * an empty batch or head count is a no-op that returns NA_OK.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "na.h")

NA_OK, NA_ERR_NULL, NA_ERR_RANK, NA_ERR_SHAPE = 0, 1, 2, 3
NA_ERR_KERNEL_SIZE, NA_ERR_DILATION, NA_ERR_WINDOW, NA_ERR_HEAD_DIM = 4, 5, 6, 7
NA_ERR_DTYPE, NA_ERR_ALIGNMENT, NA_ERR_HIP, NA_ERR_SCALE = 8, 9, 11, 12


@pytest.fixture(scope="module")
def lib():
    import paper_2403_04690_amd as na

    if not os.path.exists(na.library_path()):
        pytest.fail("libna.so is not built (run __graft_entry__.build())")
    return na.load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(na_[a-z_]+)\s*\(", text)
    return sorted(set(names))


def test_header_declares_expected_entry_points():
    names = _declared_functions()
    for n in ("na_forward", "na_backward", "na_validate",
              "na_status_string", "na_debug_windows", "na_version"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name


def _args(rank=2, ext=(10, 12), ks=(3, 5), ds=(2, 1)):
    e = (ctypes.c_int64 * len(ext))(*ext)
    k = (ctypes.c_int32 * len(ks))(*ks)
    d = (ctypes.c_int32 * len(ds))(*ds)
    return rank, e, k, d


def _validate(lib, rank=2, ext=(10, 12), ks=(3, 5), ds=(2, 1), B=2, H=3, D=64, dt=1, scale=0.125):
    r, e, k, d = _args(rank, ext, ks, ds)
    return lib.na_validate(r, e, k, d, None, B, H, D, dt, scale)


def test_validate_statuses(lib):
    assert _validate(lib) == NA_OK
    assert _validate(lib, rank=0) == NA_ERR_RANK
    assert _validate(lib, rank=4, ext=(2, 2, 2, 2), ks=(1,) * 4, ds=(1,) * 4) == NA_ERR_RANK
    assert _validate(lib, ext=(0, 12)) == NA_ERR_SHAPE
    assert _validate(lib, ks=(0, 5)) == NA_ERR_KERNEL_SIZE
    assert _validate(lib, ds=(2, 0)) == NA_ERR_DILATION
    assert _validate(lib, ks=(6, 5)) == NA_ERR_WINDOW  # 6 * 2 > 10
    assert _validate(lib, ks=(5, 5), ds=(2, 3)) == NA_ERR_WINDOW  # 5 * 3 > 12
    assert _validate(lib, ks=(5, 12), ds=(2, 1)) == NA_OK  # k * d == extent is legal
    for D in (16, 48, 96, 256):
        assert _validate(lib, D=D) == NA_ERR_HEAD_DIM
    for D in (32, 64, 128):
        assert _validate(lib, D=D) == NA_OK
    for dt in (3, 99, -1, 1 << 30):  # any int may come through the C interface
        assert _validate(lib, dt=dt) == NA_ERR_DTYPE
    assert _validate(lib, scale=float("inf")) == NA_ERR_SCALE
    assert _validate(lib, scale=float("nan")) == NA_ERR_SCALE
    assert _validate(lib, B=-1) == NA_ERR_SHAPE
    # token index limit: N * D must stay below 2^31
    assert _validate(lib, rank=1, ext=(1 << 25,), ks=(3,), ds=(1,), D=64) == NA_ERR_SHAPE
    assert _validate(lib, rank=1, ext=(1 << 24,), ks=(3,), ds=(1,), D=64) == NA_OK


def test_validate_accepts_causal_flags(lib):
    r, e, k, d = _args()
    c = (ctypes.c_int32 * 2)(1, 0)
    assert lib.na_validate(r, e, k, d, c, 2, 3, 64, 1, 0.125) == NA_OK
    # the usual window rule still applies on a causal axis
    r, e, k, d = _args(ks=(6, 5))
    assert lib.na_validate(r, e, k, d, c, 2, 3, 64, 1, 0.125) == NA_ERR_WINDOW


def test_status_strings(lib):
    for s in list(range(10)) + [11, 12]:
        text = lib.na_status_string(s).decode()
        assert text and text != "unknown status"
    for s in (10, 14, 99, -1):  # 10 is not a status code
        assert lib.na_status_string(s).decode() == "unknown status"
    assert lib.na_version() >= 100


FAKE = 0x10000  # aligned, never dereferenced: validation fails first


def _fwd(lib, ptrs, **kw):
    r, e, k, d = _args()
    B, H, D = kw.get("B", 2), kw.get("H", 3), kw.get("D", 64)
    return lib.na_forward(r, e, k, d, None, B, H, D, 1, 0.125, *ptrs, None)


def test_forward_rejects_before_launch(lib):
    good = [FAKE] * 5
    assert _fwd(lib, [None] + good[1:]) == NA_ERR_NULL
    assert _fwd(lib, good[:4] + [None]) == NA_ERR_NULL
    assert _fwd(lib, [FAKE + 2] + good[1:]) == NA_ERR_ALIGNMENT
    assert _fwd(lib, good[:4] + [FAKE + 4]) == NA_ERR_ALIGNMENT
    assert _fwd(lib, good, D=80) == NA_ERR_HEAD_DIM
    # empty batch / heads: a no-op, pointers are not even looked at
    assert _fwd(lib, [None] * 5, B=0) == NA_OK
    assert _fwd(lib, [None] * 5, H=0) == NA_OK


def test_backward_rejects_before_launch(lib):
    r, e, k, d = _args()
    ptrs = [FAKE] * 9
    bwd = lambda p, B=2: lib.na_backward(r, e, k, d, None, B, 3, 64, 1, 0.125, *p, None)
    assert bwd([None] + ptrs[1:]) == NA_ERR_NULL
    assert bwd(ptrs[:8] + [None]) == NA_ERR_NULL
    assert bwd(ptrs[:8] + [FAKE + 1]) == NA_ERR_ALIGNMENT
    assert bwd([FAKE + 8] + ptrs[1:]) == NA_ERR_ALIGNMENT
    assert bwd([None] * 9, B=0) == NA_OK
    bad_rank = lib.na_backward(0, e, k, d, None, 2, 3, 64, 1, 0.125, *ptrs, None)
    assert bad_rank == NA_ERR_RANK


def test_debug_windows_rejects_before_launch(lib):
    r, e, k, d = _args(ks=(6, 5))
    assert lib.na_debug_windows(r, e, k, d, None, FAKE, FAKE, FAKE, None) == NA_ERR_WINDOW
    r, e, k, d = _args()
    assert lib.na_debug_windows(r, e, k, d, None, None, FAKE, FAKE, None) == NA_ERR_NULL


# ---------------------------------------------------------------- tilings
NA_ERR_TILING = 13


def _tiling_type():
    import paper_2403_04690_amd as na

    return na._NaTiling  # the na_tiling struct the binding declared the entry points with


TILING_PROBLEMS = [
    # (extents, kernel, dilation, head_dim, dtype code)
    ((56, 56), (7, 7), (1, 1), 32, 1),
    ((16, 64, 64), (7, 7, 7), (1, 2, 2), 64, 1),
    ((32768,), (1023,), (4,), 64, 1),
    ((256,), (7,), (1,), 32, 0),
    ((128, 128), (13, 13), (2, 2), 64, 2),
    ((5, 9, 11), (5, 3, 3), (1, 3, 3), 32, 0),
]


def _pow2(x):
    return x >= 1 and x & (x - 1) == 0


@pytest.mark.parametrize("ext,ks,ds,D,dt", TILING_PROBLEMS)
@pytest.mark.parametrize("fwd", [1, 0])
def test_candidate_tilings_are_valid_and_start_with_the_heuristic(lib, ext, ks, ds, D, dt, fwd):
    _Tiling = _tiling_type()
    rank = len(ext)
    r, e, k, d = _args(rank, ext, ks, ds)
    n = lib.na_candidate_tilings(r, e, k, d, 2, 4, D, dt, fwd, None, 0)
    assert n >= 1
    buf = (_Tiling * n)()
    assert lib.na_candidate_tilings(r, e, k, d, 2, 4, D, dt, fwd, buf, n) == n
    # a short buffer gets the first entries and the call still returns the total
    short = (_Tiling * 2)()
    assert lib.na_candidate_tilings(r, e, k, d, 2, 4, D, dt, fwd, short, 1) == n
    assert short[1].blocks_per_wave == 0
    assert (short[0].blocks_per_wave, tuple(short[0].wave_tile)) == \
        (buf[0].blocks_per_wave, tuple(buf[0].wave_tile))
    seen = set()
    for t in buf:
        wt, wg = tuple(t.wave_tile), tuple(t.waves)
        assert t.blocks_per_wave in (1, 2)
        assert all(_pow2(x) for x in wt + wg)
        assert all(wt[a] == 1 and wg[a] == 1 for a in range(rank, 3))
        assert wt[0] * wt[1] * wt[2] == 16 * t.blocks_per_wave
        p = wg[0] * wg[1] * wg[2]
        assert p == 4 or (p == 8 and fwd and rank == 1 and dt != 0)
        key = (t.blocks_per_wave, wt, wg)
        assert key not in seen
        seen.add(key)
    cur = _Tiling()
    assert lib.na_current_tiling(r, e, k, d, None, 2, 4, D, dt, fwd, ctypes.byref(cur)) == NA_OK
    assert (cur.blocks_per_wave, tuple(cur.wave_tile), tuple(cur.waves)) == \
        (buf[0].blocks_per_wave, tuple(buf[0].wave_tile), tuple(buf[0].waves))


# Problems whose candidate tilings were all timed on the MI355X (the tuner,
# and every 2-D wave-tile shape of both blocks-per-wave values): the
# heuristic forward tiling must be the fastest measured, or within 2 % of it.
# The backward takes the same tiling, except one block per wave at head
# dim 128.
FASTEST_FORWARD = [
    # (extents, kernel, dilation, batch, heads, head dim, dtype code, fastest forward tiling)
    ((56, 56), (7, 7), (1, 1), 4, 4, 32, 1, (1, (2, 8, 1), (4, 1, 1))),
    ((56, 56), (7, 7), (1, 1), 16, 4, 32, 1, (1, (2, 8, 1), (4, 1, 1))),
    ((56, 56), (7, 7), (1, 1), 8, 8, 64, 1, (1, (2, 8, 1), (4, 1, 1))),
    ((64, 64), (5, 5), (1, 1), 8, 8, 32, 1, (1, (2, 8, 1), (4, 1, 1))),
    ((96, 96), (9, 9), (1, 1), 4, 8, 64, 1, (1, (2, 8, 1), (4, 1, 1))),
    ((128, 128), (7, 7), (2, 2), 2, 8, 64, 1, (1, (2, 8, 1), (4, 1, 1))),
    ((128, 128), (13, 13), (2, 2), 2, 8, 64, 2, (1, (4, 4, 1), (4, 1, 1))),
    ((128, 128), (15, 15), (1, 1), 1, 8, 64, 1, (2, (2, 16, 1), (4, 1, 1))),
    ((128, 128), (21, 21), (1, 1), 1, 8, 64, 1, (2, (4, 8, 1), (4, 1, 1))),
    ((128, 128), (31, 31), (1, 1), 1, 8, 64, 1, (2, (2, 16, 1), (4, 1, 1))),
    ((8192,), (7,), (1,), 4, 8, 64, 1, (1, (16, 1, 1), (4, 1, 1))),
    ((16384,), (31,), (1,), 2, 8, 64, 1, (1, (16, 1, 1), (4, 1, 1))),
    ((32768,), (63,), (1,), 2, 8, 32, 1, (2, (32, 1, 1), (4, 1, 1))),
    ((32768,), (127,), (1,), 1, 16, 64, 1, (2, (32, 1, 1), (4, 1, 1))),
    ((4096,), (255,), (1,), 4, 8, 128, 2, (2, (32, 1, 1), (4, 1, 1))),
    ((65536,), (1023,), (1,), 1, 8, 64, 1, (2, (32, 1, 1), (8, 1, 1))),
    ((16, 64, 64), (7, 7, 7), (1, 2, 2), 1, 8, 64, 1, (2, (2, 2, 8), (2, 2, 1))),
    ((32, 32, 32), (7, 7, 7), (1, 1, 1), 1, 8, 64, 1, (2, (2, 2, 8), (2, 2, 1))),
    ((8, 56, 56), (3, 7, 7), (1, 1, 1), 1, 8, 64, 1, (1, (1, 2, 8), (2, 2, 1))),
    ((16, 48, 48), (5, 9, 9), (1, 1, 1), 1, 8, 64, 2, (1, (1, 2, 8), (2, 2, 1))),
    ((16384,), (127,), (1,), 2, 8, 64, 0, (1, (16, 1, 1), (4, 1, 1))),
    ((8192,), (255,), (1,), 2, 8, 128, 0, (1, (16, 1, 1), (4, 1, 1))),
    ((32, 32, 32), (7, 7, 7), (1, 1, 1), 1, 4, 64, 0, (1, (1, 2, 8), (2, 2, 1))),
    ((128, 128), (31, 31), (1, 1), 1, 8, 128, 1, (2, (2, 16, 1), (4, 1, 1))),
    ((32768,), (511,), (1,), 1, 8, 128, 1, (2, (32, 1, 1), (4, 1, 1))),
    ((32, 32, 32), (7, 7, 7), (1, 1, 1), 1, 4, 128, 2, (2, (2, 2, 8), (2, 2, 1))),
]


@pytest.mark.parametrize("ext,ks,ds,B,H,D,dt,best", FASTEST_FORWARD)
def test_heuristic_picks_the_fastest_measured_tiling(lib, monkeypatch, ext, ks, ds, B, H, D, dt,
                                                     best):
    monkeypatch.delenv("NA_WAVE_BLOCKS", raising=False)
    monkeypatch.delenv("NA_FWD_WAVES", raising=False)
    lib.na_tune_clear()
    r, e, k, d = _args(len(ext), ext, ks, ds)
    got = []
    for fwd in (1, 0):
        cur = _tiling_type()()
        assert lib.na_current_tiling(r, e, k, d, None, B, H, D, dt, fwd, ctypes.byref(cur)) == NA_OK
        got.append((cur.blocks_per_wave, tuple(cur.wave_tile), tuple(cur.waves)))
    assert got[0] == best
    if D == 128:
        assert got[1][0] == 1
    else:
        assert got[1] == (best[0], best[1], (4, 1, 1) if len(ext) < 3 else (2, 2, 1))


def _tiling(m, wt, wg):
    return _tiling_type()(m, (ctypes.c_int32 * 3)(*wt), (ctypes.c_int32 * 3)(*wg))


@pytest.mark.parametrize("t,rank", [
    ((3, (16, 1, 1), (4, 1, 1)), 1),    # blocks per wave
    ((1, (8, 1, 1), (4, 1, 1)), 1),     # wave tile product != 16
    ((1, (2, 8, 1), (2, 1, 1)), 2),     # waves product 2
    ((1, (2, 8, 1), (8, 1, 1)), 2),     # 8 waves outside the 1-D forward
    ((1, (3, 8, 1), (4, 1, 1)), 2),     # not a power of two
    ((1, (2, 8, 2), (4, 1, 1)), 2),     # axis beyond the rank
    ((1, (16, 1, 1), (8, 1, 1)), 1),    # 8 waves in fp32
])
def test_tiled_entry_points_reject_invalid_tilings(lib, t, rank):
    ext, ks, ds = ((10, 12), (3, 5), (2, 1)) if rank == 2 else ((40,), (3,), (2,))
    r, e, k, d = _args(rank, ext, ks, ds)
    dt = 0 if t[2][0] == 8 and rank == 1 else 1
    tl = _tiling(*t)
    fake = ctypes.c_void_p(4096)  # never dereferenced: validation fails first
    assert lib.na_forward_tiled(r, e, k, d, None, 2, 3, 64, dt, 0.125, ctypes.byref(tl),
                                *([fake] * 5), None) == NA_ERR_TILING
    if t[2][0] != 8:
        assert lib.na_backward_tiled(r, e, k, d, None, 2, 3, 64, dt, 0.125, ctypes.byref(tl),
                                     *([fake] * 9), None) == NA_ERR_TILING
    assert lib.na_forward_tiled(r, e, k, d, None, 2, 3, 64, dt, 0.125, None,
                                *([fake] * 5), None) == NA_ERR_NULL


def test_tiling_status_string_and_cache_clear(lib):
    assert b"tiling" in lib.na_status_string(NA_ERR_TILING)
    lib.na_tune_clear()  # empty cache: the current tiling is the heuristic one
    r, e, k, d = _args()
    cur = _tiling_type()()
    assert lib.na_current_tiling(r, e, k, d, None, 2, 3, 64, 1, 1, ctypes.byref(cur)) == NA_OK
    assert cur.blocks_per_wave in (1, 2)


def test_candidate_count_is_the_total_beyond_the_tuner_default(lib):
    """3-D 7x7x7 with dilation (1, 2, 2): more admissible tilings than na_tune times by
    default (64); na_candidate_tilings counts them all."""
    r, e, k, d = _args(3, (16, 64, 64), (7, 7, 7), (1, 2, 2))
    n = lib.na_candidate_tilings(r, e, k, d, 1, 8, 64, 1, 1, None, 0)
    assert n > 64
    buf = (_tiling_type() * n)()
    assert lib.na_candidate_tilings(r, e, k, d, 1, 8, 64, 1, 1, buf, n) == n
    keys = {(t.blocks_per_wave, tuple(t.wave_tile), tuple(t.waves)) for t in buf}
    assert len(keys) == n
    assert any(t.blocks_per_wave == 2 for t in buf[64:])


def test_tune_rejects_unknown_flags_before_any_launch(lib):
    r, e, k, d = _args()
    fake = ctypes.c_void_p(4096)  # never dereferenced: the flags are checked first
    st = lib.na_tune(r, e, k, d, None, 2, 3, 64, 1, 0.125, *([fake] * 9), 3, 4, None, None,
                     None, None)
    assert st == NA_ERR_TILING


def test_autotune_mode_set_and_read(lib):
    before = lib.na_autotune()
    try:
        for m in (1, 2, 0):
            lib.na_set_autotune(m)
            assert lib.na_autotune() == m
        lib.na_set_autotune(7)  # unknown modes turn it off
        assert lib.na_autotune() == 0
    finally:
        lib.na_set_autotune(before)


@pytest.mark.parametrize("B,H,ok", [(1 << 22, 1, True), (1 << 23, 1, False), (1 << 12, 1 << 10, True),
                                    (1 << 12, 1 << 11, False)])
def test_launches_beyond_the_grid_limit_are_rejected(lib, B, H, ok):
    """1-D L = 16 (one 64-query tile per slice): the backward launches 2 * B * H workgroups of
    256 threads, which must stay below 2^32 threads, so B * H < 2^23."""
    r, e, k, d = _args(1, (16,), (3,), (1,))
    want = NA_OK if ok else NA_ERR_SHAPE
    assert lib.na_validate(r, e, k, d, None, B, H, 32, 1, 0.125) == want
    fake = ctypes.c_void_p(4096)
    if not ok:  # refused before any pointer is read
        assert lib.na_forward(r, e, k, d, None, B, H, 32, 1, 0.125, *([fake] * 5), None) == want
        assert lib.na_backward(r, e, k, d, None, B, H, 32, 1, 0.125, *([fake] * 9), None) == want


def test_fast_marshalling_matches_ctypes(lib):
    """The binding's argument-marshalling extension (_na_fast, built beside libna.so) calls
    the same entry points: on invalid and empty problems (no launch) it returns exactly the
    statuses the ctypes calls return."""
    import paper_2403_04690_amd as na

    if na._fast is None:
        pytest.skip("_na_fast is not built")
    cases = [  # (extents, kernel, dilation, B, H, D, dtype)
        ((10, 12), (3, 5), (2, 1), 2, 3, 48, 1), ((10, 12), (6, 5), (2, 1), 2, 3, 64, 1),
        ((10, 12), (3, 5), (2, 1), 2, 3, 64, 7), ((10, 12), (3, 5), (2, 1), 0, 3, 64, 1),
        ((40,), (7,), (1,), -1, 1, 32, 0), ((4, 4, 4), (3, 3, 3), (1, 1, 1), 1, 1, 32, 2),
    ]
    for ext, ks, ds, B, H, D, dt in cases:
        rank, e, k, d, cs, addrs = na._problem(ext, ks, ds)
        want_f = lib.na_forward(rank, e, k, d, cs, B, H, D, dt, 0.5, None, None, None, None,
                                None, None)
        want_b = lib.na_backward(rank, e, k, d, cs, B, H, D, dt, 0.5, *([None] * 10))
        got_f = na._fast.forward(na._fast_fn["fwd"], rank, *addrs, B, H, D, dt, 0.5, *([0] * 6))
        got_b = na._fast.backward(na._fast_fn["bwd"], rank, *addrs, B, H, D, dt, 0.5,
                                  *([0] * 10))
        assert (got_f, got_b) == (want_f, want_b), (ext, ks, ds, B, H, D, dt)
    with pytest.raises(TypeError):
        na._fast.forward(na._fast_fn["fwd"], 1)
    # another build swapped in (as A/B comparisons do): the addresses follow it
    saved = na._lib
    try:
        other = ctypes.CDLL(na.library_path(), mode=ctypes.RTLD_LOCAL)
        na._lib = other
        assert na._fast_for(other)["fwd"] == ctypes.cast(other.na_forward, ctypes.c_void_p).value
    finally:
        na._lib = saved
        na._fast_for(saved)
