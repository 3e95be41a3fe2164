"""CPU checks of the C ABI: the library loads, exports every function that
include/ue5m3.h declares, and validates arguments on the host (these calls
return before anything is enqueued, so no GPU is needed)."""

import ctypes
import os
import re

import pytest

import paper_2609_02846_amd as ue
from paper_2609_02846_amd import build as ue_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ue.LIB_PATH):
        ue_build.build(verbose=False)
    return ue.load_library()


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "ue5m3.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ue5m3_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert set(names) == set(ue.EXPORTED_SYMBOLS)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.ue5m3_version() == 200


def test_status_strings(lib):
    for s in range(7):
        assert ue.status_string(s)
    assert ue.status_string(99) == "unknown status"


FAKE = ctypes.c_void_p(0x100000)          # aligned, never dereferenced
FAKE_MIS = ctypes.c_void_p(0x100004)      # 4-byte but not 16-byte aligned
NULL = None


def test_quantize_1d_validation(lib):
    q = lib.ue5m3_quantize_1d
    args = dict(x=FAKE, rows=32, cols=32, axis=1, amax=FAKE, T=448.0, mode=0, seed=0, tid=0,
                p=FAKE, s=FAKE, d=NULL, st=NULL)

    def call(**kw):
        a = dict(args, **kw)
        return q(a["x"], a["rows"], a["cols"], a["axis"], a["amax"], a["T"], a["mode"], a["seed"],
                 a["tid"], a["p"], a["s"], a["d"], a["st"])
    assert call(axis=2) == ue.UE5M3_EINVAL
    assert call(mode=7) == ue.UE5M3_EINVAL
    assert call(amax=NULL) == ue.UE5M3_EINVAL
    for bad_t in [0.0, -1.0, float("inf"), float("nan"), 1e38]:
        assert call(T=bad_t) == ue.UE5M3_EINVAL
    assert call(cols=24) == ue.UE5M3_ESHAPE             # axis 1 needs cols % 16
    assert call(rows=-1) == ue.UE5M3_ESHAPE
    assert call(axis=0, rows=24) == ue.UE5M3_ESHAPE     # axis 0 needs rows % 16
    assert call(axis=0, cols=33) == ue.UE5M3_ESHAPE     # and cols % 2
    assert call(x=NULL) == ue.UE5M3_EINVAL
    assert call(p=NULL) == ue.UE5M3_EINVAL
    assert call(x=FAKE_MIS) == ue.UE5M3_EALIGN
    assert call(s=FAKE_MIS) == ue.UE5M3_EALIGN
    assert call(rows=0) == ue.UE5M3_OK                  # empty: nothing to do
    assert call(cols=0, x=NULL, p=NULL, s=NULL) == ue.UE5M3_OK


def test_quantize_2d_validation(lib):
    q = lib.ue5m3_quantize_2d

    def call(rows=32, cols=32, w=FAKE, amax=FAKE, T=448.0, mode=0, p=FAKE, s=FAKE, pt=NULL, st=NULL):
        return q(w, rows, cols, amax, T, mode, 0, 0, p, s, pt, st, NULL, NULL)
    assert call(rows=24) == ue.UE5M3_ESHAPE
    assert call(cols=40) == ue.UE5M3_ESHAPE
    assert call(mode=2) == ue.UE5M3_EINVAL
    assert call(T=0.0) == ue.UE5M3_EINVAL
    assert call(pt=FAKE_MIS) == ue.UE5M3_EALIGN
    assert call(st=FAKE_MIS) == ue.UE5M3_EALIGN
    assert call(w=NULL) == ue.UE5M3_EINVAL
    assert call(rows=0) == ue.UE5M3_OK


ROW16, COL16T, TILE16, ROW32, COL32T, TILE32 = range(6)
# recipe blockings per layout (Table 5): NT X rows / W tiles, NN dY rows / W
# tiles (transposed copy), TN dY and X down columns (stored transposed)
RECIPE = {0: (ROW16, TILE16), 1: (ROW16, TILE16), 2: (COL16T, COL16T)}


def test_gemm_validation(lib):
    g = lib.ue5m3_gemm

    def call(layout=0, M=32, N=32, K=32, a=FAKE, b=FAKE, c=FAKE, ctype=0, ad=FAKE, bd=FAKE, ab=None, bb=None):
        da, db = RECIPE.get(layout, (ROW16, TILE16))
        ab = da if ab is None else ab
        bb = db if bb is None else bb
        return g(layout, M, N, K, a, FAKE, ab, ad, b, FAKE, bb, bd, c, ctype, NULL)
    for lay in (0, 1, 2):
        assert call(layout=lay, M=0) == ue.UE5M3_OK
    assert call(layout=3) == ue.UE5M3_ELAYOUT
    assert call(K=40) == ue.UE5M3_ESHAPE
    assert call(N=40) == ue.UE5M3_ESHAPE                 # weight tiles need N % 16
    assert call(layout=1, N=40) == ue.UE5M3_ESHAPE
    assert call(N=40, bb=ROW16, M=0) == ue.UE5M3_OK       # a 1D-blocked weight does not
    assert call(M=-1) == ue.UE5M3_ESHAPE
    assert call(ctype=5) == ue.UE5M3_EINVAL
    assert call(c=NULL) == ue.UE5M3_EINVAL
    assert call(ad=NULL) == ue.UE5M3_EINVAL
    assert call(a=FAKE_MIS) == ue.UE5M3_EALIGN
    assert call(M=0) == ue.UE5M3_OK and call(N=0) == ue.UE5M3_OK
    # blocks of 32 and unknown values are not blockings of this call
    for bad in (ROW32, COL32T, TILE32, 6, -1):
        assert call(ab=bad, M=0) == ue.UE5M3_EINVAL and call(bb=bad, M=0) == ue.UE5M3_EINVAL


def test_gemm_blocking_rule(lib):
    """Every operand must be blocked along its GEMM's contraction
    (eq:microscaling, Sec. 4.3): for each layout, every blocking pair is
    accepted exactly when A is 1D along the contraction and B is 1D along it
    or tiled; all other pairs are UE5M3_ELAYOUT, checked before anything is
    enqueued (M = 0 would otherwise return OK)."""
    a_rows = {0: True, 1: True, 2: False}       # A source contracted along its rows?
    b_rows = {0: True, 1: False, 2: False}
    for fn in ("ue5m3_gemm", "ue5m3_gemm_ex", "ue5m3_gemm_pm"):
        g = getattr(lib, fn)
        for lay in (0, 1, 2):
            for ab in (ROW16, COL16T, TILE16):
                for bb in (ROW16, COL16T, TILE16):
                    ok_a = ab == (ROW16 if a_rows[lay] else COL16T)
                    ok_b = bb == TILE16 or bb == (ROW16 if b_rows[lay] else COL16T)
                    want = ue.UE5M3_OK if ok_a and ok_b else ue.UE5M3_ELAYOUT
                    args = (lay, 0, 32, 64, FAKE, FAKE, ab, FAKE, FAKE, FAKE, bb, FAKE, FAKE, 0)
                    if fn == "ue5m3_gemm":
                        st = g(*args, NULL)
                    elif fn == "ue5m3_gemm_ex":
                        st = g(*args, 0, NULL)
                    else:
                        st = g(*args, 0, 1024, NULL)
                    assert st == want, (fn, lay, ab, bb, st)
                    # the same rule with blocks of 32 (_ex, _pm)
                    if fn != "ue5m3_gemm":
                        args32 = args[:6] + (ab + 3,) + args[7:10] + (bb + 3,) + args[11:]
                        st32 = g(*args32, 0, NULL) if fn == "ue5m3_gemm_ex" else g(*args32, 0, 1024, NULL)
                        assert st32 == want, (fn, lay, ab + 3, bb + 3, st32)


def test_amax_state_host_logic(lib):
    """The refresh decision is host-only: with a cache present, steps inside
    the period enqueue nothing (eq:delayed-amax)."""
    st = ue.AmaxStateC()
    assert lib.ue5m3_amax_state_init(ctypes.byref(st), NULL, 50) == ue.UE5M3_EINVAL
    assert lib.ue5m3_amax_state_init(ctypes.byref(st), FAKE, -1) == ue.UE5M3_EINVAL
    assert lib.ue5m3_amax_state_init(ctypes.byref(st), FAKE, 50) == ue.UE5M3_OK
    assert st.has_cache == 0 and st.period == 50
    st.has_cache, st.last_refresh = 1, 100
    flag = ctypes.c_int32(-1)
    for step in [100, 120, 149]:
        assert lib.ue5m3_amax_sample(ctypes.byref(st), FAKE, 64, step, ctypes.byref(flag), NULL) == 0
        assert flag.value == 0 and st.last_refresh == 100
    assert lib.ue5m3_amax_sample(ctypes.byref(st), FAKE, -1, 150, ctypes.byref(flag), NULL) == ue.UE5M3_ESHAPE
    assert lib.ue5m3_amax_sample(ctypes.byref(st), FAKE_MIS, 64, 150, ctypes.byref(flag), NULL) == ue.UE5M3_EALIGN
    lib.ue5m3_amax_state_reset(ctypes.byref(st))
    assert st.has_cache == 0
    lib.ue5m3_amax_state_reset(None)


def test_amax_hold_and_freeze_host_logic(lib):
    """Period 0 holds the first measurement until reset; freeze holds the
    reference already in amax_dev (inference policies, Table
    tab:inference-scale-summary).  Only host integers are involved."""
    st = ue.AmaxStateC()
    assert lib.ue5m3_amax_state_init(ctypes.byref(st), FAKE, 0) == ue.UE5M3_OK
    st.has_cache, st.last_refresh = 1, 3           # as after the first refresh
    flag = ctypes.c_int32(-1)
    for step in [3, 53, 10**15]:
        assert lib.ue5m3_amax_sample(ctypes.byref(st), FAKE, 64, step, ctypes.byref(flag), NULL) == 0
        assert flag.value == 0 and st.last_refresh == 3
    assert lib.ue5m3_amax_state_init(ctypes.byref(st), FAKE, 50) == ue.UE5M3_OK
    lib.ue5m3_amax_state_freeze(ctypes.byref(st))
    assert st.has_cache == 1 and st.period == 0
    assert lib.ue5m3_amax_sample(ctypes.byref(st), FAKE, 64, 500, ctypes.byref(flag), NULL) == 0
    assert flag.value == 0
    lib.ue5m3_amax_state_freeze(None)
    st.period = -2
    assert lib.ue5m3_amax_sample(ctypes.byref(st), FAKE, 64, 0, ctypes.byref(flag), NULL) == ue.UE5M3_EINVAL


def test_amax_accumulate_validation(lib):
    acc = lib.ue5m3_amax_accumulate
    assert acc(FAKE, 64, NULL, 1, NULL) == ue.UE5M3_EINVAL
    assert acc(NULL, 64, FAKE, 1, NULL) == ue.UE5M3_EINVAL
    assert acc(FAKE, 64, FAKE, 2, NULL) == ue.UE5M3_EINVAL
    assert acc(FAKE, -1, FAKE, 0, NULL) == ue.UE5M3_ESHAPE
    assert acc(FAKE_MIS, 64, FAKE, 0, NULL) == ue.UE5M3_EALIGN
    assert acc(FAKE, 64, ctypes.c_void_p(0x100002), 0, NULL) == ue.UE5M3_EALIGN


def test_format_entry_points_validation(lib):
    """_ex calls: scale kind, block length, E8M0 without amax, 2D E8M0, the
    block-32 shapes and the E8M0 GEMM's K % 256 requirement are checked on
    the host."""
    q = lib.ue5m3_quantize_1d_ex

    def call(kind=1, block=16, amax=FAKE, rows=32, cols=32, axis=1):
        return q(FAKE, rows, cols, axis, amax, 448.0, 0, 0, 0, kind, block, FAKE, FAKE, NULL, NULL)
    assert call(kind=3) == ue.UE5M3_EINVAL
    assert call(kind=1, block=32, rows=0) == ue.UE5M3_OK      # block-size control
    assert call(kind=0, block=32, cols=48) == ue.UE5M3_ESHAPE
    assert call(kind=0, block=32, axis=0, rows=48) == ue.UE5M3_ESHAPE
    assert call(kind=0, block=8) == ue.UE5M3_EINVAL and call(kind=1, block=64) == ue.UE5M3_EINVAL
    assert call(kind=2, block=16) == ue.UE5M3_EINVAL          # E8M0 blocks are 32
    assert call(kind=1, amax=NULL) == ue.UE5M3_EINVAL         # E4M3 needs the held amax
    assert call(kind=2, block=32, amax=NULL, rows=0) == ue.UE5M3_OK   # E8M0 does not
    assert call(kind=2, block=32, cols=48) == ue.UE5M3_ESHAPE
    assert call(kind=2, block=32, axis=0, rows=48) == ue.UE5M3_ESHAPE
    q2 = lib.ue5m3_quantize_2d_ex

    def q2call(kind=0, tile=16, rows=32, cols=32):
        return q2(FAKE, rows, cols, FAKE, 448.0, 0, 0, 0, kind, tile, FAKE, FAKE, NULL, NULL, NULL, NULL)
    assert q2call(kind=2) == ue.UE5M3_EINVAL and q2call(kind=2, tile=32) == ue.UE5M3_EINVAL
    assert q2call(kind=1, rows=0) == ue.UE5M3_OK and q2call(tile=32, rows=0) == ue.UE5M3_OK
    assert q2call(tile=8) == ue.UE5M3_EINVAL and q2call(tile=64) == ue.UE5M3_EINVAL
    assert q2call(tile=32, rows=48) == ue.UE5M3_ESHAPE and q2call(tile=32, cols=48) == ue.UE5M3_ESHAPE
    g = lib.ue5m3_gemm_ex

    def gcall(kind=2, M=32, N=32, K=256, layout=0, block=None, ab=None, bb=None):
        block = (32 if kind == 2 else 16) if block is None else block
        da, db = RECIPE.get(layout, (ROW16, TILE16))
        if kind == 2 and layout in (0, 1):
            db = ROW16 if layout == 0 else COL16T          # E8M0 weights are 1D
        off = 3 if block == 32 else 0
        ab = da + off if ab is None else ab
        bb = db + off if bb is None else bb
        return g(layout, M, N, K, FAKE, FAKE, ab, FAKE, FAKE, FAKE, bb, FAKE, FAKE, 0, kind, NULL)
    assert gcall(kind=5) == ue.UE5M3_EINVAL
    assert gcall(K=128) == ue.UE5M3_ESHAPE                    # E8M0 needs K % 256
    assert gcall(kind=1, K=128, N=40) == ue.UE5M3_ESHAPE      # E4M3 NT: N % 16
    assert gcall(block=16) == ue.UE5M3_EINVAL                 # E8M0 blocks are 32
    assert gcall(ab=TILE32, layout=2, M=0) == ue.UE5M3_EINVAL   # and 1D only
    assert gcall(bb=TILE32, M=0) == ue.UE5M3_EINVAL
    assert gcall(kind=0, ab=ROW16, bb=TILE32, M=0) == ue.UE5M3_EINVAL   # block lengths differ
    assert gcall(kind=0, block=32, K=48) == ue.UE5M3_ESHAPE   # block 32: K % 32
    assert gcall(kind=1, block=32, N=48) == ue.UE5M3_ESHAPE   # and N % 32 for tiles
    assert gcall(kind=1, block=32, N=48, layout=1) == ue.UE5M3_ESHAPE
    assert gcall(kind=0, block=32, N=48, layout=2, M=0) == ue.UE5M3_OK
    assert gcall(layout=3) == ue.UE5M3_ELAYOUT
    assert gcall(M=0) == ue.UE5M3_OK
    assert gcall(M=1 << 20, N=1 << 20) == ue.UE5M3_ESHAPE     # 32-bit offsets


def test_dual_quantizer_validation(lib):
    d = lib.ue5m3_quantize_dual

    def call(rows=32, cols=32, kind=0, mode=0, amax=FAKE):
        return d(FAKE, rows, cols, amax, 448.0, mode, 0, 1, 2, kind, FAKE, FAKE, FAKE, FAKE, NULL, NULL)
    assert call(kind=2) == ue.UE5M3_EINVAL          # E8M0 blocks are 32
    assert call(mode=3) == ue.UE5M3_EINVAL
    assert call(amax=NULL) == ue.UE5M3_EINVAL
    assert call(rows=24) == ue.UE5M3_ESHAPE
    assert call(cols=40) == ue.UE5M3_ESHAPE
    assert call(rows=0) == ue.UE5M3_OK


def test_gemm_pm_validation(lib):
    g = lib.ue5m3_gemm_pm

    def call(layout=0, M=32, N=32, K=64, kind=0, grid=1024, ctype=0, a=FAKE, c=FAKE, block=16):
        da, db = RECIPE.get(layout, (ROW16, TILE16))
        if block not in (16, 32):
            da, db = 6, 6                                     # no blocking of that length
        elif block == 32:
            da, db = da + 3, db + 3
        return g(layout, M, N, K, a, FAKE, da, FAKE, FAKE, FAKE, db, FAKE, c, ctype, kind, grid, NULL)
    assert call(layout=3) == ue.UE5M3_ELAYOUT
    assert call(kind=2) == ue.UE5M3_EINVAL                 # E8M0 has no probe-matched path
    for bad in (-1, 1000, 3, (1 << 31) - 1):
        assert call(grid=bad) == ue.UE5M3_EINVAL
    assert call(K=40) == ue.UE5M3_ESHAPE
    assert call(N=40) == ue.UE5M3_ESHAPE and call(layout=1, N=40) == ue.UE5M3_ESHAPE
    assert call(ctype=3) == ue.UE5M3_EINVAL
    assert call(c=NULL) == ue.UE5M3_EINVAL
    assert call(a=FAKE_MIS) == ue.UE5M3_EALIGN
    assert call(M=0) == ue.UE5M3_OK and call(N=0) == ue.UE5M3_OK
    assert call(block=8) == ue.UE5M3_EINVAL and call(block=64) == ue.UE5M3_EINVAL
    assert call(block=32, K=48) == ue.UE5M3_ESHAPE and call(block=32, N=48) == ue.UE5M3_ESHAPE
    assert call(block=32, M=0) == ue.UE5M3_OK


def test_rht_entry_points_validation(lib):
    st = ue.AmaxStateC()
    assert lib.ue5m3_amax_state_init(ctypes.byref(st), FAKE, 1) == ue.UE5M3_OK
    smp = lib.ue5m3_amax_sample_rht
    flag = ctypes.c_int32(-1)
    assert smp(ctypes.byref(st), FAKE, 24, 8, 0, 0, ctypes.byref(flag), NULL) == ue.UE5M3_ESHAPE
    assert smp(ctypes.byref(st), FAKE, 32, 7, 0, 0, ctypes.byref(flag), NULL) == ue.UE5M3_ESHAPE
    assert smp(ctypes.byref(st), FAKE, 32, 8, 1 << 16, 0, ctypes.byref(flag), NULL) == ue.UE5M3_EINVAL
    assert smp(ctypes.byref(st), FAKE_MIS, 32, 8, 0, 0, ctypes.byref(flag), NULL) == ue.UE5M3_EALIGN
    st.has_cache, st.last_refresh = 1, 5
    assert smp(ctypes.byref(st), FAKE, 32, 8, 0, 5, ctypes.byref(flag), NULL) == 0 and flag.value == 0
    q = lib.ue5m3_quantize_cols_rht

    def call(rows=32, cols=8, amax=FAKE, T=448.0, mode=0, mask=0x1234, x=FAKE, p=FAKE):
        return q(x, rows, cols, amax, T, mode, 0, 0, mask, p, FAKE, NULL, NULL)
    assert call(mode=2) == ue.UE5M3_EINVAL
    assert call(amax=NULL) == ue.UE5M3_EINVAL
    assert call(T=0.0) == ue.UE5M3_EINVAL
    assert call(mask=1 << 16) == ue.UE5M3_EINVAL
    assert call(rows=24) == ue.UE5M3_ESHAPE and call(cols=9) == ue.UE5M3_ESHAPE
    assert call(x=NULL) == ue.UE5M3_EINVAL and call(p=NULL) == ue.UE5M3_EINVAL
    assert call(x=FAKE_MIS) == ue.UE5M3_EALIGN
    assert call(rows=0) == ue.UE5M3_OK
