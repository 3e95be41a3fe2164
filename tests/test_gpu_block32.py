"""GPU parity of the block-size control (Sec. "Recipe comparison", Table
tab:results): UE5M3 (and E4M3) block scales over blocks of 32 elements for
activations and gradients and 32 x 32 tiles for weights, through the C
ABI's _ex calls.
Quantizer payloads and scales bit-exact with the oracle (same per-block
arithmetic, one scale code per 32 elements or per 32 x 32 tile); decoded
GEMMs to the 1e-3 / fp32-accumulation bar of tests/gpu_util.gemm_check;
probe-matched GEMMs equal to the oracle's output model at every compared
output."""

import numpy as np
import pytest
import torch

import paper_2609_02846_amd as ue
import synthetic
from oracle import accumulate as oacc
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc
from tests.gpu_util import f32_scalar_dev, gemm_check, host, say, set_amax, to_dev, u8_to_dev
from tests.test_gpu_quantize import _all_bf16

pytestmark = pytest.mark.gpu

FMTS = ["ue5m3", "e4m3"]
ROWS = [(1, 32), (3, 64), (37, 96), (100, 1056), (256, 512), (64, 4128)]
COLS = [(32, 2), (64, 38), (96, 100), (512, 300), (160, 1030), (1024, 256), (2080, 64)]
TILES = [(32, 32), (64, 96), (96, 160), (512, 1024), (224, 4096), (1056, 288)]


def _amax_dev(g):
    a = torch.zeros(1, dtype=torch.float32, device="cuda")
    set_amax(a, g)
    return a


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_quantize_rows_and_cols_block32(fmt, mode):
    for axis, cases in [(1, ROWS), (0, COLS)]:
        for shape in cases:
            say("block32", fmt, mode, "axis", axis, shape)
            bits = synthetic.gradient(8, *shape, 1e-4, 2.0) if mode == "sr" else \
                synthetic.activation(8, *shape, 0.01, 50.0)
            g = osc.amax(bits)
            p, s, d = ue.quantize_1d(to_dev(bits), axis, _amax_dev(g), 448.0, mode, seed=2, tensor_id=5,
                                     fmt=fmt, block=32)
            po, so, do = oq.quantize_1d(bits, axis, g, 448.0, mode, 2, 5, fmt=fmt, block=32)
            assert np.array_equal(host(s), so), (fmt, mode, axis, shape)
            assert np.array_equal(host(p), po), (fmt, mode, axis, shape)
            assert np.float32(d.item()) == do


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_quantize_tiles_32(fmt, mode):
    for shape in TILES:
        say("tiles 32", fmt, mode, shape)
        bits = synthetic.weight(9, *shape)
        g = osc.amax(bits)
        p, s, pt, d, st = ue.quantize_2d(to_dev(bits), _amax_dev(g), 448.0, mode, seed=4, tensor_id=6,
                                         fmt=fmt, tile=32)
        po, so, pto, do = oq.quantize_2d(bits, g, 448.0, mode, 4, 6, fmt=fmt, tile=32)
        assert so.shape == (shape[0] // 32, shape[1] // 32)
        assert np.array_equal(host(s), so) and np.array_equal(host(p), po), shape
        assert np.array_equal(host(pt), pto) and np.array_equal(host(st), so.T), shape
        assert np.float32(d.item()) == do
    say("tiles 32 without the transposed outputs", fmt, mode)
    bits = synthetic.weight(10, 96, 160)
    g = osc.amax(bits)
    p, s, pt, d, st = ue.quantize_2d(to_dev(bits), _amax_dev(g), 448.0, mode, seed=4, tensor_id=6,
                                     transposed=False, fmt=fmt, tile=32)
    po, so, _, _ = oq.quantize_2d(bits, g, 448.0, mode, 4, 6, fmt=fmt, tile=32)
    assert pt is None and st is None
    assert np.array_equal(host(s), so) and np.array_equal(host(p), po)


@pytest.mark.parametrize("g", [1.0, 3.0e4, 2.0 ** -20])
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_every_bf16_value_block32(g, mode):
    """Every non-NaN bf16 value through the block-32 rows and columns
    quantizers and the 32 x 32 tiles (UE5M3), held references below, inside
    and above range."""
    say("every bf16 value block32", g, mode)
    bits = _all_bf16(256, 512, 23)
    xd = to_dev(bits)
    amax = _amax_dev(g)
    for axis in [1, 0]:
        p, s, d = ue.quantize_1d(xd, axis, amax, 448.0, mode, seed=13, tensor_id=3, block=32)
        po, so, do = oq.quantize_1d(bits, axis, np.float32(g), 448.0, mode, 13, 3, block=32)
        assert np.array_equal(host(s), so), axis
        assert np.array_equal(host(p), po), axis
    p, s, pt, d, st = ue.quantize_2d(xd, amax, 448.0, mode, seed=13, tensor_id=4, tile=32)
    po, so, pto, do = oq.quantize_2d(bits, np.float32(g), 448.0, mode, 13, 4, tile=32)
    assert np.array_equal(host(s), so) and np.array_equal(host(p), po)
    assert np.array_equal(host(pt), pto)


def _operands(fmt, T, K, N, seed, dy_mode="sr"):
    """Oracle block-32 quantization of the three operands of one linear and
    the decoded matrices of each product, in GEMM operand order."""
    x = synthetic.activation(seed, T, K, 1e-2, 50.0)
    w = synthetic.weight(seed, N, K)
    dy = synthetic.gradient(seed, T, N, 1e-3, 1.0)
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    q = lambda b, axis, g, mode="rn", tid=0: oq.quantize_1d(b, axis, g, 448.0, mode, 1, tid, fmt=fmt, block=32)
    dec = lambda r, axis: oq.decoded_1d(r[0], r[1], axis, fmt=fmt, block=32)
    xr, xc = q(x, 1, gx), q(x, 0, gx)
    dr, dc = q(dy, 1, gd, dy_mode, 1), q(dy, 0, gd, dy_mode, 2)
    wq = oq.quantize_2d(w, gw, fmt=fmt, tile=32)
    W = oq.decoded_2d(wq[0], wq[1], fmt=fmt, tile=32)
    U, D = u8_to_dev, f32_scalar_dev
    X, dY = dec(xr, 1), dec(dr, 1)
    Xc, dYc = dec(xc, 0), dec(dc, 0)
    return [
        ("nt", T, N, K, (U(xr[0]), U(xr[1]), D(xr[2]), U(wq[0]), U(wq[1]), D(wq[3])), X, W,
         ogemm.alpha(xr[2], wq[3])),
        ("nn", T, K, N, (U(dr[0]), U(dr[1]), D(dr[2]), U(wq[2]), U(np.ascontiguousarray(wq[1].T)), D(wq[3])),
         dY, np.ascontiguousarray(W.T), ogemm.alpha(dr[2], wq[3])),
        ("tn", N, K, T, (U(dc[0]), U(dc[1]), D(dc[2]), U(xc[0]), U(xc[1]), D(xc[2])),
         np.ascontiguousarray(dYc.T), np.ascontiguousarray(Xc.T), ogemm.alpha(dc[2], xc[2])),
    ]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("T,K,N", [(32, 32, 32), (96, 320, 160), (288, 352, 224), (512, 1024, 768)])
def test_gemm_block32_three_layouts(fmt, T, K, N):
    for lay, M_, N_, K_, args, A, B, al in _operands(fmt, T, K, N, 3):
        say("gemm block32", fmt, lay, M_, N_, K_)
        c = ue.gemm(lay, M_, N_, K_, *args, fmt=fmt, block=32)
        torch.cuda.synchronize()
        gemm_check(host(c), ogemm.fprop(A, B, al), al, ogemm.abs_product(A, B), K_,
                   f"{fmt} b32 {lay} {M_}x{N_}x{K_}")


def test_gemm_block32_persistent_and_bf16():
    """More 256 x 256 tiles than compute units for the persistent decoded
    kernel (fp32 and bf16 outputs), then smaller calls on the same stream
    (the expanded-scale workspace is reused).  Round-to-nearest dY keeps the
    oracle's share of the run short."""
    for T, K, N in [(4096, 1024, 4608), (256, 512, 256)]:
        for lay, M_, N_, K_, args, A, B, al in _operands("ue5m3", T, K, N, 4, "rn"):
            say("gemm block32 persistent", lay, M_, N_, K_)
            ref = ogemm.fprop(A, B, al)
            c = ue.gemm(lay, M_, N_, K_, *args, block=32)
            torch.cuda.synchronize()
            gemm_check(host(c), ref, al, ogemm.abs_product(A, B), K_, f"b32 {lay} {M_}x{N_}x{K_}")
            if lay == "nt":
                c16 = host(ue.gemm(lay, M_, N_, K_, *args, block=32, out_dtype=torch.bfloat16).float())
                e = float(al) * K_ * 2.0 ** -23 * ogemm.abs_product(A, B)
                ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref) + e, 1e-30))) - 7)
                assert np.all(np.abs(c16.astype(np.float64) - ref) <= e + 1.01 * ulp + 1e-30)


def _pm_ref(A, B, al, d, idx):
    return np.array([oacc.dot(A[m] * B[n], d, al)[0] for m, n in idx], np.float32)


@pytest.mark.parametrize("fmt", FMTS)
def test_gemm_pm_block32(fmt):
    """Probe-matched GEMM on block-32 operands: sampled outputs (tile
    corners, edges, random) equal the oracle's model exactly."""
    T, K, N = 288, 352, 160                   # K: 5 groups of 64 and a half group
    rng = np.random.default_rng(7)
    for lay, M_, N_, K_, args, A, B, al in _operands(fmt, T, K, N, 5):
        ms = sorted({0, M_ - 1, 127, 128, 255, 256})
        ns = sorted({0, N_ - 1, 127, 128})
        idx = sorted({(m, n) for m in ms if m < M_ for n in ns if n < N_} |
                     {(int(rng.integers(M_)), int(rng.integers(N_))) for _ in range(300)})
        for d in (1024, 0):
            say("gemm_pm block32", fmt, lay, M_, N_, K_, "grid", d)
            c = ue.gemm_pm(lay, M_, N_, K_, *args, grid=d, fmt=fmt, block=32)
            torch.cuda.synchronize()
            got = host(c)
            g = np.array([got[m, n] for m, n in idx], np.float32)
            ref = _pm_ref(A, B, al, d, idx)
            bad = np.nonzero(g != ref)[0]
            assert bad.size == 0, (f"{fmt} {lay} d={d}: {bad.size}/{len(idx)} differ, first {idx[bad[0]]}: "
                                   f"{g[bad[0]]!r} vs {ref[bad[0]]!r}")


def test_quantizers_feed_gemm_block32_end_to_end():
    """GPU block-32 quantizers then the GPU GEMM equal the oracle's
    quantize-then-GEMM."""
    T, K, N = 256, 512, 384
    x = synthetic.activation(31, T, K, 1e-2, 50.0)
    w = synthetic.weight(31, N, K)
    gx, gw = osc.amax(x), osc.amax(w)
    say("block32 end to end")
    xr = ue.quantize_1d(to_dev(x), 1, _amax_dev(gx), block=32)
    wq = ue.quantize_2d(to_dev(w), _amax_dev(gw), tile=32)
    c = ue.gemm("nt", T, N, K, *xr, wq[0], wq[1], wq[3], block=32)
    xo = oq.quantize_1d(x, 1, gx, block=32)
    wo = oq.quantize_2d(w, gw, tile=32)
    X, W = oq.decoded_1d(xo[0], xo[1], 1, block=32), oq.decoded_2d(wo[0], wo[1], tile=32)
    al = ogemm.alpha(xo[2], wo[3])
    gemm_check(host(c), ogemm.fprop(X, W, al), al, ogemm.abs_product(X, W), K, "b32 end to end")


def test_gemm_block32_empty_and_k_zero():
    say("gemm block32 K=0 and empty")
    one = f32_scalar_dev(1.0)
    dummy = torch.zeros(16, dtype=torch.uint8, device="cuda")
    c = torch.full((8, 32), 7.0, device="cuda")
    ue.gemm("nt", 8, 32, 0, dummy, dummy, one, dummy, dummy, one, out=c, block=32)
    torch.cuda.synchronize()
    assert (host(c) == 0).all()
    c = torch.full((8, 32), 7.0, device="cuda")
    ue.gemm_pm("nt", 8, 32, 0, dummy, dummy, one, dummy, dummy, one, out=c, block=32)
    torch.cuda.synchronize()
    assert (host(c) == 0).all()
    ue.gemm("nt", 0, 32, 64, dummy, dummy, one, dummy, dummy, one, out=torch.empty(0, device="cuda"), block=32)
