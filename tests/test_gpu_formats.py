"""GPU parity of the comparison scale formats (Sec. 2, Table tab:formats):
E4M3 block scales (blocks of 16 under the tensor scale) and E8M0 block
scales (blocks of 32, no tensor scale), through the C ABI's _ex calls.
Quantizer payloads and scales bit-exact with the oracle; GEMMs to the
1e-3 / fp32-accumulation bar of tests/gpu_util.gemm_check."""

import numpy as np
import pytest
import torch

import paper_2609_02846_amd as ue
import synthetic
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc
from tests.gpu_util import f32_scalar_dev, gemm_check, host, say, set_amax, to_dev, u8_to_dev
from tests.test_gpu_quantize import _all_bf16

pytestmark = pytest.mark.gpu


def _amax_dev(bits):
    a = torch.zeros(1, dtype=torch.float32, device="cuda")
    set_amax(a, osc.amax(bits))
    return a


ROWS = {"e4m3": [(1, 16), (37, 48), (100, 1040), (256, 512)],
        "e8m0": [(1, 32), (3, 64), (37, 96), (100, 1056), (256, 512)]}
COLS = {"e4m3": [(16, 2), (48, 38), (512, 300), (80, 1030)],
        "e8m0": [(32, 2), (64, 38), (96, 100), (512, 300), (160, 1030), (1024, 256)]}


@pytest.mark.parametrize("fmt", ["e4m3", "e8m0"])
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_quantize_rows_and_cols(fmt, mode):
    for axis, cases in [(1, ROWS[fmt]), (0, COLS[fmt])]:
        for shape in cases:
            say("formats", fmt, mode, axis, shape)
            bits = synthetic.gradient(8, *shape, 1e-4, 2.0) if mode == "sr" else \
                synthetic.activation(8, *shape, 0.01, 50.0)
            xd = to_dev(bits)
            g = osc.amax(bits)
            amax = None if fmt == "e8m0" else _amax_dev(bits)
            p, s, d = ue.quantize_1d(xd, axis, amax, 448.0, mode, seed=2, tensor_id=5, fmt=fmt)
            po, so, do = oq.quantize_1d(bits, axis, g, 448.0, mode, 2, 5, fmt=fmt)
            assert np.array_equal(host(s), so), (fmt, mode, axis, shape)
            assert np.array_equal(host(p), po), (fmt, mode, axis, shape)
            assert np.float32(d.item()) == do


@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_quantize_tiles_e4m3(mode):
    for shape in [(16, 16), (48, 80), (512, 1024), (208, 4096)]:
        say("tiles e4m3", mode, shape)
        bits = synthetic.weight(9, *shape)
        xd = to_dev(bits)
        p, s, pt, d, stt = ue.quantize_2d(xd, _amax_dev(bits), 448.0, mode, seed=4, tensor_id=6, fmt="e4m3")
        po, so, pto, do = oq.quantize_2d(bits, osc.amax(bits), 448.0, mode, 4, 6, fmt="e4m3")
        assert np.array_equal(host(s), so) and np.array_equal(host(p), po)
        assert np.array_equal(host(pt), pto) and np.array_equal(host(stt), so.T)
        assert np.float32(d.item()) == do


@pytest.mark.parametrize("fmt,g", [("e4m3", 1.0), ("e4m3", 3.0e4), ("e4m3", 2.0 ** -20), ("e8m0", 0.0)])
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_every_bf16_value(fmt, g, mode):
    """Every non-NaN bf16 value through the rows and columns quantizers (and
    the E4M3 tiles), under held references below, inside and above range."""
    say("every bf16 value", fmt, g, mode)
    bits = _all_bf16(256, 512, 23)
    xd = to_dev(bits)
    amax = None
    if fmt != "e8m0":
        amax = torch.zeros(1, dtype=torch.float32, device="cuda")
        set_amax(amax, g)
    for axis in [1, 0]:
        p, s, d = ue.quantize_1d(xd, axis, amax, 448.0, mode, seed=13, tensor_id=3, fmt=fmt)
        po, so, do = oq.quantize_1d(bits, axis, np.float32(g), 448.0, mode, 13, 3, fmt=fmt)
        assert np.array_equal(host(s), so), axis
        assert np.array_equal(host(p), po), axis
        assert np.float32(d.item()) == do
    if fmt == "e4m3":
        p, s, pt, d, st = ue.quantize_2d(xd, amax, 448.0, mode, seed=13, tensor_id=4, fmt=fmt)
        po, so, pto, do = oq.quantize_2d(bits, np.float32(g), 448.0, mode, 13, 4, fmt=fmt)
        assert np.array_equal(host(s), so) and np.array_equal(host(p), po)
        assert np.array_equal(host(pt), pto)


def _three(fmt, T, K, N, seed=0, out_dtype=torch.float32):
    """fprop, dgrad and wgrad on oracle-quantized operands of one format."""
    x = synthetic.activation(seed, T, K, 1e-2, 50.0)
    w = synthetic.weight(seed, N, K)
    dy = synthetic.gradient(seed, T, N, 1e-3, 1.0)
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    q = lambda b, axis, g, mode="rn", tid=0: oq.quantize_1d(b, axis, g, 448.0, mode, 1, tid, fmt=fmt)
    dec = lambda r, axis: oq.decoded_1d(r[0], r[1], axis, fmt=fmt)
    xr, xc = q(x, 1, gx), q(x, 0, gx)
    dr, dc = q(dy, 1, gd, "sr", 1), q(dy, 0, gd, "sr", 2)
    D = f32_scalar_dev
    X, Xc, dY, dYc = dec(xr, 1), dec(xc, 0), dec(dr, 1), dec(dc, 0)
    if fmt == "e8m0":
        # W in 1D blocks of 32 along each product's contraction
        wr, wc = q(w, 1, gw), q(w, 0, gw)
        Wf, Wd = dec(wr, 1), dec(wc, 0)
        bf = (wr[0], wr[1], wr[2])
        bd = (wc[0], wc[1], wc[2])
    else:
        wq = oq.quantize_2d(w, gw, fmt=fmt)
        Wf = Wd = oq.decoded_2d(wq[0], wq[1], fmt=fmt)
        bf = (wq[0], wq[1], wq[3])
        bd = (wq[2], wq[1].T, wq[3])
    U = u8_to_dev
    out = {}
    al = ogemm.alpha(xr[2], bf[2])
    c = ue.gemm("nt", T, N, K, U(xr[0]), U(xr[1]), D(xr[2]), U(bf[0]), U(bf[1]), D(bf[2]),
                out_dtype=out_dtype, fmt=fmt)
    out["fprop"] = (c, ogemm.fprop(X, Wf, al), ogemm.abs_product(X, Wf), al, K)
    al = ogemm.alpha(dr[2], bd[2])
    c = ue.gemm("nn", T, K, N, U(dr[0]), U(dr[1]), D(dr[2]), U(bd[0]), U(bd[1]), D(bd[2]),
                out_dtype=out_dtype, fmt=fmt)
    out["dgrad"] = (c, ogemm.dgrad(dY, Wd, al), ogemm.abs_product(dY, Wd.T), al, N)
    al = ogemm.alpha(dc[2], xc[2])
    c = ue.gemm("tn", N, K, T, U(dc[0]), U(dc[1]), D(dc[2]), U(xc[0]), U(xc[1]), D(xc[2]),
                out_dtype=out_dtype, fmt=fmt)
    out["wgrad"] = (c, ogemm.wgrad(dYc, Xc, al), ogemm.abs_product(dYc.T, Xc.T), al, T)
    return out


@pytest.mark.parametrize("T,K,N", [(64, 128, 64), (144, 208, 272), (256, 512, 384), (96, 192, 320)])
def test_gemm_e4m3(T, K, N):
    say("gemm e4m3", T, K, N)
    for name, (c, ref, ap, al, kk) in _three("e4m3", T, K, N).items():
        gemm_check(host(c), ref, al, ap, kk, f"e4m3 {name} {T}x{K}x{N}")


@pytest.mark.parametrize("T,K,N", [(256, 256, 256), (256, 512, 512), (512, 1024, 256), (768, 256, 512),
                                   (512, 768, 1280)])
def test_gemm_e8m0(T, K, N):
    say("gemm e8m0", T, K, N)
    for name, (c, ref, ap, al, kk) in _three("e8m0", T, K, N).items():
        gemm_check(host(c), ref, al, ap, kk, f"e8m0 {name} {T}x{K}x{N}")


def test_gemm_e8m0_ragged_and_bf16():
    """M and N not multiples of the 256 x 256 tile; bf16 output within one
    bf16 ulp of the fp32 reference."""
    say("gemm e8m0 ragged")
    M, N, K = 300, 200, 512
    a = synthetic.activation(21, M, K, 1e-2, 50.0)
    b = synthetic.weight(21, N, K)
    ar = oq.quantize_1d(a, 1, 0.0, fmt="e8m0")
    br = oq.quantize_1d(b, 1, 0.0, fmt="e8m0")
    A, B = oq.decoded_1d(ar[0], ar[1], 1, fmt="e8m0"), oq.decoded_1d(br[0], br[1], 1, fmt="e8m0")
    ref, ap = ogemm.fprop(A, B, 1.0), ogemm.abs_product(A, B)
    args = (u8_to_dev(ar[0]), u8_to_dev(ar[1]), f32_scalar_dev(1.0),
            u8_to_dev(br[0]), u8_to_dev(br[1]), f32_scalar_dev(1.0))
    c = ue.gemm("nt", M, N, K, *args, fmt="e8m0")
    gemm_check(host(c), ref, 1.0, ap, K, "e8m0 ragged fp32")
    c16 = ue.gemm("nt", M, N, K, *args, out_dtype=torch.bfloat16, fmt="e8m0").float().cpu().numpy()
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
    assert np.all(np.abs(c16.astype(np.float64) - ref) <= ulp * 1.01 + 1e-30)


def test_gemm_e8m0_split_and_persistent():
    """272 tiles (a split partial last wave, workgroups running a whole tile
    and a part) and 456 tiles (two whole tiles per workgroup)."""
    for M, N, K in [(4096, 4352, 1024), (4864, 6144, 512)]:
        say("gemm e8m0 persistent", M, N, K)
        a = synthetic.activation(23, M, K, 1e-2, 50.0)
        b = synthetic.weight(23, N, K)
        ar = oq.quantize_1d(a, 1, 0.0, fmt="e8m0")
        br = oq.quantize_1d(b, 1, 0.0, fmt="e8m0")
        A, B = oq.decoded_1d(ar[0], ar[1], 1, fmt="e8m0"), oq.decoded_1d(br[0], br[1], 1, fmt="e8m0")
        c = ue.gemm("nt", M, N, K, u8_to_dev(ar[0]), u8_to_dev(ar[1]), f32_scalar_dev(1.0),
                    u8_to_dev(br[0]), u8_to_dev(br[1]), f32_scalar_dev(1.0), fmt="e8m0")
        gemm_check(host(c), ogemm.fprop(A, B, 1.0), 1.0, ogemm.abs_product(A, B), K, f"e8m0 {M}x{N}x{K}")


def test_quantizers_feed_gemm_end_to_end():
    """GPU quantizers then GPU GEMMs for both formats equal the oracle's
    quantize-then-GEMM (the quantizers are bit-exact, so the operands are)."""
    T, K, N = 256, 512, 384
    x = synthetic.activation(31, T, K, 1e-2, 50.0)
    w = synthetic.weight(31, N, K)
    for fmt in ["e4m3", "e8m0"]:
        say("end to end", fmt)
        xd, wd = to_dev(x), to_dev(w)
        ax = None if fmt == "e8m0" else _amax_dev(x)
        aw = None if fmt == "e8m0" else _amax_dev(w)
        xr = ue.quantize_1d(xd, 1, ax, fmt=fmt)
        if fmt == "e8m0":
            wq = ue.quantize_1d(wd, 1, aw, fmt=fmt)
            b = (wq[0], wq[1], wq[2])
            wo = oq.quantize_1d(w, 1, 0.0, fmt=fmt)
            W = oq.decoded_1d(wo[0], wo[1], 1, fmt=fmt)
            dw = wo[2]
        else:
            wq = ue.quantize_2d(wd, aw, fmt=fmt)
            b = (wq[0], wq[1], wq[3])
            wo = oq.quantize_2d(w, osc.amax(w), fmt=fmt)
            W = oq.decoded_2d(wo[0], wo[1], fmt=fmt)
            dw = wo[3]
        xo = oq.quantize_1d(x, 1, osc.amax(x), fmt=fmt)
        X = oq.decoded_1d(xo[0], xo[1], 1, fmt=fmt)
        c = ue.gemm("nt", T, N, K, xr[0], xr[1], xr[2], *b, fmt=fmt)
        al = ogemm.alpha(xo[2], dw)
        gemm_check(host(c), ogemm.fprop(X, W, al), al, ogemm.abs_product(X, W), K, f"{fmt} end to end")


# ------------------------------------------------ both axes in one pass ----
@pytest.mark.parametrize("fmt", ["ue5m3", "e4m3"])
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_quantize_dual_equals_both_axes(fmt, mode):
    """ue5m3_quantize_dual writes exactly the axis-1 result (words keyed on
    tensor_id_r) and the transposed axis-0 result (tensor_id_c).  1024 x 8192
    (512 tiles of 128 x 128) takes the superblock walk of the tiles."""
    for shape in [(16, 16), (48, 80), (128, 128), (256, 512), (208, 4096), (400, 1040), (1024, 8192)]:
        say("dual", fmt, mode, shape)
        bits = synthetic.gradient(12, *shape, 1e-4, 2.0) if mode == "sr" else \
            synthetic.activation(12, *shape, 0.01, 50.0)
        xd = to_dev(bits)
        g = osc.amax(bits)
        (pr, sr_, d), (pc, sc, _) = ue.quantize_dual(xd, _amax_dev(bits), 448.0, mode, seed=5,
                                                     tensor_id_r=1, tensor_id_c=2, fmt=fmt)
        por, sor, do = oq.quantize_1d(bits, 1, g, 448.0, mode, 5, 1, fmt=fmt)
        poc, soc, _ = oq.quantize_1d(bits, 0, g, 448.0, mode, 5, 2, fmt=fmt)
        assert np.array_equal(host(sr_), sor) and np.array_equal(host(pr), por), (shape, "rows")
        assert np.array_equal(host(sc), soc) and np.array_equal(host(pc), poc), (shape, "cols")
        assert np.float32(d.item()) == do


@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_quantize_dual_every_bf16_value(mode):
    say("dual every bf16 value", mode)
    bits = _all_bf16(256, 512, 29)
    xd = to_dev(bits)
    for g in [1.0, 3.0e4, 2.0 ** -20]:
        amax = torch.zeros(1, dtype=torch.float32, device="cuda")
        set_amax(amax, g)
        (pr, sr_, _), (pc, sc, _) = ue.quantize_dual(xd, amax, 448.0, mode, seed=17, tensor_id_r=3,
                                                     tensor_id_c=4)
        por, sor, _ = oq.quantize_1d(bits, 1, np.float32(g), 448.0, mode, 17, 3)
        poc, soc, _ = oq.quantize_1d(bits, 0, np.float32(g), 448.0, mode, 17, 4)
        assert np.array_equal(host(sr_), sor) and np.array_equal(host(pr), por), g
        assert np.array_equal(host(sc), soc) and np.array_equal(host(pc), poc), g
