"""GPU parity of the decoded-operand FP4 GEMM (fprop NT, dgrad NN, wgrad TN)
against the oracle, through the C ABI.  The operands are quantized by the
ORACLE and uploaded, so the GEMM is checked in isolation; the bar is the
1e-3 max relative error plus the elementwise fp32 accumulation bound of
tests/gpu_util.gemm_check."""

import numpy as np
import pytest
import torch

import paper_2609_02846_amd as ue
import synthetic
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc
from tests.gpu_util import (f32_scalar_dev, gemm_check, host, oracle_cols, oracle_rows,
                            ref_product, row_elem_index, say, to_dev, u8_to_dev)

pytestmark = pytest.mark.gpu


def _linear(seed, T, K, N, dy_std=1e-3):
    x = synthetic.activation(seed, T, K, 1e-2, 50.0)
    w = synthetic.weight(seed, N, K)
    dy = synthetic.gradient(seed, T, N, dy_std, 1.0)
    return x, w, dy


def _run_three(T, K, N, seed=0, out_dtype=torch.float32):
    x, w, dy = _linear(seed, T, K, N)
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    xr = oq.quantize_1d(x, 1, gx)
    xc = oq.quantize_1d(x, 0, gx)
    wq = oq.quantize_2d(w, gw)
    dr = oq.quantize_1d(dy, 1, gd, 448.0, "sr", 1, 1)
    dc = oq.quantize_1d(dy, 0, gd, 448.0, "sr", 1, 2)
    X, Xc = oq.decoded_1d(xr[0], xr[1], 1), oq.decoded_1d(xc[0], xc[1], 0)
    W = oq.decoded_2d(wq[0], wq[1])
    dY, dYc = oq.decoded_1d(dr[0], dr[1], 1), oq.decoded_1d(dc[0], dc[1], 0)
    D = lambda v: f32_scalar_dev(v)
    out = {}
    # fprop: Y = X W^T
    al = ogemm.alpha(xr[2], wq[3])
    c = ue.gemm("nt", T, N, K, u8_to_dev(xr[0]), u8_to_dev(xr[1]), D(xr[2]),
                u8_to_dev(wq[0]), u8_to_dev(wq[1]), D(wq[3]), out_dtype=out_dtype)
    out["fprop"] = (c, ogemm.fprop(X, W, al), ogemm.abs_product(X, W), al, K)
    # dgrad: dX = dY W   (B operand = transposed weight payload and tile scales)
    al = ogemm.alpha(dr[2], wq[3])
    c = ue.gemm("nn", T, K, N, u8_to_dev(dr[0]), u8_to_dev(dr[1]), D(dr[2]),
                u8_to_dev(wq[2]), u8_to_dev(wq[1].T), D(wq[3]), out_dtype=out_dtype)
    out["dgrad"] = (c, ogemm.dgrad(dY, W, al), ogemm.abs_product(dY, W.T), al, N)
    # wgrad: dW = dY^T X  (both operands re-blocked along tokens)
    al = ogemm.alpha(dc[2], xc[2])
    c = ue.gemm("tn", N, K, T, u8_to_dev(dc[0]), u8_to_dev(dc[1]), D(dc[2]),
                u8_to_dev(xc[0]), u8_to_dev(xc[1]), D(xc[2]), out_dtype=out_dtype)
    out["wgrad"] = (c, ogemm.wgrad(dYc, Xc, al), ogemm.abs_product(dYc.T, Xc.T), al, T)
    return out


@pytest.mark.parametrize("T,K,N", [(16, 16, 16), (48, 80, 48), (64, 128, 64), (128, 256, 128),
                                   (144, 208, 272), (256, 512, 384), (512, 1024, 256),
                                   # odd numbers of 64-wide K slices (1, 3, 5, 7)
                                   (96, 192, 320), (192, 64, 448)])
def test_three_products(T, K, N):
    say("gemm three products", T, K, N)
    for name, (c, ref, ap, al, kk) in _run_three(T, K, N).items():
        gemm_check(host(c), ref, al, ap, kk, f"{name} {T}x{K}x{N}")


def test_ragged_m_and_n():
    """M not a multiple of the tile (fprop rows), N ragged for wgrad."""
    say("gemm ragged")
    for M, N, K in [(37, 48, 80), (130, 144, 48), (1, 16, 16), (200, 16, 1024)]:
        a = synthetic.activation(3, M, K, 1e-2, 50.0)
        w = synthetic.weight(3, N, K)
        ar = oq.quantize_1d(a, 1, osc.amax(a))
        wq = oq.quantize_2d(w, osc.amax(w))
        A, W = oq.decoded_1d(ar[0], ar[1], 1), oq.decoded_2d(wq[0], wq[1])
        al = ogemm.alpha(ar[2], wq[3])
        c = ue.gemm("nt", M, N, K, u8_to_dev(ar[0]), u8_to_dev(ar[1]), f32_scalar_dev(ar[2]),
                    u8_to_dev(wq[0]), u8_to_dev(wq[1]), f32_scalar_dev(wq[3]))
        gemm_check(host(c), ogemm.fprop(A, W, al), al, ogemm.abs_product(A, W), K, f"nt {M}x{N}x{K}")
    # TN with N not a multiple of 16 (row-scaled B); K = 64 and K = 512; the
    # last case has N % 4 == 2, so its output rows end inside a run of 4
    for T, Mo, No in [(64, 40, 24), (512, 300, 40), (512, 300, 42)]:
        dy = synthetic.gradient(4, T, Mo, 1e-3, 1.0)
        x = synthetic.activation(4, T, No, 1e-2, 50.0)
        dc = oq.quantize_1d(dy, 0, osc.amax(dy), 448.0, "sr", 1, 2)
        xc = oq.quantize_1d(x, 0, osc.amax(x))
        dYc, Xc = oq.decoded_1d(dc[0], dc[1], 0), oq.decoded_1d(xc[0], xc[1], 0)
        al = ogemm.alpha(dc[2], xc[2])
        c = ue.gemm("tn", Mo, No, T, u8_to_dev(dc[0]), u8_to_dev(dc[1]), f32_scalar_dev(dc[2]),
                    u8_to_dev(xc[0]), u8_to_dev(xc[1]), f32_scalar_dev(xc[2]))
        gemm_check(host(c), ogemm.wgrad(dYc, Xc, al), al, ogemm.abs_product(dYc.T, Xc.T), T,
                   f"tn ragged {Mo}x{No}x{T}")
    # bf16 output with N % 8 == 4 and N % 4 == 2 (the narrower store paths)
    for T, Mo, No in [(512, 300, 44), (512, 300, 42)]:
        dy = synthetic.gradient(5, T, Mo, 1e-3, 1.0)
        x = synthetic.activation(5, T, No, 1e-2, 50.0)
        dc = oq.quantize_1d(dy, 0, osc.amax(dy), 448.0, "sr", 1, 2)
        xc = oq.quantize_1d(x, 0, osc.amax(x))
        dYc, Xc = oq.decoded_1d(dc[0], dc[1], 0), oq.decoded_1d(xc[0], xc[1], 0)
        al = ogemm.alpha(dc[2], xc[2])
        c = ue.gemm("tn", Mo, No, T, u8_to_dev(dc[0]), u8_to_dev(dc[1]), f32_scalar_dev(dc[2]),
                    u8_to_dev(xc[0]), u8_to_dev(xc[1]), f32_scalar_dev(xc[2]), out_dtype=torch.bfloat16)
        ref = ogemm.wgrad(dYc, Xc, al)
        c16 = c.float().cpu().numpy().astype(np.float64)
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
        assert np.all(np.abs(c16 - ref) <= ulp * 1.01 + 1e-30), f"tn bf16 {Mo}x{No}x{T}"


def test_k_zero_writes_zeros():
    say("gemm K=0")
    c = torch.full((8, 16), 7.0, device="cuda")
    one = f32_scalar_dev(1.0)
    dummy = torch.zeros(16, dtype=torch.uint8, device="cuda")
    ue.gemm("nt", 8, 16, 0, dummy, dummy, one, dummy, dummy, one, out=c)
    torch.cuda.synchronize()
    assert (host(c) == 0).all()


def test_bf16_output_within_one_ulp():
    say("gemm bf16 output")
    res32 = _run_three(128, 256, 128, seed=2)
    res16 = _run_three(128, 256, 128, seed=2, out_dtype=torch.bfloat16)
    for name in res32:
        c16 = res16[name][0].float().cpu().numpy().astype(np.float64)
        ref = res32[name][1]
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
        assert np.all(np.abs(c16 - ref) <= ulp * 1.01 + 1e-30), name


def test_gemm_on_gpu_quantized_operands_matches():
    """End to end on the GPU path: quantizers then GEMMs, compared with the
    oracle's quantize-then-GEMM (quantizers are bit-exact, so the operands
    are identical)."""
    say("end-to-end linear step small")
    T, K, N = 256, 384, 512
    x, w, dy = _linear(9, T, K, N)
    xd, wd, dyd = to_dev(x), to_dev(w), to_dev(dy)
    sx, sw, sd = ue.AmaxState(1), ue.AmaxState(1), ue.AmaxState(1)
    for st, t in [(sx, xd), (sw, wd), (sd, dyd)]:
        ue.amax_sample(st, t, 0)
    xr = ue.quantize_1d(xd, 1, sx.amax)
    xc = ue.quantize_1d(xd, 0, sx.amax)
    wq = ue.quantize_2d(wd, sw.amax)
    dr = ue.quantize_1d(dyd, 1, sd.amax, 448.0, "sr", 1, 1)
    dc = ue.quantize_1d(dyd, 0, sd.amax, 448.0, "sr", 1, 2)
    y = ue.gemm("nt", T, N, K, xr[0], xr[1], xr[2], wq[0], wq[1], wq[3])
    dx = ue.gemm("nn", T, K, N, dr[0], dr[1], dr[2], wq[2], wq[4], wq[3])
    dw = ue.gemm("tn", N, K, T, dc[0], dc[1], dc[2], xc[0], xc[1], xc[2])
    ref = _run_three(T, K, N, seed=9)
    for name, c in [("fprop", y), ("dgrad", dx), ("wgrad", dw)]:
        _, r, ap, al, kk = ref[name]
        gemm_check(host(c), r, al, ap, kk, name)


def test_ffn_up_projection_sampled():
    """The Nemotron-H-8B FFN up-projection step (T=8192, K=4096, N=21504):
    full GPU path, outputs compared with the oracle on sampled rows and
    columns of each product."""
    T, K, N = 8192, 4096, 21504
    say("ffn up-projection full size", T, K, N)
    wl = synthetic.ffn_step(0, T, K, N)
    x, w, dy = wl["x"], wl["w"], wl["dy"]
    xd, wd, dyd = to_dev(x), to_dev(w), to_dev(dy)
    sx, sw, sd = ue.AmaxState(50), ue.AmaxState(50), ue.AmaxState(50)
    for st, t in [(sx, xd), (sw, wd), (sd, dyd)]:
        assert ue.amax_sample(st, t, 0)
    xr = ue.quantize_1d(xd, 1, sx.amax)
    xc = ue.quantize_1d(xd, 0, sx.amax)
    wq = ue.quantize_2d(wd, sw.amax)
    dr = ue.quantize_1d(dyd, 1, sd.amax, 448.0, "sr", 1, 1)
    dc = ue.quantize_1d(dyd, 0, sd.amax, 448.0, "sr", 1, 2)
    y = ue.gemm("nt", T, N, K, xr[0], xr[1], xr[2], wq[0], wq[1], wq[3])
    dx = ue.gemm("nn", T, K, N, dr[0], dr[1], dr[2], wq[2], wq[4], wq[3])
    dw = ue.gemm("tn", N, K, T, dc[0], dc[1], dc[2], xc[0], xc[1], xc[2])
    torch.cuda.synchronize()
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    assert np.float32(sx.amax.item()) == gx and np.float32(sw.amax.item()) == gw
    assert np.float32(sd.amax.item()) == gd
    rng = np.random.default_rng(1)
    rows = np.sort(np.concatenate([[0, T - 1], rng.choice(T, 30, replace=False)]))
    # fprop rows x sampled tile-rows of W
    wt = np.sort(rng.choice(N // 16, 8, replace=False))
    ncols = (wt[:, None] * 16 + np.arange(16)).ravel()
    xo = oracle_rows(x, rows, gx, 448.0, "rn", 0, 0)
    Xs = oq.decoded_1d(xo[0], xo[1], 1)
    Ws = np.concatenate([oq.decoded_2d(*oq.quantize_2d(w[16 * t:16 * t + 16], gw)[:2]) for t in wt])
    al = ogemm.alpha(xo[2], oq.quantize_2d(w[:16], gw)[3])
    gemm_check(host(y)[rows][:, ncols], ogemm.fprop(Xs, Ws, al), al, ogemm.abs_product(Xs, Ws), K,
               "fprop sampled")
    # dgrad rows x sampled tile-columns of W (all of N)
    kt = np.sort(rng.choice(K // 16, 3, replace=False))
    kcols = (kt[:, None] * 16 + np.arange(16)).ravel()
    dro = oracle_rows(dy, rows, gd, 448.0, "sr", 1, 1)
    dYs = oq.decoded_1d(dro[0], dro[1], 1)
    Wk = np.concatenate([oq.decoded_2d(*oq.quantize_2d(np.ascontiguousarray(w[:, 16 * t:16 * t + 16]), gw)[:2])
                         for t in kt], axis=1)                        # [N, 48]
    al = ogemm.alpha(dro[2], oq.quantize_2d(w[:16], gw)[3])
    gemm_check(host(dx)[rows][:, kcols], ogemm.dgrad(dYs, Wk, al), al,
               ogemm.abs_product(dYs, Wk.T), N, "dgrad sampled")
    # wgrad sampled rows (dY columns) x sampled columns (X columns)
    nsel = np.sort(rng.choice(N, 24, replace=False))
    ksel = np.sort(rng.choice(K, 24, replace=False))
    dco = oracle_cols(dy, nsel, gd, 448.0, "sr", 1, 2)
    xco = oracle_cols(x, ksel, gx, 448.0, "rn", 0, 0)
    dYc = oq.decoded_1d(dco[0], dco[1], 0)                            # [T, 24]
    Xc = oq.decoded_1d(xco[0], xco[1], 0)                             # [T, 24]
    al = ogemm.alpha(dco[2], xco[2])
    gemm_check(host(dw)[nsel][:, ksel], ogemm.wgrad(dYc, Xc, al), al,
               ogemm.abs_product(dYc.T, Xc.T), T, "wgrad sampled")


def test_split_tail_tiles():
    """A partial last wave of tiles: 16 x 17 = 272 tiles of 256 x 256 on 256
    CUs leave 16 tiles, which run split along K (2 parts of 2 stages each)
    and are summed by the second kernel; 32 workgroups run a whole tile and
    then a part.  Every output is compared."""
    say("gemm split tail")
    M, N, K = 4096, 4352, 1024
    a = synthetic.activation(13, M, K, 1e-2, 50.0)
    w = synthetic.weight(13, N, K)
    ar = oq.quantize_1d(a, 1, osc.amax(a))
    wq = oq.quantize_2d(w, osc.amax(w))
    A, W = oq.decoded_1d(ar[0], ar[1], 1), oq.decoded_2d(wq[0], wq[1])
    al = ogemm.alpha(ar[2], wq[3])
    ref, ap = ogemm.fprop(A, W, al), ogemm.abs_product(A, W)
    for out_dtype in [torch.float32, torch.bfloat16]:
        for rep in range(2):          # the workspace is reused by the second call
            c = ue.gemm("nt", M, N, K, u8_to_dev(ar[0]), u8_to_dev(ar[1]), f32_scalar_dev(ar[2]),
                        u8_to_dev(wq[0]), u8_to_dev(wq[1]), f32_scalar_dev(wq[3]), out_dtype=out_dtype)
            if out_dtype == torch.float32:
                gemm_check(host(c), ref, al, ap, K, f"split nt fp32 call {rep}")
            else:
                c16 = c.float().cpu().numpy().astype(np.float64)
                ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
                assert np.all(np.abs(c16 - ref) <= ulp * 1.01 + 1e-30), rep


def test_persistent_several_tiles_per_workgroup():
    """19 x 24 = 456 tiles on 256 CUs: the leftover 200 tiles are too many to
    split, so 200 workgroups run two whole tiles each, the second one's first
    stages loaded during the first one's last.  Every output is compared."""
    say("gemm persistent")
    M, N, K = 4864, 6144, 512
    a = synthetic.activation(17, M, K, 1e-2, 50.0)
    w = synthetic.weight(17, N, K)
    ar = oq.quantize_1d(a, 1, osc.amax(a))
    wq = oq.quantize_2d(w, osc.amax(w))
    A, W = oq.decoded_1d(ar[0], ar[1], 1), oq.decoded_2d(wq[0], wq[1])
    al = ogemm.alpha(ar[2], wq[3])
    ref, ap = ogemm.fprop(A, W, al), ogemm.abs_product(A, W)
    for out_dtype in [torch.float32, torch.bfloat16]:
        c = ue.gemm("nt", M, N, K, u8_to_dev(ar[0]), u8_to_dev(ar[1]), f32_scalar_dev(ar[2]),
                    u8_to_dev(wq[0]), u8_to_dev(wq[1]), f32_scalar_dev(wq[3]), out_dtype=out_dtype)
        if out_dtype == torch.float32:
            gemm_check(host(c), ref, al, ap, K, "persistent nt fp32")
        else:
            c16 = c.float().cpu().numpy().astype(np.float64)
            ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
            assert np.all(np.abs(c16 - ref) <= ulp * 1.01 + 1e-30)


def test_single_small_linear_fprop():
    """The single small linear (X [256, 512] N(0,1) with 1% x50 outliers,
    W [256, 512] N(0, 0.02), seed 0): current amax of each operand, X rows
    and W tiles by RN through the GPU quantizers, then the NT GEMM; payloads
    and scales bit-exact and every output to the GEMM bar."""
    say("single small linear fprop")
    wl = synthetic.linear_fprop_small(0)
    x, w = wl["x"], wl["w"]
    T, K = x.shape
    N = w.shape[0]
    xd, wd = to_dev(x), to_dev(w)
    sx, sw = ue.AmaxState(1), ue.AmaxState(1)
    assert ue.amax_sample(sx, xd, 0) and ue.amax_sample(sw, wd, 0)
    xr = ue.quantize_1d(xd, 1, sx.amax)
    wq = ue.quantize_2d(wd, sw.amax, transposed=False)
    for out_dtype in (torch.float32, torch.bfloat16):
        y = ue.gemm("nt", T, N, K, *xr, wq[0], wq[1], wq[3], out_dtype=out_dtype)
        torch.cuda.synchronize()
        gx, gw = osc.amax(x), osc.amax(w)
        xo, wo = oq.quantize_1d(x, 1, gx), oq.quantize_2d(w, gw)
        assert np.array_equal(host(xr[0]), xo[0]) and np.array_equal(host(xr[1]), xo[1])
        assert np.array_equal(host(wq[0]), wo[0]) and np.array_equal(host(wq[1]), wo[1])
        X, W = oq.decoded_1d(xo[0], xo[1], 1), oq.decoded_2d(wo[0], wo[1])
        al = ogemm.alpha(xo[2], wo[3])
        ref, ap = ogemm.fprop(X, W, al), ogemm.abs_product(X, W)
        if out_dtype == torch.float32:
            gemm_check(host(y), ref, al, ap, K, "small linear fprop")
        else:
            e = float(al) * K * 2.0 ** -23 * ap
            ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref) + e, 1e-30))) - 7)
            assert np.all(np.abs(host(y.float()).astype(np.float64) - ref) <= e + 1.01 * ulp + 1e-30)


@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_vector_epilogue_edges(out):
    """The staged whole-tile epilogue (bf16 with N % 8 == 0, fp32 with
    N % 4 == 0): output rows past M inside a 32-row round, 8-column (4-column)
    runs past N inside a 64-column (32-column) round, and more than one tile
    in each direction."""
    say("gemm vector epilogue edges", out)
    Ns = [8, 24, 40, 136, 264] if out == "bf16" else [4, 12, 36, 132, 260]
    for M, N, K in [(1, Ns[0], 64), (37, Ns[1], 128), (259, Ns[2], 256), (300, Ns[3], 512), (517, Ns[4], 256)]:
        a = synthetic.activation(6, M, K, 1e-2, 50.0)
        w = synthetic.weight(6, N, K)
        ar = oq.quantize_1d(a, 1, osc.amax(a))
        # row-scaled B keeps N free of the tile constraint (N % 16)
        wr = oq.quantize_1d(w, 1, osc.amax(w))
        A, W = oq.decoded_1d(ar[0], ar[1], 1), oq.decoded_1d(wr[0], wr[1], 1)
        al = ogemm.alpha(ar[2], wr[2])
        dt = torch.bfloat16 if out == "bf16" else torch.float32
        c = ue.gemm("nt", M, N, K, u8_to_dev(ar[0]), u8_to_dev(ar[1]), f32_scalar_dev(ar[2]),
                    u8_to_dev(wr[0]), u8_to_dev(wr[1]), f32_scalar_dev(wr[2]), out_dtype=dt,
                    a_blk=ue.ROW16, b_blk=ue.ROW16)
        ref = ogemm.fprop(A, W, al)
        got = c.float().cpu().numpy().astype(np.float64)
        if out == "bf16":
            ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
            assert np.all(np.abs(got - ref) <= ulp * 1.01 + 1e-30), f"bf16 {M}x{N}x{K}"
        else:
            gemm_check(got, ref, al, ogemm.abs_product(A, W), K, f"f32 {M}x{N}x{K}")


def test_bf16_small_m_wide_n():
    """bf16 output with few rows and very many columns (16 x 12582912, K =
    256: the register-decode kernel): the padded tile rows' byte offsets pass
    2^32 there, so the vector epilogue (which drops rows past M by their
    offset) must not be used.  B repeats a block of 768 random rows, so every
    output column equals one of 768 columns the oracle computes, and all
    201 million outputs are compared with it."""
    M, N, K, P = 16, 3 << 22, 256, 768
    say("gemm bf16 small M wide N", M, N, K)
    rng = np.random.default_rng(21)
    a = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    a_s = rng.integers(100, 130, (M, K // 16)).astype(np.uint8)
    bp = rng.integers(0, 256, (P, K // 2), dtype=np.uint8)
    bp_s = rng.integers(100, 130, (P, K // 16)).astype(np.uint8)
    b = u8_to_dev(bp).repeat(N // P, 1)
    b_s = u8_to_dev(bp_s).repeat(N // P, 1)
    dec = np.float32(1.0 / 64.0)
    c = ue.gemm("nt", M, N, K, u8_to_dev(a), u8_to_dev(a_s), f32_scalar_dev(dec), b, b_s,
                f32_scalar_dev(dec), out_dtype=torch.bfloat16, a_blk=ue.ROW16, b_blk=ue.ROW16)
    torch.cuda.synchronize()
    al = ogemm.alpha(dec, dec)
    ref = ogemm.fprop(oq.decoded_1d(a, a_s, 1), oq.decoded_1d(bp, bp_s, 1), al)      # [M, P]
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
    r = torch.from_numpy(ref).cuda()[:, None, :]
    tol = torch.from_numpy(ulp * 1.01 + 1e-30).cuda()[:, None, :]
    bad = (c.view(M, N // P, P).double() - r).abs() > tol
    assert not bool(bad.any()), f"{int(bad.sum())} outputs differ"


_SENTINEL = {torch.bfloat16: (torch.int16, 0x7FC1), torch.float32: (torch.int32, 0x7FC00001)}


def _random_operands(g, M, N, K, block, codes):
    lo, hi = codes
    a = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device="cuda", generator=g)
    a_s = torch.randint(lo, hi, (M, K // block), dtype=torch.uint8, device="cuda", generator=g)
    b = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device="cuda", generator=g)
    b_s = torch.randint(lo, hi, (N, K // block), dtype=torch.uint8, device="cuda", generator=g)
    return a, a_s, b, b_s


@pytest.mark.parametrize("entry,M,N,K,dt,fmt,block", [
    ("gemm", 300, 136, 512, "bf16", "ue5m3", 16),      # vector epilogue, bf16
    ("gemm", 300, 132, 512, "f32", "ue5m3", 16),       # vector epilogue, fp32
    ("gemm", 37, 140, 512, "bf16", "ue5m3", 16),       # per-element epilogue (N % 8 = 4)
    ("gemm", 37, 130, 512, "f32", "ue5m3", 16),        # per-element epilogue (N % 4 = 2)
    ("gemm", 4252, 4096, 1024, "bf16", "ue5m3", 16),   # split leftover tiles, ragged M
    ("gemm", 300, 136, 192, "bf16", "ue5m3", 16),      # K % 256 != 0: staged kernel
    ("gemm", 37, 40, 48, "f32", "ue5m3", 16),          # K % 64 != 0: general kernel
    ("gemm", 300, 136, 512, "bf16", "ue5m3", 32),      # blocks of 32
    ("gemm", 300, 136, 512, "bf16", "e8m0", 32),       # E8M0 scales
    ("gemm_pm", 300, 136, 512, "bf16", "ue5m3", 16),   # probe-matched
    ("gemm_pm", 37, 132, 512, "f32", "ue5m3", 16),
    ("gemm_noalloc", 300, 136, 512, "bf16", "ue5m3", 16),
])
def test_writes_exactly_c(entry, M, N, K, dt, fmt, block):
    """C lies inside a larger buffer filled with a NaN bit pattern that the
    product of finite operands never yields.  After one call every element of
    C has been written (none holds the pattern) and nothing before or after
    C has: the guard after C spans the rows of the padded 256-row tile grid
    past M and one more tile row, which holds every store a tile of C could
    address.  Covers ragged M inside a tile and inside an epilogue round, the
    vector and per-element epilogues, split leftover tiles, the staged and
    general kernels, blocks of 32, E8M0 scales and the probe-matched GEMM."""
    say("gemm writes exactly C", entry, M, N, K, dt, fmt, block)
    dt = torch.bfloat16 if dt == "bf16" else torch.float32
    g = torch.Generator(device="cuda").manual_seed(M * 7 + N)
    codes = (120, 131) if fmt == "e8m0" else (100, 131)
    a, a_s, b, b_s = _random_operands(g, M, N, K, block, codes)
    it, pat = _SENTINEL[dt]
    pre = 4096
    post = ((M + 255) // 256 * 256 - M + 256) * N
    buf = torch.full((pre + M * N + post,), pat, dtype=it, device="cuda")
    out = buf[pre:pre + M * N].view(dt).view(M, N)
    dec = f32_scalar_dev(1.0 / 64.0)
    kw = dict(out=out, a_blk=ue.ROW16 if block == 16 else ue.ROW32, b_blk=ue.ROW16 if block == 16 else ue.ROW32)
    if entry == "gemm":
        ue.gemm("nt", M, N, K, a, a_s, dec, b, b_s, dec, fmt=fmt, block=block, **kw)
    elif entry == "gemm_pm":
        ue.gemm_pm("nt", M, N, K, a, a_s, dec, b, b_s, dec, **kw)
    else:
        ue.gemm_noalloc("nt", M, N, K, a, a_s, dec, b, b_s, dec, **kw)
    torch.cuda.synchronize()
    assert bool((buf[:pre] == pat).all()), "written before C"
    assert bool((buf[pre + M * N:] == pat).all()), "written after C"
    assert not bool((buf[pre:pre + M * N] == pat).any()), "elements of C left unwritten"
    assert bool(torch.isfinite(out).all())
