"""FFN up-projection (T = 8192, K = 4096, N = 21504) at full size, parity on
whole outputs: the GPU quantizers as the bench step runs them (X both 1D
blockings from one read, W 16 x 16 tiles with the transposed copy, dY rows
and columns by SR) against the oracle on every payload byte and scale code
of every output; then 256 random rows of each product against the oracle
over all their columns, to the GEMM bar of tests/gpu_util.gemm_check.  The
fprop and dgrad GEMMs also run with the bf16 outputs the training step
writes: every element equals the bf16 rounding of the fp32 result, and the
sampled rows lie within one bf16 ulp of the oracle."""

import numpy as np
import pytest
import torch

import paper_2609_02846_amd as ue
import synthetic
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc
from tests.gpu_util import gemm_check, host, say, to_dev

pytestmark = pytest.mark.gpu


def _bf16_check(c_bf16, ref, bound, what):
    """bf16 output against the oracle's exact product: within the fp32
    accumulation bound plus one bf16 ulp of the result (the rounding of the
    fp32 value to bf16 is at most half an ulp)."""
    c = np.asarray(c_bf16, np.float64)
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref) + bound, 1e-30))) - 7)
    bad = np.abs(c - ref) > bound + ulp + 1e-30
    assert not bad.any(), f"{what}: {int(bad.sum())} outputs beyond one bf16 ulp plus the accumulation bound"


def test_ffn_up_projection_whole_outputs():
    T, K, N = 8192, 4096, 21504
    say("full-size parity", T, K, N)
    wl = synthetic.ffn_step(0, T, K, N)
    x, w, dy = wl["x"], wl["w"], wl["dy"]
    xd, wd, dyd = to_dev(x), to_dev(w), to_dev(dy)
    sx, sw, sd = ue.AmaxState(50), ue.AmaxState(50), ue.AmaxState(50)
    for st, t in [(sx, xd), (sw, wd), (sd, dyd)]:
        assert ue.amax_sample(st, t, 0)
    xr, xc = ue.quantize_dual(xd, sx.amax)
    wq = ue.quantize_2d(wd, sw.amax)
    dr = ue.quantize_1d(dyd, 1, sd.amax, 448.0, "sr", 1, 1)
    dc = ue.quantize_1d(dyd, 0, sd.amax, 448.0, "sr", 1, 2)
    y = ue.gemm("nt", T, N, K, *xr, wq[0], wq[1], wq[3])
    dx = ue.gemm("nn", T, K, N, *dr, wq[2], wq[4], wq[3])
    dw = ue.gemm("tn", N, K, T, *dc, xc[0], xc[1], xc[2])
    # the bf16-output instances the training step runs for fprop and dgrad
    y_bf = ue.gemm("nt", T, N, K, *xr, wq[0], wq[1], wq[3], out_dtype=torch.bfloat16)
    dx_bf = ue.gemm("nn", T, K, N, *dr, wq[2], wq[4], wq[3], out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    say("bf16 fprop and dgrad outputs: every element is the RNE of the fp32 result")
    # the two instances differ only in the store: same tiles, split plan and
    # accumulation order, so the bf16 output is exactly bf16(fp32 output)
    assert torch.equal(y_bf, y.to(torch.bfloat16))
    assert torch.equal(dx_bf, dx.to(torch.bfloat16))
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    assert (np.float32(sx.amax.item()), np.float32(sw.amax.item()), np.float32(sd.amax.item())) == (gx, gw, gd)

    say("X rows and columns, every byte")
    xro = oq.quantize_1d(x, 1, gx)
    assert np.array_equal(host(xr[1]), xro[1]) and np.array_equal(host(xr[0]), xro[0])
    assert np.float32(xr[2].item()) == xro[2]
    xco = oq.quantize_1d(x, 0, gx)
    assert np.array_equal(host(xc[1]), xco[1]) and np.array_equal(host(xc[0]), xco[0])

    say("W tiles and the transposed copy, every byte")
    wo = oq.quantize_2d(w, gw)
    assert np.array_equal(host(wq[1]), wo[1]) and np.array_equal(host(wq[4]), wo[1].T)
    assert np.array_equal(host(wq[0]), wo[0]) and np.array_equal(host(wq[2]), wo[2])
    assert np.float32(wq[3].item()) == wo[3]

    rng = np.random.default_rng(7)
    say("dY rows (SR), every byte")
    drows = np.arange(T)
    dro = oq.quantize_1d(dy, 1, gd, 448.0, "sr", 1, 1)
    assert np.array_equal(host(dr[1]), dro[1]) and np.array_equal(host(dr[0]), dro[0])
    say("dY columns (SR), every byte")
    dcols = np.arange(N)
    dco = oq.quantize_1d(dy, 0, gd, 448.0, "sr", 1, 2)
    assert np.array_equal(host(dc[1]), dco[1]) and np.array_equal(host(dc[0]), dco[0])

    say("fprop: 256 rows x all 21504 columns")
    W = oq.decoded_2d(wo[0], wo[1])                                   # [N, K]
    rows = np.sort(rng.choice(T, 256, replace=False))
    X = oq.decoded_1d(xro[0][rows], xro[1][rows], 1)
    al = ogemm.alpha(xro[2], wo[3])
    gemm_check(host(y[torch.from_numpy(rows).cuda()]), ogemm.fprop(X, W, al), al, ogemm.abs_product(X, W), K,
               "fprop 256 rows")

    say("fprop bf16 output: the same rows within one bf16 ulp of the oracle")
    _bf16_check(host(y_bf[torch.from_numpy(rows).cuda()].float()), ogemm.fprop(X, W, al),
                float(al) * K * 2.0 ** -23 * ogemm.abs_product(X, W), "fprop bf16")
    del X

    say("dgrad: 256 rows x all 4096 columns")
    pick = np.sort(rng.choice(len(drows), 256, replace=False))
    dY = oq.decoded_1d(dro[0][pick], dro[1][pick], 1)                 # [256, N]
    al = ogemm.alpha(dro[2], wo[3])
    Wt = np.ascontiguousarray(W.T)
    ref = ogemm.dgrad(dY, W, al)
    ap = ogemm.abs_product(dY, Wt)
    gemm_check(host(dx[torch.from_numpy(drows[pick]).cuda()]), ref, al, ap, N, "dgrad 256 rows")
    say("dgrad bf16 output: the same rows within one bf16 ulp of the oracle")
    _bf16_check(host(dx_bf[torch.from_numpy(drows[pick]).cuda()].float()), ref,
                float(al) * N * 2.0 ** -23 * ap, "dgrad bf16")
    del W, Wt, ref, ap

    say("wgrad: 256 rows x all 4096 columns")
    pick = np.sort(rng.choice(len(dcols), 256, replace=False))
    dYc = oq.decoded_1d(dco[0][pick], dco[1][pick], 0)                # [T, 256]
    Xc = oq.decoded_1d(xco[0], xco[1], 0)                             # [T, K]
    al = ogemm.alpha(dco[2], xco[2])
    gemm_check(host(dw[torch.from_numpy(dcols[pick]).cuda()]), ogemm.wgrad(dYc, Xc, al), al,
               ogemm.abs_product(np.ascontiguousarray(dYc.T), np.ascontiguousarray(Xc.T)), T, "wgrad 256 rows")
