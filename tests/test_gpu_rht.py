"""GPU parity of the randomized Hadamard transform of the wgrad operands
(ue5m3_amax_sample_rht, ue5m3_quantize_cols_rht) with the oracle
(oracle.rht): the transformed amax and the COL16 payload and scales are
bit-exact (RN and SR, several masks, column counts with 4 | C and 2 | C
only, several row groups); the FP4 Linear with rht_wgrad reproduces the
oracle's weight gradient on transformed operands; full-size sampled
columns of the FFN step."""

import numpy as np
import pytest
import torch

import synthetic
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import rht as orht
from oracle import scaling as osc
import paper_2609_02846_amd as ue
from paper_2609_02846_amd.linear import Linear
from tests.gpu_util import host, row_elem_index, say, to_dev
from tests.test_gpu_linear import bf16_check

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rows,cols", [(16, 8), (64, 48), (96, 34), (1040, 136), (2048, 4096)])
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_quantize_cols_rht_bit_exact(rows, cols, mode):
    mask = {16: 0x0001, 64: 0xFFFF, 96: 0x1234, 1040: 0xBEEF, 2048: 0x5A5A}[rows]
    say("quantize_cols_rht", rows, cols, mode, hex(mask))
    x = synthetic.activation(rows + cols, rows, cols, 1e-2, 40.0)
    xd = to_dev(x)
    st = ue.AmaxState(1)
    assert ue.amax_sample_rht(st, xd, mask, 0)
    p, s, d = ue.quantize_cols_rht(xd, st.amax, mask, 448.0, mode, 77, 9)
    torch.cuda.synchronize()
    g = orht.amax_rht(x, mask)
    assert np.float32(st.amax.item()) == g
    rp, rs, rd = orht.quantize_cols_rht(x, g, mask, 448.0, mode, 77, 9)
    assert np.array_equal(host(p), rp) and np.array_equal(host(s), rs)
    assert np.float32(d.item()) == rd


def test_amax_rht_outlier_and_held_reference():
    """An outlier spreads over its block: the transformed amax is the sum
    of |x|/4 over the block when signs align; the held reference is reused
    until the period ends."""
    x = np.zeros((32, 4), np.float32)
    x[:16, 1] = 2.0                                  # H16 row 0 sums the block: 16 * 2 / 4 = 8
    x[20, 2] = -100.0
    bits = synthetic.f32_to_bf16_bits(x)
    st = ue.AmaxState(3)
    xd = to_dev(bits)
    ue.amax_sample_rht(st, xd, 0, 0)
    torch.cuda.synchronize()
    assert st.amax.item() == 25.0 == orht.amax_rht(bits, 0)
    x[:16, 1] = 3.0                                  # 12 now, but held
    assert not ue.amax_sample_rht(st, to_dev(synthetic.f32_to_bf16_bits(x)), 0, 2)
    assert ue.amax_sample_rht(st, to_dev(synthetic.f32_to_bf16_bits(x)), 0, 3)


def test_linear_rht_wgrad_matches_oracle():
    """Linear with rht_wgrad: Y and dX as without the transform; dW equals
    the oracle's product of the transformed, quantized dY and X."""
    T, K, N = 272, 160, 144
    say("linear rht wgrad", T, K, N)
    x = synthetic.activation(21, T, K, 1e-2, 50.0)
    w = synthetic.weight(21, N, K)
    dy = synthetic.gradient(21, T, N, 1e-3, 1.0)
    layer = Linear(K, N, period=1, seed=9, layer_id=2, rht_wgrad=True, grad_rounding="sr")
    with torch.no_grad():
        layer.weight.copy_(to_dev(w))
    xd = to_dev(x).requires_grad_(True)
    y = layer(xd)
    y.backward(to_dev(dy))
    torch.cuda.synchronize()
    m = layer.rht_mask
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    gxt, gdt = orht.amax_rht(x, m), orht.amax_rht(dy, m)
    assert np.float32(layer.amax_xt.amax.item()) == gxt and np.float32(layer.amax_dyt.amax.item()) == gdt
    # fprop and dgrad are untouched by the transform
    xr, wq = oq.quantize_1d(x, 1, gx), oq.quantize_2d(w, gw)
    X, W = oq.decoded_1d(xr[0], xr[1], 1), oq.decoded_2d(wq[0], wq[1])
    al = ogemm.alpha(xr[2], wq[3])
    bf16_check(y, ogemm.fprop(X, W, al), al, ogemm.abs_product(X, W), K, "fprop")
    dr = oq.quantize_1d(dy, 1, gd, 448.0, "sr", 9, 5)
    dY = oq.decoded_1d(dr[0], dr[1], 1)
    al = ogemm.alpha(dr[2], wq[3])
    bf16_check(xd.grad, ogemm.dgrad(dY, W, al), al, ogemm.abs_product(dY, W.T), N, "dgrad")
    # wgrad on transformed operands (SR words of dY at their source positions)
    xc = orht.quantize_cols_rht(x, gxt, m, 448.0, "rn")
    dc = orht.quantize_cols_rht(dy, gdt, m, 448.0, "sr", 9, 6)
    Xc, dYc = oq.decoded_1d(xc[0], xc[1], 0), oq.decoded_1d(dc[0], dc[1], 0)
    al = ogemm.alpha(dc[2], xc[2])
    bf16_check(layer.weight.grad, ogemm.wgrad(dYc, Xc, al), al, ogemm.abs_product(dYc.T, Xc.T), T, "wgrad")


def test_ffn_wgrad_operands_sampled_columns():
    """FFN up-projection sizes: transformed amax of X (8192 x 4096) and dY
    (8192 x 21504) exact; sampled columns of their transformed COL16
    quantization bit-exact (SR words of dY by source position)."""
    T, K, N = 8192, 4096, 21504
    say("rht ffn sampled", T, K, N)
    wl = synthetic.ffn_step(0, T, K, N)
    m = 0x3C5A
    rng = np.random.default_rng(8)
    for name, bits, mode, tid in [("x", wl["x"], "rn", 0), ("dy", wl["dy"], "sr", 2)]:
        xd = to_dev(bits)
        st = ue.AmaxState(50)
        ue.amax_sample_rht(st, xd, m, 0)
        p, s, _ = ue.quantize_cols_rht(xd, st.amax, m, 448.0, mode, 5, tid)
        torch.cuda.synchronize()
        g = orht.amax_rht(bits, m)
        assert np.float32(st.amax.item()) == g, name
        cols = np.sort(rng.choice(bits.shape[1], 6, replace=False))
        sub = np.ascontiguousarray(bits[:, cols])
        idx = row_elem_index(np.arange(T), bits.shape[1], cols)
        rp, rs, _ = orht.quantize_cols_rht(sub, g, m, 448.0, mode, 5, tid, elem_index=idx)
        assert np.array_equal(host(p)[cols], rp) and np.array_equal(host(s)[cols], rs), name
        del xd, p, s
