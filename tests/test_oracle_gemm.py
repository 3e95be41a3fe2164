"""Pins of the oracle's decoded-operand GEMM (Sec. 5.1) for the three
products of a linear (Sec. 4.3): brute-force exact sums on tiny inputs,
orientation checks, special cases, and the exactness of the bf16 decode
that the GPU GEMM relies on."""

from fractions import Fraction

import numpy as np
import torch

import synthetic
from oracle import formats, gemm, quantize, scaling


def _quant_step(seed, t, k, n):
    x = synthetic.activation(seed, t, k, 0.05, 20.0)
    w = synthetic.weight(seed, n, k)
    dy = synthetic.gradient(seed, t, n, 1e-3, 1.0)
    gx, gw, gd = scaling.amax(x), scaling.amax(w), scaling.amax(dy)
    xr = quantize.quantize_1d(x, 1, gx)
    xc = quantize.quantize_1d(x, 0, gx)
    wq = quantize.quantize_2d(w, gw)
    dr = quantize.quantize_1d(dy, 1, gd, mode="sr", seed=1, tensor_id=1)
    dc = quantize.quantize_1d(dy, 0, gd, mode="sr", seed=1, tensor_id=2)
    return xr, xc, wq, dr, dc


def _exact(a):
    return [[Fraction(float(v)) for v in row] for row in np.asarray(a)]


def test_brute_force_three_products():
    T, K, N = 16, 32, 16
    xr, xc, wq, dr, dc = _quant_step(0, T, K, N)
    X = quantize.decoded_1d(xr[0], xr[1], 1)
    Xc = quantize.decoded_1d(xc[0], xc[1], 0)
    W = quantize.decoded_2d(wq[0], wq[1])
    dY = quantize.decoded_1d(dr[0], dr[1], 1)
    dYc = quantize.decoded_1d(dc[0], dc[1], 0)
    al = gemm.alpha(xr[2], wq[3])
    Xe, We, dYe, Xce, dYce = map(_exact, (X, W, dY, Xc, dYc))
    Y = gemm.fprop(X, W, al)
    dX = gemm.dgrad(dY, W, al)
    dW = gemm.wgrad(dYc, Xc, al)
    A = Fraction(float(al))
    for t in range(T):
        for j in range(N):
            assert Y[t, j] == float(A * sum(Xe[t][k] * We[j][k] for k in range(K)))
        for k in range(K):
            assert dX[t, k] == float(A * sum(dYe[t][j] * We[j][k] for j in range(N)))
    for j in range(N):
        for k in range(K):
            assert dW[j, k] == float(A * sum(dYce[t][j] * Xce[t][k] for t in range(T)))


def test_fp32_accumulation_close_to_exact():
    xr, xc, wq, dr, dc = _quant_step(1, 64, 256, 48)
    X = quantize.decoded_1d(xr[0], xr[1], 1)
    W = quantize.decoded_2d(wq[0], wq[1])
    al = gemm.alpha(xr[2], wq[3])
    y64 = gemm.fprop(X, W, al)
    y32 = gemm.fprop(X, W, al, accumulate="fp32")
    bound = float(al) * 256 * 2.0 ** -23 * gemm.abs_product(X, W)
    assert np.all(np.abs(y32 - y64) <= bound + 1e-30)


def test_identity_weight_returns_decoded_activation():
    # W = 2 * I (exact on the E2M1 grid with tile scale ...): Y = alpha X_dec W_dec.
    k = 64
    w = synthetic.f32_to_bf16_bits(np.eye(k, dtype=np.float32) * 2.0)
    x = synthetic.activation(3, 32, k)
    gx, gw = scaling.amax(x), scaling.amax(w)
    xr = quantize.quantize_1d(x, 1, gx)
    wq = quantize.quantize_2d(w, gw)
    W = quantize.decoded_2d(wq[0], wq[1])
    diag = np.diag(W)
    assert np.all(diag == diag[0]) and np.count_nonzero(W) == k
    X = quantize.decoded_1d(xr[0], xr[1], 1)
    al = gemm.alpha(xr[2], wq[3])
    assert np.array_equal(gemm.fprop(X, W, al), float(al) * diag[0] * X)


def test_decoded_products_exact_in_bf16():
    # Every E2M1 value times every finite UE5M3 scale is exact in bf16, so
    # dequantizing to bf16 before a bf16 matrix product loses nothing.
    q = formats.E2M1_MAG
    s = formats.UE5M3_FINITE
    prod = (q[:, None] * s[None, :]).ravel()
    prod = np.concatenate([prod, -prod])
    rt = torch.from_numpy(prod).to(torch.bfloat16).double().numpy()
    assert np.array_equal(rt, prod)
