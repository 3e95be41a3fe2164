"""Decoded-operand GEMM model (oracle; test infrastructure only).

Sec. 5.1 of the paper: the FP4 operands are decoded (E2M1 value times its
UE5M3 block scale, exact) and multiplied by a standard matrix product; the
tensor decode factors enter as one scalar alpha = dec_a * dec_b applied after
accumulation (Sec. 5.2: the encoded tensor-scale product is applied last).

For a linear Y = X W^T (Sec. 4.3) the three products are
    fprop  Y  = X  W^T      (contraction over K)
    dgrad  dX = dY W        (contraction over N)
    wgrad  dW = dY^T X      (contraction over T)
Each function takes the decoded operands in their logical shapes and returns
float64 results computed as alpha * (exact-as-float64 sum); ``accumulate=
"fp32"`` gives the binary32-accumulated product instead.
"""

import numpy as np


def alpha(dec_a, dec_b):
    """Binary32 product of the two tensor decode factors."""
    return np.float32(np.float32(dec_a) * np.float32(dec_b))


def _mm(a, b, accumulate):
    if accumulate == "fp64":
        return np.asarray(a, np.float64) @ np.asarray(b, np.float64)
    if accumulate == "fp32":
        return (np.asarray(a, np.float32) @ np.asarray(b, np.float32)).astype(np.float64)
    raise ValueError(accumulate)


def fprop(x_dec, w_dec, al, accumulate="fp64"):
    """Y[t, n] = alpha * sum_k X[t, k] W[n, k]."""
    return np.float64(al) * _mm(x_dec, np.asarray(w_dec).T, accumulate)


def dgrad(dy_dec, w_dec, al, accumulate="fp64"):
    """dX[t, k] = alpha * sum_n dY[t, n] W[n, k]."""
    return np.float64(al) * _mm(dy_dec, w_dec, accumulate)


def wgrad(dy_dec, x_dec, al, accumulate="fp64"):
    """dW[n, k] = alpha * sum_t dY[t, n] X[t, k]."""
    return np.float64(al) * _mm(np.asarray(dy_dec).T, x_dec, accumulate)


def abs_product(a_dec, b_dec_t):
    """sum_k |A[m, k]| |B[n, k]| (float64): the scale of the rounding error
    bound of any binary32 accumulation of the products."""
    return np.abs(np.asarray(a_dec, np.float64)) @ np.abs(np.asarray(b_dec_t, np.float64)).T
