"""Randomized Hadamard transform of the weight-gradient operands (oracle;
test infrastructure only).

Sec. 2 (the NVFP4 recipe's outlier techniques) and Table 6 (the "UE5M3 with
Transformer Engine settings" recipe): matched orthogonal transforms are
applied only to the saved activation X and the output gradient dY that feed
the weight-gradient GEMM, along its contraction dimension (tokens), before
quantization; since the transform is orthogonal, dY^T X is unchanged in
exact arithmetic while large coordinates are spread over their block.

Readings (the paper gives neither the size nor the sign generation):
* size 16, on every block of 16 consecutive rows (tokens) of each column --
  the COL16 quantization block of the wgrad operands;
* y = (1/4) H16 diag(s) x, H16[i][j] = (-1)^popcount(i & j) (Sylvester
  order), s_i = -1 where bit i of a 16-bit sign mask is set; the same mask
  for both operands (matched transforms), drawn by the caller;
* binary32 evaluation order: s_i x_i (exact), then four butterfly stages
  h = 1, 2, 4, 8, each replacing (u_i, u_{i+h}) for every i with bit h clear
  by (u_i + u_{i+h}, u_i - u_{i+h}) with one RNE rounding per operation,
  then the exact scaling by 1/4;
* the tensor reference of a transformed operand is the amax of the
  transformed tensor (current scaling in that recipe, D = 1).
"""

import numpy as np

from . import quantize, scaling


def hadamard16():
    """H16 with entries +-1 (Sylvester order)."""
    i = np.arange(16)
    pc = np.vectorize(lambda v: bin(v).count("1"))(i[:, None] & i[None, :])
    return np.where(pc % 2 == 0, 1, -1).astype(np.int64)


def signs(mask):
    """The diagonal of diag(s) for a 16-bit mask (float32 +-1)."""
    if mask < 0 or mask > 0xFFFF:
        raise ValueError("sign mask must fit 16 bits")
    return np.array([-1.0 if (mask >> i) & 1 else 1.0 for i in range(16)], np.float32)


def transform_cols(x, mask):
    """Transform every 16-row block of each column of a float32 [R, C]
    matrix (R % 16 == 0) in the binary32 order of the module header."""
    x = np.asarray(x, np.float32)
    R, C = x.shape
    if R % 16:
        raise ValueError("rows must be a multiple of 16")
    u = (x.reshape(R // 16, 16, C) * signs(mask)[None, :, None]).astype(np.float32)
    for h in (1, 2, 4, 8):
        lo = np.array([i for i in range(16) if not i & h])
        a, b = u[:, lo, :].copy(), u[:, lo + h, :].copy()
        u[:, lo, :] = (a + b).astype(np.float32)
        u[:, lo + h, :] = (a - b).astype(np.float32)
    return (u * np.float32(0.25)).astype(np.float32).reshape(R, C)


def amax_rht(x_bits, mask):
    """Tensor amax of the transformed bf16 matrix (float32, exact max)."""
    y = transform_cols(scaling.bf16_to_f32(x_bits), mask)
    return np.float32(np.max(np.abs(y))) if y.size else np.float32(0.0)


def quantize_cols_rht(x_bits, g, mask, target=448.0, mode="rn", seed=0, tensor_id=0, elem_index=None):
    """COL16 quantization (``quantize.quantize_1d`` axis 0 layout: payload
    [C, R/2], scales [C, R/16]) of the transformed bf16 matrix with held
    reference g (the transformed tensor's amax).  SR words follow each
    element's position (r, c) in the source tensor."""
    y = transform_cols(scaling.bf16_to_f32(x_bits), mask)
    return quantize.quantize_1d_values(y, 0, g, target, mode, seed, tensor_id, elem_index)
