"""Helpers shared by the GPU parity tests: device transfer of the seeded
inputs, oracle quantization of sampled parts of a tensor, GEMM tolerances."""

import sys

import numpy as np
import torch

from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc


def say(*msg):
    """Name the case on stdout before GPU work (a crash keeps the last line)."""
    print("[case]", *msg, flush=True)
    sys.stdout.flush()


def to_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def u8_to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()


def f32_scalar_dev(v):
    return torch.tensor([float(np.float32(v))], dtype=torch.float32, device="cuda")


def host(t):
    return t.detach().cpu().numpy()


def set_amax(dev_tensor, g):
    dev_tensor.fill_(float(np.float32(g)))


def row_elem_index(rows, ncols_total, col_ids=None):
    """Row-major source indices of the sub-matrix rows x col_ids."""
    rows = np.asarray(rows, np.int64)
    cols = np.arange(ncols_total, dtype=np.int64) if col_ids is None else np.asarray(col_ids, np.int64)
    return rows[:, None] * ncols_total + cols[None, :]


def oracle_rows(bits, rows, g, T, mode, seed, tid):
    """Oracle axis-1 quantization of the selected rows of ``bits``."""
    sub = bits[rows]
    idx = row_elem_index(rows, bits.shape[1])
    return oq.quantize_1d(sub, 1, g, T, mode, seed, tid, elem_index=idx)


def oracle_cols(bits, cols, g, T, mode, seed, tid):
    """Oracle axis-0 quantization of the selected columns (output rows of the
    transposed layout)."""
    sub = np.ascontiguousarray(bits[:, cols])
    idx = row_elem_index(np.arange(bits.shape[0]), bits.shape[1], cols)
    return oq.quantize_1d(sub, 0, g, T, mode, seed, tid, elem_index=idx)


def gemm_check(c_gpu, c_ref, al, absprod, K, what):
    """Parity bar for the decoded-operand GEMM (fp32 output):
    (1) max |C - C_ref| / max |C_ref| <= 1e-3;
    (2) |C - C_ref| / |C_ref| <= 1e-3 for every element with
        |C_ref| >= 1e-2 max |C_ref|;
    (3) elementwise |C - C_ref| <= alpha * K * 2^-23 * sum_k |A||B| +
        2^-23 |C_ref| (the fp32 accumulation bound with a 2x margin, plus the
        epilogue rounding), which catches a single wrong decoded element."""
    c_gpu = np.asarray(c_gpu, np.float64)
    err = np.abs(c_gpu - c_ref)
    scale = max(np.max(np.abs(c_ref)), 1e-300)
    rel = err.max() / scale
    assert rel <= 1e-3, f"{what}: max rel error {rel:.3e}"
    big = np.abs(c_ref) >= 1e-2 * scale
    if big.any():
        rel_big = np.max(err[big] / np.abs(c_ref[big]))
        assert rel_big <= 1e-3, f"{what}: elementwise rel error {rel_big:.3e} on an output >= 1% of the max"
    bound = float(al) * max(K, 1) * 2.0 ** -23 * absprod + 2.0 ** -23 * np.abs(c_ref) + 1e-38
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements beyond the fp32 accumulation bound, "
                           f"worst ratio {np.max(err / bound):.3g}")
    return rel


def ref_product(a_dec, b_dec_t, al):
    """alpha * A_dec B_dec^T in float64 and the sum of |products|."""
    return ogemm.fprop(a_dec, b_dec_t, al), ogemm.abs_product(a_dec, b_dec_t)
