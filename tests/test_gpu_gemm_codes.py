"""GPU parity of the decoded-operand GEMM on every block-scale code.

The realistic operands of the other GEMM tests use a narrow band of scale
codes.  Here the payload bytes are uniform (all 16 nibbles, -0 included) and
the block-scale codes run over every finite code of the format -- UE5M3
0x00..0xF7 (subnormals m 2^-17, the 0x08 boundary 2^-14, up to 61440; Sec. 3
and Table tab:scale-range) and E4M3 0x00..0x7E -- each code appearing many
times in both operands.  The products run through all three decode kernels
(K % 256 == 0: the persistent register-decode kernel; K % 64 == 0: the
staged kernel; K % 16 == 0: the general kernel) for the three layouts'
B-scale forms (tile scales for fprop and dgrad, row scales for wgrad).  The
operands are contraction-contiguous in every layout, so the reference is
alpha * A_hat B_hat^T of the oracle's decoded operands, checked to the GEMM
bar of tests/gpu_util.gemm_check."""

import numpy as np
import pytest
import torch

import paper_2609_02846_amd as ue
from oracle import gemm as ogemm
from oracle import quantize as oq
from tests.gpu_util import f32_scalar_dev, gemm_check, host, say, u8_to_dev

pytestmark = pytest.mark.gpu

LAST_CODE = {"ue5m3": 0xF7, "e4m3": 0x7E}


def _codes(rng, shape, fmt):
    """Every finite code of the format (the lowest ones when shape holds
    fewer), repeated and shuffled over shape."""
    n = int(np.prod(shape))
    ncodes = LAST_CODE[fmt] + 1
    c = np.arange(n) % ncodes
    rng.shuffle(c)
    return c.reshape(shape).astype(np.uint8)


@pytest.mark.parametrize("fmt", ["ue5m3", "e4m3"])
@pytest.mark.parametrize("layout", ["nt", "nn", "tn"])
@pytest.mark.parametrize("K", [512, 192, 80])
def test_every_scale_code(fmt, layout, K):
    M, N = 272, 288                         # two tile rows / columns, ragged
    rng = np.random.default_rng(11 + K)
    say("gemm every scale code", fmt, layout, M, N, K)
    a = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    b = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    a_s = _codes(rng, (M, K // 16), fmt)
    tiled = layout != "tn"
    b_s = _codes(rng, (N // 16, K // 16) if tiled else (N, K // 16), fmt)
    # every code occurs in A, and in B as far as its scale array holds them
    ncodes = LAST_CODE[fmt] + 1
    assert len(np.unique(a_s)) == ncodes and len(np.unique(b_s)) == min(b_s.size, ncodes)
    A = oq.decoded_1d(a, a_s, 1, fmt=fmt)                              # [M, K]
    B = oq.decoded_2d(b, b_s, fmt=fmt) if tiled else oq.decoded_1d(b, b_s, 1, fmt=fmt)
    dec_a, dec_b = np.float32(1.0 / 2688.0), np.float32(0.75 / 2688.0)
    al = ogemm.alpha(dec_a, dec_b)
    ref = ogemm.fprop(A, B, al)
    c = ue.gemm(layout, M, N, K, u8_to_dev(a), u8_to_dev(a_s), f32_scalar_dev(dec_a), u8_to_dev(b),
                u8_to_dev(b_s), f32_scalar_dev(dec_b), fmt=fmt)
    torch.cuda.synchronize()
    gemm_check(host(c), ref, al, ogemm.abs_product(A, B), K, f"{fmt} {layout} K={K}")


@pytest.mark.parametrize("fmt", ["ue5m3", "e4m3"])
def test_smallest_codes_only(fmt):
    """Operands made of the subnormal scale codes alone (UE5M3 0x01..0x07,
    E4M3 0x01..0x07) and the smallest normal one: the decoded values reach
    0.5 x 2^-17 (UE5M3), i.e. 2^-21 on the matrix cores' fp16 operands, and
    every product and sum must stay exact."""
    M, N, K = 256, 256, 512
    rng = np.random.default_rng(5)
    say("gemm smallest codes", fmt)
    a = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    b = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    a_s = rng.integers(1, 9, (M, K // 16)).astype(np.uint8)
    b_s = rng.integers(1, 9, (N // 16, K // 16)).astype(np.uint8)
    A = oq.decoded_1d(a, a_s, 1, fmt=fmt)
    B = oq.decoded_2d(b, b_s, fmt=fmt)
    al = ogemm.alpha(np.float32(1.0), np.float32(1.0))
    ref = ogemm.fprop(A, B, al)
    # the exact sums are multiples of the smallest product: no rounding at all
    # while they stay below 2^24 of it
    c = ue.gemm("nt", M, N, K, u8_to_dev(a), u8_to_dev(a_s), f32_scalar_dev(1.0), u8_to_dev(b),
                u8_to_dev(b_s), f32_scalar_dev(1.0), fmt=fmt)
    torch.cuda.synchronize()
    assert np.array_equal(host(c).astype(np.float64), ref), fmt
