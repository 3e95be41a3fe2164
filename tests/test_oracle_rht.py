"""Pins of the oracle's randomized Hadamard transform of the wgrad operands
(Sec. 2 recipe techniques, Table 6 "UE5M3 with Transformer Engine
settings"): the Hadamard matrix, the butterfly against the matrix product
where the latter is exact, a hand-derived case where the binary32 butterfly
order decides the result, orthogonality (the transform inverts itself and
matched transforms leave dY^T X unchanged), outlier spreading, and the
quantizer on transformed values."""

import numpy as np
import pytest

import synthetic
from oracle import quantize, rht, scaling


def test_hadamard_matrix():
    H = rht.hadamard16()
    assert H.shape == (16, 16) and set(np.unique(H)) == {-1, 1}
    assert (H @ H.T == 16 * np.eye(16)).all()
    assert (H[0] == 1).all() and (H[:, 0] == 1).all()
    assert H[1, 1] == -1 and H[3, 3] == 1 and H[7, 7] == -1 and H[15, 15] == 1   # (-1)^popcount(i & j)


def test_butterfly_equals_matrix_product_when_exact():
    rng = np.random.default_rng(0)
    x = rng.integers(-300, 300, (48, 5)).astype(np.float32)
    for mask in (0, 0xFFFF, 0x1234, 0xBEEF):
        y = rht.transform_cols(x, mask)
        s = rht.signs(mask)
        ref = 0.25 * np.einsum("ij,bjc->bic", rht.hadamard16(), s[None, :, None] * x.reshape(3, 16, 5))
        assert np.array_equal(y.reshape(3, 16, 5), ref.astype(np.float32))


def test_binary32_butterfly_order():
    """x = (2^24, 1, 1, 0, ...): the exact y_0 = (2^24 + 2) / 4 is
    representable, but the butterfly rounds 2^24 + 1 to 2^24 (tie to even)
    in stage h = 1 and again in stage h = 2, giving 2^22.  Worked by hand:
    after h = 1: (2^24, 2^24 - 1, 1, 1); after h = 2: (2^24, 2^24,
    2^24 - 1, 2^24 - 2); h = 4 and 8 copy these into the zero halves."""
    x = np.zeros((16, 1), np.float32)
    x[0, 0], x[1, 0], x[2, 0] = 2.0 ** 24, 1.0, 1.0
    y = rht.transform_cols(x, 0).ravel()
    q = np.array([2 ** 24, 2 ** 24, 2 ** 24 - 1, 2 ** 24 - 2], np.float64) / 4
    assert np.array_equal(y, np.tile(q, 4).astype(np.float32))
    assert y[0] != np.float32((2.0 ** 24 + 2) / 4)


def test_self_inverse_and_matched_product():
    rng = np.random.default_rng(1)
    x = rng.integers(-64, 64, (64, 6)).astype(np.float32)
    assert np.array_equal(rht.transform_cols(rht.transform_cols(x, 0), 0), x)   # H H / 16 = I
    a = rng.integers(-64, 64, (64, 7)).astype(np.float32)
    b = rng.integers(-64, 64, (64, 5)).astype(np.float32)
    m = 0x5A3C
    ta, tb = rht.transform_cols(a, m), rht.transform_cols(b, m)
    assert np.array_equal(ta.astype(np.float64).T @ tb, a.astype(np.float64).T @ b)
    # unmatched masks do not preserve it
    assert not np.array_equal(rht.transform_cols(a, 1).astype(np.float64).T @ tb, a.astype(np.float64).T @ b)


def test_outlier_spread_over_block():
    x = np.zeros((16, 1), np.float32)
    x[5, 0] = 100.0
    y = rht.transform_cols(x, 1 << 5).ravel()             # s_5 = -1
    assert np.array_equal(np.abs(y), np.full(16, 25.0, np.float32))
    assert np.array_equal(np.sign(y), -rht.hadamard16()[:, 5].astype(np.float32))


def test_amax_and_quantizer_on_transformed_values():
    x = synthetic.activation(3, 64, 48)
    m = 0x0F0F
    y = rht.transform_cols(scaling.bf16_to_f32(x), m)
    g = rht.amax_rht(x, m)
    assert g == np.float32(np.max(np.abs(y)))
    p, s, dec = rht.quantize_cols_rht(x, g, m)
    p2, s2, dec2 = quantize.quantize_1d_values(y, 0, g)
    assert np.array_equal(p, p2) and np.array_equal(s, s2) and dec == dec2
    # the value path of the quantizer agrees with the bf16 path on bf16 inputs
    a = quantize.quantize_1d(x, 0, scaling.amax(x))
    b = quantize.quantize_1d_values(scaling.bf16_to_f32(x), 0, scaling.amax(x))
    assert all(np.array_equal(u, v) for u, v in zip(a, b))
    with pytest.raises(ValueError):
        rht.transform_cols(np.zeros((24, 2), np.float32), 0)
    with pytest.raises(ValueError):
        rht.signs(1 << 16)
