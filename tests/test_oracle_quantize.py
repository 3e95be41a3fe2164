"""Pins of the oracle's block quantizers: hand-worked blocks, grid round
trips, the RN error bound, layout identities, and the stochastic-rounding
rule of eq:sr (unbiasedness, exact up-probabilities)."""

import os

import numpy as np
import pytest

import synthetic
from oracle import formats, philox, quantize, scaling


def _worked_blocks(golden_dir):
    out = []
    for line in open(os.path.join(golden_dir, "worked_blocks.txt")):
        if not line.strip() or line.startswith("#"):
            continue
        name, g, T, xs, sc, pay = [f.strip() for f in line.split("|")]
        x = np.array([float(v) for v in xs.split()], np.float32)
        out.append((name, float(g), float(T), x, int(sc, 16),
                    np.array([int(b, 16) for b in pay.split()], np.uint8)))
    return out


def test_worked_blocks(golden_dir):
    blocks = _worked_blocks(golden_dir)
    assert len(blocks) == 4
    for name, g, T, x, sc, pay in blocks:
        bits = synthetic.f32_to_bf16_bits(x)
        assert np.array_equal(synthetic.bf16_bits_to_f32(bits), x), name   # exact in bf16
        p, s, _ = quantize.quantize_1d(bits[None, :], 1, np.float32(g), T)
        assert s[0, 0] == sc, name
        assert np.array_equal(p[0], pay), name
        # same block as a column (axis 0) and inside a 16x16 tile
        pc, scc, _ = quantize.quantize_1d(bits[:, None], 0, np.float32(g), T)
        assert scc[0, 0] == sc and np.array_equal(pc[0], pay), name


def test_worked_block_sr_keeps_grid_points(golden_dir):
    # Block D: inputs are grid points, exact midpoints and 5.5 (3/4 of the way
    # from 4 to 6); under SR grid points never move, midpoints go up with
    # probability 1/2 and 5.5 with probability 3/4.
    _, g, T, x, _, _ = [b for b in _worked_blocks(golden_dir) if b[0] == "D"][0]
    bits = synthetic.f32_to_bf16_bits(np.tile(x, (4096, 1)))
    p, s, _ = quantize.quantize_1d(bits, 1, np.float32(g), T, mode="sr", seed=11, tensor_id=3)
    q = formats.e2m1_decode(quantize._unpack_rows(p))
    on_grid = np.isin(np.abs(x), formats.E2M1_MAG) | (np.abs(x) > 6)
    assert np.all(q[:, on_grid] == np.where(np.abs(x[on_grid]) > 6, np.sign(x[on_grid]) * 6, x[on_grid]))
    frac_up = np.mean(np.abs(q[:, ~on_grid]) > np.abs(x[~on_grid]), axis=0)
    expect = np.where(np.abs(x[~on_grid]) == 5.5, 0.75, 0.5)
    assert np.all(np.abs(frac_up - expect) < 5 * 0.5 / np.sqrt(4096))


def test_zero_scale_rule_and_underflow():
    # A block whose ideal code rounds to zero stores the code of 1.0
    # (Sec. 4.3: zero block-scale code replaced with 1).
    x = np.zeros((1, 32), np.float32)
    x[0, 16] = 1e-12
    bits = synthetic.f32_to_bf16_bits(x)
    p, s, _ = quantize.quantize_1d(bits, 1, np.float32(1000.0), 448.0)
    assert list(s[0]) == [formats.UE5M3_ONE, formats.UE5M3_ONE]
    assert np.all(p == 0)


def test_grid_values_round_trip():
    # g = T = 448 gives S = 1 and G = 6: a block with maximum 6 has scale 6 and
    # r = 1, so values on the E2M1 grid are encoded exactly and decode to 6 x.
    rng = np.random.default_rng(0)
    vals = rng.choice(np.concatenate([formats.E2M1_MAG, -formats.E2M1_MAG]), (32, 64))
    vals[:, ::16] = 6.0
    bits = synthetic.f32_to_bf16_bits(vals.astype(np.float32))
    p, s, dec = quantize.quantize_1d(bits, 1, np.float32(448.0), 448.0)
    assert np.all(s == 0x8C)
    d = quantize.decoded_1d(p, s, 1)
    assert np.array_equal(d, 6.0 * vals)
    assert np.allclose(quantize.dequantize(d, dec), vals, rtol=1e-6, atol=0)


@pytest.mark.parametrize("axis", [0, 1])
def test_rn_error_bound(axis):
    bits = synthetic.activation(1, 64, 128, 0.01, 50.0)
    x = synthetic.bf16_bits_to_f32(bits).astype(np.float64)
    g = scaling.amax(bits)
    S, G, dec = scaling.tensor_multipliers(g, 448.0)
    p, s, _ = quantize.quantize_1d(bits, axis, g, 448.0)
    d = quantize.decoded_1d(p, s, axis)                       # q * s_B
    sv = formats.ue5m3_decode(s)
    sfull = np.repeat(sv, 16, axis=1)
    if axis == 0:
        sfull = sfull.T
    y = x * float(G) / sfull                                  # ideal E2M1 input
    q = d / sfull
    ay = np.abs(y)
    spacing = np.where(ay < 2, 0.5, np.where(ay < 4, 1.0, 2.0))
    err = np.abs(y - q)
    # |y - q| <= half the E2M1 spacing around y, allowing a few binary32 ulps
    # of slop from rounding G, r_B and y; saturated entries decode to +-6
    sat = ay >= 6
    assert np.all(sat | (err <= spacing / 2 + 1e-5 * ay + 1e-30))
    assert np.all(np.abs(q[sat]) == 6) and np.all(np.abs(q) <= 6)


def test_axis0_is_axis1_of_transpose():
    bits = synthetic.gradient(2, 96, 48, 1e-4, 2.0)
    g = scaling.amax(bits)
    for mode in ["rn"]:
        p0, s0, d0 = quantize.quantize_1d(bits, 0, g, 448.0, mode)
        p1, s1, d1 = quantize.quantize_1d(np.ascontiguousarray(bits.T), 1, g, 448.0, mode)
        assert np.array_equal(p0, p1) and np.array_equal(s0, s1) and d0 == d1


def test_2d_tiles():
    bits = synthetic.weight(4, 64, 96)
    g = scaling.amax(bits)
    S, G, dec = scaling.tensor_multipliers(g, 448.0)
    p, s, pt, d = quantize.quantize_2d(bits, g, 448.0)
    x = synthetic.bf16_bits_to_f32(bits)
    # one scale per 16x16 tile, from the tile maximum
    tmax = np.abs(x).reshape(4, 16, 6, 16).max(axis=(1, 3)).astype(np.float32)
    exp = formats.ue5m3_encode_rne_sat((tmax * S).astype(np.float32))
    exp = np.where(exp == 0, formats.UE5M3_ONE, exp)
    assert np.array_equal(s, exp)
    # the transposed payload holds the same nibbles
    assert np.array_equal(quantize.decoded_2d(p, s), quantize.decoded_2d_t(pt, s))
    # a tile with a single non-zero entry behaves like that entry's 1D block
    one = np.zeros((16, 16), np.float32)
    one[3, 5] = 0.75
    b1 = synthetic.f32_to_bf16_bits(one)
    p2, s2, _, _ = quantize.quantize_2d(b1, np.float32(1.0), 448.0)
    p1, s1, _ = quantize.quantize_1d(b1[3:4], 1, np.float32(1.0), 448.0)
    assert s2[0, 0] == s1[0, 0] and np.array_equal(p2[3], p1[0])


# --------------------------------------------------------------- SR ----
def test_sr_unbiased():
    """E[Q_SR(z)] = z (eq:sr) over 2**20 Philox draws per value."""
    zs = np.array([0.1, 0.3, 0.49, 0.7, 1.1, 1.9, 2.2, 3.3, 4.9, 5.99, -0.2, -2.7,
                   1e-7, 2.0 ** -30], np.float32)
    n = 1 << 20
    idx = np.arange(n, dtype=np.int64)
    for i, z in enumerate(zs):
        w = philox.sr_words(99, i, idx)
        q = formats.e2m1_decode(formats.e2m1_encode_sr(np.full(n, z, np.float32), w))
        a = abs(float(z))
        lo = formats.E2M1_MAG[np.searchsorted(formats.E2M1_MAG, a, "right") - 1]
        hi = formats.E2M1_MAG[np.searchsorted(formats.E2M1_MAG, a, "right")]
        p = (a - lo) / (hi - lo)
        sigma = (hi - lo) * np.sqrt(p * (1 - p) / n)
        assert abs(q.mean() - float(z)) <= 5 * sigma + 1e-12, z
        assert set(np.unique(np.abs(q))) <= {lo, hi}


def test_sr_up_probability_exact():
    """Over evenly spaced words the fraction that rounds up equals frac up
    to the 2**-32 word resolution (P(up) = (z - q-) / (q+ - q-))."""
    step = 1 << 12
    w = np.arange(0, 1 << 32, step, dtype=np.uint64)
    for z in [0.25, 0.3, 0.75, 1.25, 2.5, 3.999, 5.0, 0.0001, 1.0, 6.0, 7.5]:
        q = formats.e2m1_decode(formats.e2m1_encode_sr(np.full(w.size, z, np.float32), w))
        a = float(np.float32(z))
        if a >= 6:
            assert np.all(q == 6.0)
            continue
        k = np.searchsorted(formats.E2M1_MAG, a, "right") - 1
        lo, hi = formats.E2M1_MAG[k], formats.E2M1_MAG[k + 1]
        frac = (a - lo) / (hi - lo)
        up = np.mean(q > lo)
        assert abs(up - frac) <= step / 2.0 ** 32, z
        if frac == 0:
            assert np.all(q == lo)


def test_sr_deterministic_and_keyed():
    bits = synthetic.gradient(5, 32, 64, 1e-4, 2.0)
    g = scaling.amax(bits)
    a = quantize.quantize_1d(bits, 1, g, 448.0, "sr", seed=1, tensor_id=1)
    b = quantize.quantize_1d(bits, 1, g, 448.0, "sr", seed=1, tensor_id=1)
    c = quantize.quantize_1d(bits, 1, g, 448.0, "sr", seed=1, tensor_id=2)
    d = quantize.quantize_1d(bits, 1, g, 448.0, "sr", seed=2, tensor_id=1)
    assert np.array_equal(a[0], b[0])
    assert not np.array_equal(a[0], c[0]) and not np.array_equal(a[0], d[0])
    assert np.array_equal(a[1], c[1])            # scales never depend on SR
    # SR words follow the source element, whatever the blocking
    col = quantize.quantize_1d(bits, 0, g, 448.0, "sr", seed=1, tensor_id=1)
    rowT = quantize.quantize_1d(np.ascontiguousarray(bits.T), 1, g, 448.0, "sr", seed=1, tensor_id=1)
    assert np.array_equal(col[1], rowT[1])


# ------------------------------------------ comparison scale formats ----
def _format_blocks(golden_dir):
    out = []
    for line in open(os.path.join(golden_dir, "worked_blocks_formats.txt")):
        if not line.strip() or line.startswith("#"):
            continue
        name, fmt, g, T, xs, sc, pay = [f.strip() for f in line.split("|")]
        B = quantize.block_size(fmt)
        x = np.zeros(B, np.float32)
        vals = [float(v) for v in xs.split()]
        x[:len(vals)] = vals
        out.append((name, fmt, float(g), float(T), x, int(sc, 16),
                    np.array([int(b, 16) for b in pay.split()], np.uint8)))
    return out


def test_worked_blocks_comparison_formats(golden_dir):
    blocks = _format_blocks(golden_dir)
    assert {b[1] for b in blocks} == {"e4m3", "e8m0"} and len(blocks) == 11
    for name, fmt, g, T, x, sc, pay in blocks:
        bits = synthetic.f32_to_bf16_bits(x)
        assert np.array_equal(synthetic.bf16_bits_to_f32(bits).view(np.uint32), x.view(np.uint32)), name
        p, s, dec = quantize.quantize_1d(bits[None, :], 1, np.float32(g), T, fmt=fmt)
        assert s.shape == (1, 1) and s[0, 0] == sc, (name, hex(s[0, 0]))
        assert np.array_equal(p[0], pay), (name, p[0])
        if fmt == "e8m0":
            assert dec == 1.0
        pc, scc, _ = quantize.quantize_1d(bits[:, None], 0, np.float32(g), T, fmt=fmt)
        assert scc[0, 0] == sc and np.array_equal(pc[0], pay), name
        if fmt == "e4m3":
            tile = np.zeros((16, 16), np.uint16)
            tile[3] = bits
            p2, s2, pt2, _ = quantize.quantize_2d(tile, np.float32(g), T, fmt=fmt)
            assert s2[0, 0] == sc and np.array_equal(p2[3], pay), name


def test_e4m3_pipeline_differs_from_ue5m3_only_in_the_scale_code():
    # Inside E4M3's range the two 3-fraction-bit scales pick the same value,
    # so payloads agree; they part only where E4M3 saturates (448) or
    # underflows (2^-9) and UE5M3 does not (Sec. 3, Table 2).
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((64, 256)) * np.exp(rng.uniform(-3, 3, (64, 1)))).astype(np.float32)
    bits = synthetic.f32_to_bf16_bits(x)
    g = scaling.amax(bits)
    pu, su, du = quantize.quantize_1d(bits, 1, g, 448.0)
    pe, se, de = quantize.quantize_1d(bits, 1, g, 448.0, fmt="e4m3")
    vu, ve = formats.ue5m3_decode(su), formats.e4m3_decode(se)
    inside = (vu >= 2.0 ** -6) & (vu <= 448.0)          # both normal, E4M3 not saturated
    assert inside.mean() > 0.5
    assert np.array_equal(vu[inside], ve[inside]) and du == de
    rows = np.all(inside, axis=1)
    assert np.array_equal(pu[rows], pe[rows])


def test_e8m0_exponent_rule_properties():
    # OCP microscaling exponent: 2^(E+2) <= a_B < 2^(E+3) (unclamped), the
    # scaled block maximum lies in [4, 8), and y = x * 2^-E is exact.
    rng = np.random.default_rng(6)
    x = (rng.standard_normal((128, 64)) * np.exp2(rng.integers(-40, 40, (128, 1)))).astype(np.float32)
    x[5] = 0.0
    bits = synthetic.f32_to_bf16_bits(x)
    xf = synthetic.bf16_bits_to_f32(bits).astype(np.float64)
    p, s, dec = quantize.quantize_1d(bits, 1, np.float32(0), 0.0, fmt="e8m0")
    assert s.shape == (128, 2) and dec == 1.0
    a = np.abs(xf).reshape(128, 2, 32).max(axis=2)
    E = s.astype(np.int64) - 127
    nz = a > 0
    assert np.all(np.exp2(E[nz] + 2.0) <= a[nz]) and np.all(a[nz] < np.exp2(E[nz] + 3.0))
    assert np.all(s[~nz] == 0)
    q = formats.e2m1_decode(quantize._unpack_rows(p)).reshape(128, 2, 32)
    y = xf.reshape(128, 2, 32) * np.exp2(-E)[:, :, None]
    # RN error: each nibble is a nearest E2M1 value of y (saturating at 6)
    err = np.abs(np.clip(y, -6, 6) - q)
    step = np.where(np.abs(y) < 2, 0.5, np.where(np.abs(y) < 4, 1.0, 2.0))
    assert np.all(err <= step / 2 + 1e-12)
    # decoded operand = q * 2^E
    dec_v = quantize.decoded_1d(p, s, 1, fmt="e8m0")
    assert np.array_equal(dec_v.reshape(128, 2, 32), q * np.exp2(E)[:, :, None])


def test_e8m0_sr_uses_the_element_words():
    # SR under E8M0 draws the same per-element words as under UE5M3
    rng = np.random.default_rng(7)
    x = rng.standard_normal((32, 64)).astype(np.float32)
    bits = synthetic.f32_to_bf16_bits(x)
    p1, s1, _ = quantize.quantize_1d(bits, 1, np.float32(0), 0.0, mode="sr", seed=9, tensor_id=4, fmt="e8m0")
    p2, s2, _ = quantize.quantize_1d(bits, 1, np.float32(0), 0.0, mode="sr", seed=9, tensor_id=4, fmt="e8m0")
    p3, _, _ = quantize.quantize_1d(bits, 1, np.float32(0), 0.0, mode="sr", seed=10, tensor_id=4, fmt="e8m0")
    assert np.array_equal(p1, p2) and not np.array_equal(p1, p3)
    xf = synthetic.bf16_bits_to_f32(bits).astype(np.float64)
    E = s1.astype(np.int64) - 127
    y = xf.reshape(32, 2, 32) * np.exp2(-E)[:, :, None]
    q = formats.e2m1_decode(quantize._unpack_rows(p1)).reshape(32, 2, 32)
    # SR lands on one of the two E2M1 neighbours of y (6 at or above 6)
    assert np.all(np.abs(np.abs(q) - np.minimum(np.abs(y), 6.0)) <= np.where(np.abs(y) < 2, 0.5, 2.0))


# ------------------------------------------------ block-size-32 control --
def _b(vals):
    return synthetic.f32_to_bf16_bits(np.asarray(vals, np.float32))


def test_block32_hand_worked_and_halves():
    """Block-size control (blocks of 32): the worked block A (g = 100,
    T = 448, scale 0xBE) followed by a half whose largest magnitude is also
    100 keeps A's scale and nibbles; the second half (-100, 0, ...) gives
    -6 -> nibble 0xF.  A half with a larger maximum changes the shared
    scale."""
    a = [100, -37.5, 12, 0.25, 0, -0.0, 50, 25, -60, 8.5, 3, -1, 90, 75, 5.25, -16.5]
    x = _b([a + [-100] + [0] * 15])
    p, s, _ = quantize.quantize_1d(x, 1, 100.0, 448.0, block=32)
    assert s.tolist() == [[0xBE]]
    assert p[0, :8].tobytes() == bytes.fromhex("C7018035 1E8067A1".replace(" ", ""))
    assert p[0, 8:].tolist() == [0x0F] + [0] * 7
    x2 = _b([a + [400] + [0] * 15])
    p2, s2, _ = quantize.quantize_1d(x2, 1, 100.0, 448.0, block=32)
    assert s2[0, 0] != 0xBE


def test_block32_equals_block16_when_halves_share_maxima():
    """When both 16-element halves of every 32-block have the same maximum,
    blocks of 32 give the blocks of 16 result (RN and SR, rows and
    columns), and 32x32 tiles give the 16x16 result when the four sub-tiles
    share their maximum."""
    rng = np.random.default_rng(4)
    v = rng.standard_normal((64, 128)).astype(np.float32)
    v[:, ::16] = 5.0                                   # every 16-block (rows) peaks at 5
    v[::16, :] = 5.0                                   # every 16-block (columns) peaks at 5
    x = _b(v)
    for axis in (0, 1):
        for mode in ("rn", "sr"):
            p16, s16, d16 = quantize.quantize_1d(x, axis, 5.0, 448.0, mode, 3, 7)
            p32, s32, d32 = quantize.quantize_1d(x, axis, 5.0, 448.0, mode, 3, 7, block=32)
            assert np.array_equal(p16, p32) and d16 == d32
            assert np.array_equal(s16[:, ::2], s32) and np.array_equal(s16[:, 1::2], s32)
    t16 = quantize.quantize_2d(x, 5.0)
    t32 = quantize.quantize_2d(x, 5.0, tile=32)
    assert np.array_equal(t16[0], t32[0]) and np.array_equal(t16[2], t32[2])
    assert np.array_equal(t16[1][::2, ::2], t32[1]) and np.array_equal(t16[1][1::2, 1::2], t32[1])
    # decoded operands agree too
    assert np.array_equal(quantize.decoded_2d(t32[0], t32[1], tile=32), quantize.decoded_2d(t16[0], t16[1]))
    with pytest.raises(ValueError):
        quantize.quantize_1d(x, 1, 5.0, block=64)
    with pytest.raises(ValueError):
        quantize.quantize_2d(_b(np.zeros((48, 64))), 1.0, tile=32)
