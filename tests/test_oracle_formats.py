"""Pins of the oracle's number formats against the paper and against
library float types (E2M1, UE5M3, E4M3, E8M0; Sec. 2-3, Table 1, Table 2)."""

import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import formats


def _paper_values(golden_dir):
    vals = {}
    with open(os.path.join(golden_dir, "paper_values.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                name, value = line.split()[:2]
                vals[name] = float(value)
    return vals


def minifloat_value(code, ebits, mbits, bias, signed):
    """Generic IEEE-style minifloat decode (finite codes only): the test's own
    decoder, checked below against library float16 / float8 types."""
    m = code & ((1 << mbits) - 1)
    e = (code >> mbits) & ((1 << ebits) - 1)
    s = (code >> (ebits + mbits)) & 1 if signed else 0
    if e == 0:
        v = Fraction(m, 1 << mbits) * Fraction(2) ** (1 - bias)
    else:
        v = (1 + Fraction(m, 1 << mbits)) * Fraction(2) ** (e - bias)
    return -v if s else v


def test_generic_minifloat_matches_float16():
    codes = np.arange(0x7C00, dtype=np.uint16)          # all finite positives
    ref = codes.view(np.float16).astype(np.float64)
    mine = np.array([float(minifloat_value(int(c), 5, 10, 15, True)) for c in codes])
    assert np.array_equal(ref, mine)


def test_generic_minifloat_matches_torch_e4m3():
    codes = torch.arange(0x7F, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).double().numpy()
    mine = np.array([float(minifloat_value(int(c), 4, 3, 7, True)) for c in range(0x7F)])
    assert np.array_equal(ref, mine)


def test_e2m1_decode(golden_dir):
    pv = _paper_values(golden_dir)
    dec = formats.e2m1_decode(np.arange(16, dtype=np.uint8))
    # 1 sign, 2 exponent, 1 fraction bit; the bias is fixed by the paper's
    # largest magnitude F = 6: 2**(3 - bias) * 1.5 = 6  =>  bias = 1.
    ref = [float(minifloat_value(c, 2, 1, 1, True)) for c in range(16)]
    assert np.array_equal(dec, np.array(ref))
    assert np.max(np.abs(dec)) == pv["e2m1_max"]
    assert np.signbit(dec[8]) and dec[8] == 0.0           # code 8 is -0


def test_ue5m3_decode_all_codes(golden_dir):
    pv = _paper_values(golden_dir)
    codes = np.arange(256)
    dec = formats.ue5m3_decode(codes)
    # Finite codes: unsigned E5M3 with the fp16 exponent: bits c << 7 as fp16.
    fp16 = (codes[:0xF8].astype(np.uint16) << 7).view(np.float16).astype(np.float64)
    assert np.array_equal(dec[:0xF8], fp16)
    assert np.isinf(dec[0xF8]) and np.all(np.isnan(dec[0xF9:]))
    # The paper's range: eq:ue5m3max, smallest normal and subnormal, Table 2.
    assert dec[0xF7] == pv["ue5m3_max"] == 1.875 * 2 ** 15
    assert dec[0x08] == pv["ue5m3_min_normal"] == 2.0 ** -14
    assert dec[0x01] == pv["ue5m3_min_subnormal"] == 2.0 ** -17
    assert np.all(np.diff(dec[:0xF8]) > 0)
    assert dec[formats.UE5M3_ONE] == 1.0
    # Table 2 comparison with E4M3: ~137x larger max, 256x smaller min.
    assert round(dec[0xF7] / pv["e4m3_max"]) == pv["ue5m3_over_e4m3_max"]
    assert pv["e4m3_min_subnormal"] / dec[0x01] == pv["e4m3_over_ue5m3_min"]


def test_e4m3_e8m0_decode_against_torch(golden_dir):
    pv = _paper_values(golden_dir)
    codes = torch.arange(256, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).double().numpy()
    mine = formats.e4m3_decode(np.arange(256))
    fin = ~np.isnan(ref)
    assert np.array_equal(np.isnan(ref), np.isnan(mine))
    assert np.array_equal(ref[fin], mine[fin])
    assert np.nanmax(mine) == pv["e4m3_max"]
    assert mine[1] == pv["e4m3_min_subnormal"]
    ref8 = codes.view(torch.float8_e8m0fnu).double().numpy()
    mine8 = formats.e8m0_decode(np.arange(256))
    assert np.array_equal(np.isnan(ref8), np.isnan(mine8))
    assert np.array_equal(ref8[:255], mine8[:255])


# ----------------------------------------------------------- encoders ----
def _f32(x):
    return np.asarray(x, dtype=np.float32)


def _neighbours(vals, k=3):
    """float32 values within k ulps of each value in ``vals``."""
    v = _f32(vals)
    out = [v]
    lo, hi = v.copy(), v.copy()
    for _ in range(k):
        lo = np.nextafter(lo, np.float32(-np.inf))
        hi = np.nextafter(hi, np.float32(np.inf))
        out += [lo, hi]
    return np.concatenate(out)


def _brute_nearest(u, codebook_vals, max_code):
    """Exact nearest-code search with Fractions; ties -> even code;
    above the largest finite value -> max_code."""
    uf = Fraction(float(u))
    top = Fraction(float(codebook_vals[max_code]))
    if uf > top:
        return max_code
    best, bestd = None, None
    for c in range(max_code + 1):
        d = abs(uf - Fraction(float(codebook_vals[c])))
        if bestd is None or d < bestd or (d == bestd and c % 2 == 0):
            best, bestd = c, d
    return best


def test_ue5m3_encode_boundaries_brute_force():
    vals = formats.UE5M3_FINITE
    mids = (vals[:-1] + vals[1:]) / 2.0
    sample = _neighbours(np.concatenate([vals, mids, [61440.0 * 1.01, 1e9, 1e-30, 0.0]]), 2)
    sample = sample[sample >= 0]
    got = formats.ue5m3_encode_rne_sat(sample)
    exp = np.array([_brute_nearest(u, vals, 0xF7) for u in sample])
    assert np.array_equal(got, exp)


def test_ue5m3_encode_random_brute_force():
    rng = np.random.default_rng(1)
    u = _f32(np.exp(rng.uniform(np.log(2.0 ** -20), np.log(1e5), 4000)))
    got = formats.ue5m3_encode_rne_sat(u)
    exp = np.array([_brute_nearest(x, formats.UE5M3_FINITE, 0xF7) for x in u])
    assert np.array_equal(got, exp)


def test_ue5m3_encode_examples():
    # Exact codes, ties to even, subnormal rounding, saturation.
    cases = {1.0: 0x78, 1.0625: 0x78, 1.1875: 0x7A, 2.0 ** -18: 0x00,
             3 * 2.0 ** -18: 0x02, 448.0: 0xBE, 464.0: 0xBE, 480.0: 0xBF,
             2048.0: 0xD0, 61440.0: 0xF7, 61441.0: 0xF7, 1e9: 0xF7, 0.0: 0x00}
    u = _f32(list(cases))
    assert list(formats.ue5m3_encode_rne_sat(u)) == list(cases.values())


def test_e2m1_encode_boundaries_brute_force():
    mags = formats.E2M1_MAG
    mids = (mags[:-1] + mags[1:]) / 2.0
    base = np.concatenate([mags, mids, [7.0, 100.0, 1e30, 1e-30, 1e-45]])
    sample = _neighbours(np.concatenate([base, -base]), 3)
    got = formats.e2m1_encode_rne(sample)
    exp = []
    for y in sample:
        c = _brute_nearest(abs(float(y)), mags, 7)
        exp.append(c | (8 if np.signbit(y) else 0))
    assert np.array_equal(got, np.array(exp, dtype=np.uint8))


def test_e2m1_ties_to_even():
    y = _f32([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -5.0, -0.0, 0.0, 6.0, 1e6, -1e6])
    exp = [0, 2, 2, 4, 4, 6, 6, 8, 14, 8, 0, 7, 7, 15]
    assert list(formats.e2m1_encode_rne(y)) == exp


def test_e4m3_encode_matches_torch_rne():
    rng = np.random.default_rng(2)
    u = _f32(np.concatenate([np.exp(rng.uniform(np.log(2.0 ** -11), np.log(448.0), 20000)),
                             formats.E4M3_FINITE_POS,
                             (formats.E4M3_FINITE_POS[:-1] + formats.E4M3_FINITE_POS[1:]) / 2]))
    got = formats.e4m3_encode_rne_sat(u)
    ref = torch.from_numpy(u).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got, ref)
    assert formats.e4m3_encode_rne_sat(_f32([449.0, 1e6]))[0] == 0x7E
