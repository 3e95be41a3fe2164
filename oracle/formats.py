"""Number formats (oracle; test infrastructure only).

E2M1 payload (Sec. 1 and Sec. 2.1 of the paper): one sign bit, two exponent
bits, one fraction bit, largest magnitude F = 6.  The paper does not list the
value set; this oracle takes the OCP E2M1 reading (exponent bias 1, one
subnormal step of 0.5, no infinities or NaNs):

    code & 7 :  0    1    2    3    4    5    6    7
    |value|  :  0   0.5  1.0  1.5  2.0  3.0  4.0  6.0

and bit 3 is the sign (code 8 decodes to -0).

UE5M3 block scale (Sec. 3.1, eq:ue5m3max, Table 2): unsigned, five exponent
bits and three fraction bits.  The paper fixes the largest finite value
U = 1.875 * 2**15 = 61440, the smallest normal 2**-14 and the smallest
subnormal 2**-17, which determine exponent bias 15.  Reading: exponent field
31 (codes 0xF8..0xFF) is not finite (0xF8 = +inf, the rest NaN), so the
finite codes are 0x00..0xF7.

Both encoders round to nearest with ties to the even code (Sec. 4.3: ties-to-
even for payloads and block scales) and saturate: a magnitude above the
largest finite value takes the largest finite code.

E4M3 (NVFP4 block scale; Table 1, Table 2: largest 448, smallest subnormal
2**-9) and E8M0 (MXFP4 block scale; Table 1: power-of-two scales) are the
comparison formats.
"""

import numpy as np

# ---------------------------------------------------------------- E2M1 ----
E2M1_MAG = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)
E2M1_MAX = 6.0


def e2m1_decode(nib):
    """Value of each E2M1 nibble (uint8 array, values 0..15) as float64."""
    nib = np.asarray(nib, dtype=np.uint8)
    mag = E2M1_MAG[nib & 7]
    return np.where((nib >> 3) & 1, -mag, mag)


def e2m1_encode_rne(y):
    """Nearest E2M1 nibble to each float32 ``y``, ties to the even code,
    magnitudes at or above 6 saturating to code 7; the sign bit copies the
    sign of ``y`` (so -0 and small negatives give nibble 8)."""
    y = np.asarray(y, dtype=np.float32)
    a = np.abs(y.astype(np.float64))
    # Candidate codes ordered even-first so that argmin (first minimum)
    # resolves an exact tie in favour of the even code.
    order = np.array([0, 2, 4, 6, 1, 3, 5, 7])
    dist = np.abs(a[..., None] - E2M1_MAG[order])
    code = order[np.argmin(dist, axis=-1)]
    code = np.where(a >= E2M1_MAX, 7, code)
    sign = np.signbit(y).astype(np.uint8)
    return (code.astype(np.uint8) | (sign << 3)).astype(np.uint8)


def e2m1_encode_sr(y, words):
    """Stochastic rounding of float32 ``y`` to E2M1 (eq:sr).

    For |y| between adjacent codebook magnitudes q_lo <= |y| < q_hi the
    magnitude rounds up with probability (|y| - q_lo) / (q_hi - q_lo).  The
    random choice uses one uniform 32-bit word w per element: round up iff
    w < ceil(frac * 2**32) (unsigned compare), so P(up) equals frac to within
    2**-32.  Magnitudes at or above 6 give code 7.  Sign as in RNE.
    """
    y = np.asarray(y, dtype=np.float32)
    w = np.asarray(words, dtype=np.uint64)
    a = np.abs(y.astype(np.float64))
    lo = np.searchsorted(E2M1_MAG, a, side="right") - 1
    lo = np.clip(lo, 0, 6)
    q_lo = E2M1_MAG[lo]
    q_hi = E2M1_MAG[lo + 1]
    frac = (a - q_lo) / (q_hi - q_lo)          # exact: power-of-two spacing
    thr = np.ceil(np.minimum(frac, 1.0) * 2.0 ** 32)
    up = w.astype(np.float64) < thr
    code = lo + up.astype(np.int64)
    code = np.where(a >= E2M1_MAX, 7, code)
    sign = np.signbit(y).astype(np.uint8)
    return (code.astype(np.uint8) | (sign << 3)).astype(np.uint8)


# --------------------------------------------------------------- UE5M3 ----
UE5M3_MAX = 61440.0
UE5M3_MAX_CODE = 0xF7
UE5M3_ONE = 0x78          # code of the value 1.0 (exponent field 15)


def ue5m3_decode(code):
    """Value of each UE5M3 byte as float64 (0xF8 = +inf, 0xF9..0xFF = NaN)."""
    c = np.asarray(code, dtype=np.int64)
    e = c >> 3
    m = c & 7
    sub = m * 2.0 ** -17
    nrm = (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 15.0)
    v = np.where(e == 0, sub, nrm)
    v = np.where(e == 31, np.where(m == 0, np.inf, np.nan), v)
    return v


UE5M3_FINITE = ue5m3_decode(np.arange(UE5M3_MAX_CODE + 1))   # ascending


def _nearest_code_even(values_sorted, u):
    """Index of the entry of ascending ``values_sorted`` nearest to ``u``
    (float64, all >= values_sorted[0]), ties to the even index."""
    hi = np.searchsorted(values_sorted, u, side="left")
    hi = np.clip(hi, 1, len(values_sorted) - 1)
    lo = hi - 1
    v_lo = values_sorted[lo]
    v_hi = values_sorted[hi]
    # 2u against (v_lo + v_hi): both sides exact in float64 for the operands
    # used here (binary32 inputs, codebook values of <= 4 significant bits).
    twice = 2.0 * u
    mid = v_lo + v_hi
    pick_hi = (twice > mid) | ((twice == mid) & (hi % 2 == 0))
    idx = np.where(pick_hi, hi, lo)
    idx = np.where(u <= values_sorted[0], 0, idx)
    return idx


def ue5m3_encode_rne_sat(u):
    """UE5M3 byte nearest to each non-negative float32 ``u`` (ties to even
    code); every u above 61440 saturates to 0xF7."""
    u = np.asarray(u, dtype=np.float32).astype(np.float64)
    idx = _nearest_code_even(UE5M3_FINITE, np.minimum(u, UE5M3_MAX))
    idx = np.where(u > UE5M3_MAX, UE5M3_MAX_CODE, idx)
    return idx.astype(np.uint8)


# ---------------------------------------------------------------- E4M3 ----
E4M3_MAX = 448.0
E4M3_ONE = 0x38


def e4m3_decode(code):
    """OCP E4M3FN: bias 7, no infinities, 0x7F/0xFF NaN.  Sign bit 7."""
    c = np.asarray(code, dtype=np.int64)
    s = (c >> 7) & 1
    e = (c >> 3) & 15
    m = c & 7
    v = np.where(e == 0, m * 2.0 ** -9,
                 (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0))
    v = np.where((e == 15) & (m == 7), np.nan, v)
    return np.where(s == 1, -v, v)


E4M3_FINITE_POS = e4m3_decode(np.arange(0x7F))   # codes 0x00..0x7E ascending


def e4m3_encode_rne_sat(u):
    """Non-negative float32 ``u`` -> E4M3 byte, nearest (ties to even code),
    saturating above 448 to 0x7E."""
    u = np.asarray(u, dtype=np.float32).astype(np.float64)
    idx = _nearest_code_even(E4M3_FINITE_POS, np.minimum(u, E4M3_MAX))
    idx = np.where(u > E4M3_MAX, 0x7E, idx)
    return idx.astype(np.uint8)


# ---------------------------------------------------------------- E8M0 ----
def e8m0_decode(code):
    """E8M0: value 2**(code - 127); 0xFF is NaN."""
    c = np.asarray(code, dtype=np.int64)
    v = np.exp2(c.astype(np.float64) - 127.0)
    return np.where(c == 255, np.nan, v)
