"""Block quantizers and dequantization (oracle; test infrastructure only).

Per block (eq:microscaling, eq:scale-target, Table 5 of the paper):
  1. a_B = max |x_i| over the block (exact);
  2. u_B = a_B * S, the ideal block-scale code (S = T / g);
  3. s_B = Q_UE5M3(u_B): nearest UE5M3 code, ties to even, saturating;
  4. a code that rounds to zero is replaced by the code of 1.0 before the
     reciprocal and dequantization (the proposed run's zero-scale rule);
  5. r_B = G / s_B (the reciprocal of the decode factor g_dec * s_B,
     G = T F / g);
  6. y_i = x_i * r_B;
  7. q_i = Q_E2M1(y_i): ties-to-even (RN) or stochastic rounding (SR, only
     for the upstream gradient dY, eq:sr).
Each step is one binary32 operation rounded to nearest-even (this
implementation's reading; see ``scaling``).  The reconstructed value is
x_hat_i = dec * s_B * q_i with dec = g / (T F).

Blockings (Sec. 2.3 and Table 5: 1D blocks of 16 along the GEMM contraction
dimension for activations and gradients, 2D 16x16 tiles for weights):

* ``quantize_1d(axis=1)``: blocks of 16 consecutive elements of a row.
  payload [R, C/2] (byte [r, c/2] = nib(r, c) | nib(r, c+1) << 4),
  scales [R, C/16].
* ``quantize_1d(axis=0)``: blocks of 16 consecutive rows of a column.  The
  output is stored transposed, i.e. as the row blocking of x^T:
  payload [C, R/2] (byte [c, r/2] = nib(r, c) | nib(r+1, c) << 4),
  scales [C, R/16].
* ``quantize_2d``: 16x16 tiles aligned at (0, 0).  payload [R, C/2],
  scales [R/16, C/16], and the transposed payload [C, R/2] of the same
  nibbles.

SR words: element (r, c) of an R x C source uses ``philox.sr_words(seed,
tensor_id, r * C + c)``, independent of the blocking.

Comparison scale formats (``fmt``; Sec. 2, Table tab:formats):

* ``"ue5m3"`` (default): the recipe above, blocks of 16 (``block=32`` and
  ``tile=32``: the block-size control, 1D blocks of 32 and 32x32 weight
  tiles, same arithmetic on the larger blocks).
* ``"e4m3"``: the NVFP4 arrangement -- blocks of 16 with an E4M3 block scale
  under the FP32 tensor scale.  Same steps with step 3 the nearest E4M3 code
  (ties to even, saturating at 448) and the zero rule giving the E4M3 code
  of 1.0 (0x38).
* ``"e8m0"``: the MXFP4 arrangement -- blocks of 32, a power-of-two E8M0
  block scale and no tensor scale (dec = 1).  The paper gives no exponent
  rule; this oracle takes the OCP microscaling one: with a_B > 0,
  E = clamp(floor(log2 a_B) - 2, -127, 127) (2 = exponent of E2M1's largest
  value 6), code = E + 127, r_B = 2**-E, y_i = x_i * r_B (exact), so
  |y| < 8 and E2M1 saturation clips (6, 8) to 6; a_B = 0 gives code 0.
"""

import numpy as np

from . import formats, philox, scaling


FORMATS = ("ue5m3", "e4m3", "e8m0")


def block_size(fmt, block=None):
    """Elements per block (1D) for a scale format: E8M0 32; UE5M3 and E4M3
    16, or 32 for the block-size control (``block=32``)."""
    if fmt not in FORMATS:
        raise ValueError(fmt)
    if fmt == "e8m0":
        if block not in (None, 32):
            raise ValueError("E8M0 blocks are 32")
        return 32
    if block not in (None, 16, 32):
        raise ValueError("block must be 16 or 32")
    return block or 16


def scale_decode(fmt, code):
    """Value of block-scale codes of a format (float64)."""
    if fmt == "ue5m3":
        return formats.ue5m3_decode(code)
    if fmt == "e4m3":
        return formats.e4m3_decode(code)
    if fmt == "e8m0":
        return formats.e8m0_decode(code)
    raise ValueError(fmt)


def _e8m0_codes(a_B):
    """OCP microscaling exponent of each block maximum (module header)."""
    a = np.asarray(a_B, dtype=np.float64)
    _, e = np.frexp(a)                                      # a = m 2**e, m in [0.5, 1)
    E = np.clip(e.astype(np.int64) - 1 - 2, -127, 127)
    return np.where(a > 0, E + 127, 0).astype(np.uint8)


def _block_codes(xb, S, G, mode, words, fmt="ue5m3", chunk=1 << 16):
    """xb: float32 [nb, B].  Returns (scale codes uint8 [nb], nibbles [nb, B]).
    Blocks are independent; large inputs are processed ``chunk`` blocks at a
    time only to bound memory."""
    xb = np.asarray(xb, dtype=np.float32)
    if xb.shape[0] > chunk:
        parts = [_block_codes(xb[i:i + chunk], S, G, mode,
                              None if words is None else words[i:i + chunk], fmt, chunk)
                 for i in range(0, xb.shape[0], chunk)]
        return (np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts]))
    a_B = np.max(np.abs(xb), axis=1) if xb.shape[1] else np.zeros(xb.shape[0], np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        if fmt == "e8m0":
            code = _e8m0_codes(a_B)
            r_B = np.ldexp(np.float32(1.0), 127 - code.astype(np.int32)).astype(np.float32)
        else:
            u_B = (a_B * np.float32(S)).astype(np.float32)
            if fmt == "ue5m3":
                code = formats.ue5m3_encode_rne_sat(u_B)
                code = np.where(code == 0, formats.UE5M3_ONE, code).astype(np.uint8)
            elif fmt == "e4m3":
                code = formats.e4m3_encode_rne_sat(u_B)
                code = np.where(code == 0, formats.E4M3_ONE, code).astype(np.uint8)
            else:
                raise ValueError(fmt)
            s_hat = scale_decode(fmt, code).astype(np.float32)
            r_B = (np.float32(G) / s_hat).astype(np.float32)
        y = (xb * r_B[:, None]).astype(np.float32)
    if mode == "rn":
        nib = formats.e2m1_encode_rne(y)
    elif mode == "sr":
        nib = formats.e2m1_encode_sr(y, words)
    else:
        raise ValueError(mode)
    return code, nib


def _pack_rows(nib):
    """[R, C] nibbles -> [R, C/2] bytes, low nibble = even column."""
    nib = np.asarray(nib, dtype=np.uint8)
    return (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)


def _unpack_rows(payload):
    p = np.asarray(payload, dtype=np.uint8)
    out = np.empty((p.shape[0], p.shape[1] * 2), dtype=np.uint8)
    out[:, 0::2] = p & 15
    out[:, 1::2] = p >> 4
    return out


def _words_for(shape, seed, tensor_id, mode, elem_index):
    if mode != "sr":
        return None
    R, C = shape
    if elem_index is None:
        elem_index = np.arange(R * C, dtype=np.int64).reshape(R, C)
    return philox.sr_words(seed, tensor_id, np.asarray(elem_index, np.int64))


def quantize_1d(x_bits, axis, g, target=448.0, mode="rn", seed=0, tensor_id=0, elem_index=None,
                fmt="ue5m3", block=None):
    """1D block quantization of a bf16 matrix (blocks of 16, or 32 for
    E8M0).  Returns (payload, scales, dec) in the layouts described in the
    module header.  ``elem_index`` (SR only) gives each element's row-major
    index in the source tensor when ``x_bits`` is a sampled part of it
    (default: x itself is the source).  E8M0 ignores g and target (no tensor
    scale) and returns dec = 1."""
    return quantize_1d_values(scaling.bf16_to_f32(x_bits), axis, g, target, mode, seed, tensor_id,
                              elem_index, fmt, block)


def quantize_1d_values(x, axis, g, target=448.0, mode="rn", seed=0, tensor_id=0, elem_index=None,
                       fmt="ue5m3", block=None):
    """``quantize_1d`` of a float32 matrix (values already widened, or a
    transformed operand)."""
    x = np.asarray(x, dtype=np.float32)
    R, C = x.shape
    B = block_size(fmt, block)
    if fmt == "e8m0":
        S, G, dec = np.float32(1.0), np.float32(1.0), np.float32(1.0)
    else:
        S, G, dec = scaling.tensor_multipliers(g, target)
    words = _words_for((R, C), seed, tensor_id, mode, elem_index)
    if axis == 1:
        if C % B:
            raise ValueError(f"cols must be a multiple of {B}")
        xb = x.reshape(R * (C // B), B)
        wb = None if words is None else words.reshape(R * (C // B), B)
        code, nib = _block_codes(xb, S, G, mode, wb, fmt)
        return _pack_rows(nib.reshape(R, C)), code.reshape(R, C // B), dec
    if axis == 0:
        if R % B:
            raise ValueError(f"rows must be a multiple of {B}")
        xt = np.ascontiguousarray(x.T)                     # [C, R]
        xb = xt.reshape(C * (R // B), B)
        wb = None if words is None else np.ascontiguousarray(words.T).reshape(C * (R // B), B)
        code, nib = _block_codes(xb, S, G, mode, wb, fmt)
        return _pack_rows(nib.reshape(C, R)), code.reshape(C, R // B), dec
    raise ValueError("axis must be 0 or 1")


def quantize_2d(x_bits, g, target=448.0, mode="rn", seed=0, tensor_id=0, elem_index=None,
                fmt="ue5m3", tile=16):
    """tile x tile quantization (UE5M3 or E4M3 scales; 16, or 32 for the
    block-size control).  Returns (payload [R, C/2], scales [R/tile,
    C/tile], payload_t [C, R/2], dec)."""
    if fmt not in ("ue5m3", "e4m3"):
        raise ValueError("2D tiles take UE5M3 or E4M3 scales")
    if tile not in (16, 32):
        raise ValueError("tile must be 16 or 32")
    x = scaling.bf16_to_f32(x_bits)
    R, C = x.shape
    B = tile
    if R % B or C % B:
        raise ValueError(f"rows and cols must be multiples of {B}")
    S, G, dec = scaling.tensor_multipliers(g, target)
    words = _words_for((R, C), seed, tensor_id, mode, elem_index)
    tiles = x.reshape(R // B, B, C // B, B).transpose(0, 2, 1, 3).reshape(-1, B * B)
    wt = None
    if words is not None:
        wt = words.reshape(R // B, B, C // B, B).transpose(0, 2, 1, 3).reshape(-1, B * B)
    code, nib = _block_codes(tiles, S, G, mode, wt, fmt)
    nib = nib.reshape(R // B, C // B, B, B).transpose(0, 2, 1, 3).reshape(R, C)
    return (_pack_rows(nib), code.reshape(R // B, C // B),
            _pack_rows(np.ascontiguousarray(nib.T)), dec)


# ------------------------------------------------------ dequantization ----
def decoded_1d(payload, scales, axis, fmt="ue5m3", block=None):
    """Decoded operand q * s_B (float64, exact) in the logical [R, C] shape
    of the tensor that ``quantize_1d`` consumed."""
    q = formats.e2m1_decode(_unpack_rows(payload))         # [rows_stored, L]
    s = scale_decode(fmt, scales)
    v = q * np.repeat(s, block_size(fmt, block), axis=1)
    return v if axis == 1 else np.ascontiguousarray(v.T)


def decoded_2d(payload, scales, fmt="ue5m3", tile=16):
    """Decoded weight q * s_tile (float64, exact), logical [R, C]."""
    q = formats.e2m1_decode(_unpack_rows(payload))
    s = scale_decode(fmt, scales)
    return q * np.repeat(np.repeat(s, tile, axis=0), tile, axis=1)


def decoded_2d_t(payload_t, scales, fmt="ue5m3", tile=16):
    """Decoded weight from the transposed payload, logical [R, C]."""
    q = formats.e2m1_decode(_unpack_rows(payload_t)).T
    s = scale_decode(fmt, scales)
    return q * np.repeat(np.repeat(s, tile, axis=0), tile, axis=1)


def dequantize(decoded, dec):
    """x_hat = dec * (q * s_B) in float64."""
    return np.float64(np.float32(dec)) * decoded
