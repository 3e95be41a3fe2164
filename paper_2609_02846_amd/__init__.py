"""UE5M3 FP4 quantize-and-GEMM for MI355X (gfx950).

Thin Python binding of the C ABI in include/ue5m3.h (libue5m3.so, built
in-tree by ``paper_2609_02846_amd.build``).  Every step of the hot path runs
in the library's HIP kernels; this module only marshals arguments: torch
tensors supply device memory and the current HIP stream.

The library is required: importing the binding functions raises if
libue5m3.so is missing, and there is no CPU fallback.
"""

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libue5m3.so")

UE5M3_OK, UE5M3_EINVAL, UE5M3_ESHAPE, UE5M3_EALIGN, UE5M3_ELAYOUT, UE5M3_EHIP, UE5M3_ESCRATCH = range(7)
RN, SR = 0, 1
NT, NN, TN = 0, 1, 2
OUT_F32, OUT_BF16 = 0, 1
_MODES = {"rn": RN, "sr": SR}
_LAYOUTS = {"nt": NT, "nn": NN, "tn": TN}
ROW16, COL16T, TILE16, ROW32, COL32T, TILE32 = range(6)
_BLOCKINGS = {("row", 16): ROW16, ("colT", 16): COL16T, ("tile", 16): TILE16,
              ("row", 32): ROW32, ("colT", 32): COL32T, ("tile", 32): TILE32}
SCALE_UE5M3, SCALE_E4M3, SCALE_E8M0 = 0, 1, 2
_FORMATS = {"ue5m3": SCALE_UE5M3, "e4m3": SCALE_E4M3, "e8m0": SCALE_E8M0}
BLOCK = {"ue5m3": 16, "e4m3": 16, "e8m0": 32}

EXPORTED_SYMBOLS = (
    "ue5m3_amax_state_init", "ue5m3_amax_state_reset", "ue5m3_amax_sample",
    "ue5m3_amax_state_freeze", "ue5m3_amax_accumulate",
    "ue5m3_quantize_1d", "ue5m3_quantize_2d", "ue5m3_gemm",
    "ue5m3_quantize_1d_ex", "ue5m3_quantize_2d_ex", "ue5m3_gemm_ex", "ue5m3_quantize_dual",
    "ue5m3_gemm_pm", "ue5m3_amax_sample_rht", "ue5m3_quantize_cols_rht",
    "ue5m3_status_string", "ue5m3_version", "ue5m3_gemm_noalloc",
)


class AmaxStateC(ctypes.Structure):
    """Mirror of ue5m3_amax_state_t."""
    _fields_ = [("amax_dev", ctypes.c_void_p), ("last_refresh", ctypes.c_int64),
                ("period", ctypes.c_int32), ("has_cache", ctypes.c_int32)]


class UE5M3Error(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


_lib = None


def load_library(path=LIB_PATH):
    """Load libue5m3.so and declare the C signatures.  Raises OSError if the
    library has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise OSError(f"{path} not found: build it with `python -m paper_2609_02846_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i64, i32, u32, u64, f32 = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                   ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float)
    lib.ue5m3_amax_state_init.argtypes = [ctypes.POINTER(AmaxStateC), vp, i32]
    lib.ue5m3_amax_state_init.restype = i32
    lib.ue5m3_amax_state_reset.argtypes = [ctypes.POINTER(AmaxStateC)]
    lib.ue5m3_amax_state_reset.restype = None
    lib.ue5m3_amax_sample.argtypes = [ctypes.POINTER(AmaxStateC), vp, i64, i64,
                                      ctypes.POINTER(ctypes.c_int32), vp]
    lib.ue5m3_amax_sample.restype = i32
    lib.ue5m3_amax_state_freeze.argtypes = [ctypes.POINTER(AmaxStateC)]
    lib.ue5m3_amax_state_freeze.restype = None
    lib.ue5m3_amax_accumulate.argtypes = [vp, i64, vp, i32, vp]
    lib.ue5m3_amax_accumulate.restype = i32
    lib.ue5m3_quantize_1d.argtypes = [vp, i64, i64, i32, vp, f32, i32, u64, u32, vp, vp, vp, vp]
    lib.ue5m3_quantize_1d.restype = i32
    lib.ue5m3_quantize_2d.argtypes = [vp, i64, i64, vp, f32, i32, u64, u32, vp, vp, vp, vp, vp, vp]
    lib.ue5m3_quantize_2d.restype = i32
    lib.ue5m3_gemm.argtypes = [i32, i64, i64, i64, vp, vp, i32, vp, vp, vp, i32, vp, vp, i32, vp]
    lib.ue5m3_gemm.restype = i32
    lib.ue5m3_quantize_1d_ex.argtypes = [vp, i64, i64, i32, vp, f32, i32, u64, u32, i32, i32,
                                         vp, vp, vp, vp]
    lib.ue5m3_quantize_1d_ex.restype = i32
    lib.ue5m3_quantize_2d_ex.argtypes = [vp, i64, i64, vp, f32, i32, u64, u32, i32, i32,
                                         vp, vp, vp, vp, vp, vp]
    lib.ue5m3_quantize_2d_ex.restype = i32
    lib.ue5m3_gemm_ex.argtypes = [i32, i64, i64, i64, vp, vp, i32, vp, vp, vp, i32, vp, vp, i32, i32, vp]
    lib.ue5m3_gemm_ex.restype = i32
    lib.ue5m3_gemm_noalloc.argtypes = [i32, i64, i64, i64, vp, vp, i32, vp, vp, vp, i32, vp, vp, i32, vp]
    lib.ue5m3_gemm_noalloc.restype = i32
    lib.ue5m3_amax_sample_rht.argtypes = [ctypes.POINTER(AmaxStateC), vp, i64, i64, u32, i64,
                                          ctypes.POINTER(ctypes.c_int32), vp]
    lib.ue5m3_amax_sample_rht.restype = i32
    lib.ue5m3_quantize_cols_rht.argtypes = [vp, i64, i64, vp, f32, i32, u64, u32, u32, vp, vp, vp, vp]
    lib.ue5m3_quantize_cols_rht.restype = i32
    lib.ue5m3_gemm_pm.argtypes = [i32, i64, i64, i64, vp, vp, i32, vp, vp, vp, i32, vp, vp, i32, i32, i32,
                                  vp]
    lib.ue5m3_gemm_pm.restype = i32
    lib.ue5m3_quantize_dual.argtypes = [vp, i64, i64, vp, f32, i32, u64, u32, u32, i32,
                                        vp, vp, vp, vp, vp, vp]
    lib.ue5m3_quantize_dual.restype = i32
    lib.ue5m3_status_string.argtypes = [i32]
    lib.ue5m3_status_string.restype = ctypes.c_char_p
    lib.ue5m3_version.argtypes = []
    lib.ue5m3_version.restype = i32
    _lib = lib
    return lib


def status_string(status):
    return load_library().ue5m3_status_string(int(status)).decode()


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(status, what):
    if status != UE5M3_OK:
        raise UE5M3Error(status, what)


def _bf16_2d(x, name):
    if x.dtype != torch.bfloat16 or x.dim() != 2 or not x.is_contiguous() or not x.is_cuda:
        raise ValueError(f"{name} must be a contiguous 2-D bf16 CUDA/HIP tensor")
    return x


def _u8(shape, like):
    return torch.empty(shape, dtype=torch.uint8, device=like.device)


def _numel(shape):
    n = 1
    for d in shape:
        n *= int(d)
    return n


def _dev_buf(t, dtype, numel, name):
    """The library takes bare pointers: check that a buffer it reads or
    writes is a contiguous device tensor of the dtype with room for
    ``numel`` elements."""
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} CUDA/HIP tensor")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, {numel} needed")
    return t


def _u8_out(t, shape, name):
    return _dev_buf(t, torch.uint8, _numel(shape), name)


def _f32_out(t, name):
    return _dev_buf(t, torch.float32, 1, name)


# ------------------------------------------------------------------ API ---
class AmaxState:
    """One operand's sample-and-hold cache (eq:delayed-amax): host integers
    plus a device float holding the sampled amax.  ``period`` 50 is the
    training recipe, 1 current scaling, 0 measure-once-and-hold."""

    def __init__(self, period=50, device="cuda"):
        self.amax = torch.zeros(1, dtype=torch.float32, device=device)
        self.c = AmaxStateC()
        self.set_period(period)

    def set_period(self, period):
        """Re-initialise with another period; the cache is emptied."""
        _check(load_library().ue5m3_amax_state_init(ctypes.byref(self.c), _ptr(self.amax),
                                                     int(period)), "ue5m3_amax_state_init")

    def reset(self):
        load_library().ue5m3_amax_state_reset(ctypes.byref(self.c))

    def freeze(self):
        """Hold the reference now in ``amax`` until reset (calibrated-frozen
        policy; fill ``amax`` with ``amax_accumulate`` first)."""
        load_library().ue5m3_amax_state_freeze(ctypes.byref(self.c))

    @property
    def period(self):
        return int(self.c.period)

    @property
    def has_cache(self):
        return bool(self.c.has_cache)

    @property
    def last_refresh(self):
        return int(self.c.last_refresh)


def amax_sample(state, x, step, stream=None):
    """Refresh ``state`` from tensor ``x`` if the rule of eq:delayed-amax asks
    for it at optimizer step ``step``; returns True when a refresh was
    enqueued."""
    if x.dtype != torch.bfloat16 or not x.is_contiguous() or not x.is_cuda:
        raise ValueError("x must be a contiguous bf16 CUDA/HIP tensor")
    flag = ctypes.c_int32(0)
    _check(load_library().ue5m3_amax_sample(ctypes.byref(state.c), _ptr(x), x.numel(), int(step),
                                            ctypes.byref(flag), _stream(stream)),
           "ue5m3_amax_sample")
    return bool(flag.value)


def amax_accumulate(x, amax_dev, clear=False, stream=None):
    """Enqueue amax_dev = max(0 if clear else amax_dev, max |x|) (see
    ue5m3_amax_accumulate): the running maximum over calibration batches."""
    if x.dtype != torch.bfloat16 or not x.is_contiguous() or not x.is_cuda:
        raise ValueError("x must be a contiguous bf16 CUDA/HIP tensor")
    _f32_out(amax_dev, "amax_dev")
    _check(load_library().ue5m3_amax_accumulate(_ptr(x), x.numel(), _ptr(amax_dev), int(bool(clear)),
                                                _stream(stream)), "ue5m3_amax_accumulate")
    return amax_dev


def amax_sample_rht(state, x, sign_mask, step, stream=None):
    """amax_sample for the randomized Hadamard transform of x's 16-row
    column blocks (see ue5m3_amax_sample_rht)."""
    _bf16_2d(x, "x")
    flag = ctypes.c_int32(0)
    _check(load_library().ue5m3_amax_sample_rht(ctypes.byref(state.c), _ptr(x), x.shape[0], x.shape[1],
                                                int(sign_mask), int(step), ctypes.byref(flag),
                                                _stream(stream)), "ue5m3_amax_sample_rht")
    return bool(flag.value)


def quantize_cols_rht(x, amax_dev, sign_mask, target=448.0, mode="rn", seed=0, tensor_id=0,
                      payload_t=None, scales_t=None, dec_out=None, stream=None):
    """COL16 quantization of the transformed x (see ue5m3_quantize_cols_rht).
    Returns (payload_t [C, R/2], scales_t [C, R/16], dec_out)."""
    _bf16_2d(x, "x")
    R, C = x.shape
    payload_t = _u8((C, R // 2), x) if payload_t is None else _u8_out(payload_t, (C, R // 2), "payload_t")
    scales_t = _u8((C, R // 16), x) if scales_t is None else _u8_out(scales_t, (C, R // 16), "scales_t")
    if dec_out is None:
        dec_out = torch.empty(1, dtype=torch.float32, device=x.device)
    _f32_out(dec_out, "dec_out")
    _f32_out(amax_dev, "amax_dev")
    _check(load_library().ue5m3_quantize_cols_rht(
        _ptr(x), R, C, _ptr(amax_dev), float(target), _MODES[mode], int(seed) & (2**64 - 1),
        int(tensor_id) & 0xFFFFFFFF, int(sign_mask), _ptr(payload_t), _ptr(scales_t), _ptr(dec_out),
        _stream(stream)), "ue5m3_quantize_cols_rht")
    return payload_t, scales_t, dec_out


def quantize_1d(x, axis, amax_dev, target=448.0, mode="rn", seed=0, tensor_id=0,
                payload=None, scales=None, dec_out=None, stream=None, fmt="ue5m3", block=None):
    """1D block quantization (see ue5m3_quantize_1d and, for ``fmt`` "e4m3"
    or "e8m0" or ``block`` 32, ue5m3_quantize_1d_ex).  Returns (payload,
    scales, dec_out); axis 0 outputs are stored transposed.  E8M0 takes no
    amax (None)."""
    _bf16_2d(x, "x")
    R, C = x.shape
    B = BLOCK[fmt] if block is None else int(block)
    if axis == 1:
        pshape, sshape = (R, C // 2), (R, C // B)
    elif axis == 0:
        pshape, sshape = (C, R // 2), (C, R // B)
    else:
        raise ValueError("axis must be 0 or 1")
    payload = _u8(pshape, x) if payload is None else _u8_out(payload, pshape, "payload")
    scales = _u8(sshape, x) if scales is None else _u8_out(scales, sshape, "scales")
    if dec_out is None:
        dec_out = torch.empty(1, dtype=torch.float32, device=x.device)
    _f32_out(dec_out, "dec_out")
    if fmt != "e8m0":
        _f32_out(amax_dev, "amax_dev")
    lib = load_library()
    common = (_ptr(x), R, C, int(axis), _ptr(amax_dev), float(target), _MODES[mode],
              int(seed) & (2**64 - 1), int(tensor_id) & 0xFFFFFFFF)
    if fmt == "ue5m3" and B == 16:
        st = lib.ue5m3_quantize_1d(*common, _ptr(payload), _ptr(scales), _ptr(dec_out), _stream(stream))
    else:
        st = lib.ue5m3_quantize_1d_ex(*common, _FORMATS[fmt], B, _ptr(payload), _ptr(scales),
                                      _ptr(dec_out), _stream(stream))
    _check(st, "ue5m3_quantize_1d")
    return payload, scales, dec_out


def quantize_dual(x, amax_dev, target=448.0, mode="rn", seed=0, tensor_id_r=0, tensor_id_c=0,
                  rows_out=None, cols_out=None, dec_out=None, stream=None, fmt="ue5m3"):
    """Both 1D blockings of ``x`` from one read (see ue5m3_quantize_dual).
    Returns ((payload_r, scales_r, dec), (payload_c, scales_c, dec)) laid out
    exactly as quantize_1d's axis-1 and axis-0 results."""
    _bf16_2d(x, "x")
    R, C = x.shape
    pr, sr_ = rows_out if rows_out is not None else (_u8((R, C // 2), x), _u8((R, C // 16), x))
    pc, sc = cols_out if cols_out is not None else (_u8((C, R // 2), x), _u8((C, R // 16), x))
    _u8_out(pr, (R, C // 2), "payload_r")
    _u8_out(sr_, (R, C // 16), "scales_r")
    _u8_out(pc, (C, R // 2), "payload_c")
    _u8_out(sc, (C, R // 16), "scales_c")
    if dec_out is None:
        dec_out = torch.empty(1, dtype=torch.float32, device=x.device)
    _f32_out(dec_out, "dec_out")
    _f32_out(amax_dev, "amax_dev")
    _check(load_library().ue5m3_quantize_dual(
        _ptr(x), R, C, _ptr(amax_dev), float(target), _MODES[mode], int(seed) & (2**64 - 1),
        int(tensor_id_r) & 0xFFFFFFFF, int(tensor_id_c) & 0xFFFFFFFF, _FORMATS[fmt], _ptr(pr),
        _ptr(sr_), _ptr(pc), _ptr(sc), _ptr(dec_out), _stream(stream)), "ue5m3_quantize_dual")
    return (pr, sr_, dec_out), (pc, sc, dec_out)


def quantize_2d(w, amax_dev, target=448.0, mode="rn", seed=0, tensor_id=0, transposed=True,
                payload=None, scales=None, payload_t=None, dec_out=None, scales_t=None,
                stream=None, fmt="ue5m3", tile=16):
    """Square-tile quantization, tiles of 16 x 16 (see ue5m3_quantize_2d) or,
    with ``tile`` 32 or ``fmt`` "e4m3", ue5m3_quantize_2d_ex.  Returns
    (payload, scales, payload_t or None, dec_out, scales_t or None); the
    transposed payload and scales are the dgrad operand."""
    _bf16_2d(w, "w")
    R, C = w.shape
    T = int(tile)
    payload = _u8((R, C // 2), w) if payload is None else _u8_out(payload, (R, C // 2), "payload")
    scales = _u8((R // T, C // T), w) if scales is None else _u8_out(scales, (R // T, C // T), "scales")
    if transposed and payload_t is None:
        payload_t = _u8((C, R // 2), w)
    if transposed and scales_t is None:
        scales_t = _u8((C // T, R // T), w)
    if payload_t is not None:
        _u8_out(payload_t, (C, R // 2), "payload_t")
    if scales_t is not None:
        _u8_out(scales_t, (C // T, R // T), "scales_t")
    if dec_out is None:
        dec_out = torch.empty(1, dtype=torch.float32, device=w.device)
    _f32_out(dec_out, "dec_out")
    _f32_out(amax_dev, "amax_dev")
    lib = load_library()
    common = (_ptr(w), R, C, _ptr(amax_dev), float(target), _MODES[mode], int(seed) & (2**64 - 1),
              int(tensor_id) & 0xFFFFFFFF)
    outs = (_ptr(payload), _ptr(scales), _ptr(payload_t), _ptr(scales_t), _ptr(dec_out), _stream(stream))
    if fmt == "ue5m3" and T == 16:
        st = lib.ue5m3_quantize_2d(*common, *outs)
    else:
        st = lib.ue5m3_quantize_2d_ex(*common, _FORMATS[fmt], T, *outs)
    _check(st, "ue5m3_quantize_2d")
    return payload, scales, payload_t, dec_out, scales_t


def recipe_blockings(layout, fmt="ue5m3"):
    """The operand blockings the recipe's quantizers produce for each product
    (Table 5): fprop A rows, B weight tiles; dgrad A rows, B transposed
    weight tiles; wgrad both operands blocked down their columns (stored
    transposed).  E8M0 weights are 1D-blocked along each contraction."""
    lay = _LAYOUTS[layout] if isinstance(layout, str) else int(layout)
    if lay == TN:
        return "colT", "colT"
    if fmt == "e8m0":
        return "row", ("row" if lay == NT else "colT")
    return "row", "tile"


def _blocking(kind, Bk):
    if isinstance(kind, int):
        return kind
    return _BLOCKINGS[(kind, Bk)]


def _gemm_args(layout, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, out, out_dtype, fmt, Bk,
               a_blk, b_blk):
    lay = _LAYOUTS[layout] if isinstance(layout, str) else int(layout)
    da, db = recipe_blockings(lay, fmt)
    a_blk = da if a_blk is None else a_blk
    b_blk = db if b_blk is None else b_blk
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=a.device)
    ctype = OUT_BF16 if out.dtype == torch.bfloat16 else OUT_F32
    if out.dtype not in (torch.float32, torch.bfloat16) or not out.is_contiguous():
        raise ValueError("out must be a contiguous fp32 or bf16 tensor")
    _dev_buf(out, out.dtype, int(M) * int(N), "out")
    if M > 0 and N > 0 and K > 0:
        tiled = b_blk in ("tile", TILE16, TILE32)
        _u8_out(a, (M, K // 2), "a")
        _u8_out(a_scales, (M, K // Bk), "a_scales")
        _u8_out(b, (N, K // 2), "b")
        _u8_out(b_scales, ((N + Bk - 1) // Bk, K // Bk) if tiled else (N, K // Bk), "b_scales")
    if M > 0 and N > 0:
        _f32_out(a_dec, "a_dec")
        _f32_out(b_dec, "b_dec")
    args = (lay, int(M), int(N), int(K), _ptr(a), _ptr(a_scales), _blocking(a_blk, Bk), _ptr(a_dec), _ptr(b),
            _ptr(b_scales), _blocking(b_blk, Bk), _ptr(b_dec), _ptr(out), ctype)
    return out, args


def gemm_pm(layout, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, out=None,
            out_dtype=torch.float32, grid=1024, stream=None, fmt="ue5m3", block=16, a_blk=None, b_blk=None):
    """Probe-matched GEMM (see ue5m3_gemm_pm): 64-product RNE partials,
    toward-zero cross-group adds, snap of the encoded accumulator to the
    1/``grid`` lattice (0: none), then alpha.  Operands and blockings as
    ``gemm``."""
    if fmt not in ("ue5m3", "e4m3"):
        raise ValueError("the probe-matched GEMM takes UE5M3 or E4M3 scales")
    out, args = _gemm_args(layout, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, out, out_dtype, fmt,
                           int(block), a_blk, b_blk)
    _check(load_library().ue5m3_gemm_pm(*args, _FORMATS[fmt], int(grid), _stream(stream)), "ue5m3_gemm_pm")
    return out


def gemm(layout, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, out=None,
         out_dtype=torch.float32, stream=None, fmt="ue5m3", block=None, a_blk=None, b_blk=None):
    """Decoded-operand FP4 GEMM (see ue5m3_gemm and, for ``fmt`` "e4m3" or
    "e8m0" or ``block`` 32, ue5m3_gemm_ex); layout is "nt" (fprop), "nn"
    (dgrad) or "tn" (wgrad).  ``a_blk`` / ``b_blk`` name each operand's
    blocking ("row", "colT", "tile" or a ue5m3_blocking_t value); None takes
    the recipe's blocking for the layout (``recipe_blockings``).  Returns the
    [M, N] output tensor."""
    Bk = BLOCK[fmt] if block is None else int(block)
    out, args = _gemm_args(layout, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, out, out_dtype, fmt, Bk,
                           a_blk, b_blk)
    lib = load_library()
    if fmt == "ue5m3" and Bk == 16:
        st = lib.ue5m3_gemm(*args, _stream(stream))
    else:
        st = lib.ue5m3_gemm_ex(*args, _FORMATS[fmt], _stream(stream))
    _check(st, "ue5m3_gemm")
    return out


def gemm_noalloc(layout, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, out, stream=None, a_blk=None,
                 b_blk=None):
    """ue5m3_gemm_noalloc: ``gemm`` (UE5M3, blocks of 16) with its split
    partials in the library's static scratch array, for callers that cannot
    allocate.  ``out`` (fp32 or bf16 [M, N]) is required: nothing is
    allocated here either."""
    if out is None:
        raise ValueError("gemm_noalloc allocates nothing: pass out")
    out, args = _gemm_args(layout, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, out, out.dtype, "ue5m3", 16,
                           a_blk, b_blk)
    _check(load_library().ue5m3_gemm_noalloc(*args, _stream(stream)), "ue5m3_gemm_noalloc")
    return out
