"""Tensor scale management (oracle; test infrastructure only).

* amax (Sec. 4.1): a_t = max_i |x_{t,i}| over the whole tensor.
* Periodic sample-and-hold (eq:delayed-amax): at optimizer step t the
  reference is the freshly measured a_t when no cache exists or when
  t - tau >= D (tau = step of the last refresh), otherwise the cached value;
  the cache starts empty and is reset (not restored) on resume; D = 50 with
  multiplicative factor 1 in the paper's recipe, D = 1 is current scaling.
* Inference-scale policies (Sec. "Inference with delayed scaling", Table
  tab:inference-scale-summary, App. "Inference-Scale Sensitivity"): a
  loaded weight's amax is measured once and then held (read here as period
  D = 0: refresh only while the cache is empty); activations either follow
  D = 50 from an empty cache, D = 1, or a calibrated reference -- the
  largest amax seen over calibration batches -- held fixed (``freeze``).
* Tensor multipliers (Sec. 4.2, eq:scale-target): with F = 6 and target T
  (448 by default, 2048 for the wgrad-dY override), G = T F / g and the ideal
  block-scale code of a block with maximum a_B is u_B = a_B T / g.

Binary32 reading of these real formulas (one IEEE round-to-nearest-even per
operation, no fused operations):
    TF  = RN(T * 6)
    S   = RN(T / g)          u_B = RN(a_B * S)
    G   = RN(TF / g)
    dec = RN(g / TF)         (decode multiplier, 1/G up to rounding)
Degenerate references (paper silent): if g is not a positive finite number,
or G is not below 2**110 (so that G / (smallest scale 2**-17) stays finite),
g is replaced by 1.
"""

import numpy as np

F = np.float32(6.0)
G_LIMIT = np.float32(2.0 ** 110)


def bf16_to_f32(bits):
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def amax(x_bf16_bits):
    """max |x| of a bf16 tensor as float32 (0 for an empty tensor)."""
    x = bf16_to_f32(x_bf16_bits)
    if x.size == 0:
        return np.float32(0.0)
    return np.float32(np.max(np.abs(x)))


def tensor_multipliers(g, target):
    """Return (S, G, dec) as float32 for held amax ``g`` and target T."""
    T = np.float32(target)
    g = np.float32(g)
    with np.errstate(divide="ignore", over="ignore", invalid="ignore"):
        TF = np.float32(T * F)
        ok = bool(g > 0) and bool(np.isfinite(g))
        if ok:
            G = np.float32(TF / g)
            ok = bool(np.isfinite(G)) and bool(G < G_LIMIT)
        if not ok:
            g = np.float32(1.0)
        S = np.float32(T / g)
        G = np.float32(TF / g)
        dec = np.float32(g / TF)
    return S, G, dec


def calibrated_amax(batches):
    """Calibrated-frozen reference: the largest tensor amax over a sequence
    of calibration batches (bf16 bit arrays); 0 for no batches."""
    g = np.float32(0.0)
    for b in batches:
        g = max(g, amax(b))
    return np.float32(g)


class AmaxState:
    """One operand's sample-and-hold cache (eq:delayed-amax).  ``period`` 0
    holds the first measurement until ``reset``."""

    def __init__(self, period=50):
        if period < 0:
            raise ValueError("period must be >= 0")
        self.period = int(period)
        self.reset()

    def reset(self):
        """Empty cache: the next observation refreshes (process launch or
        resume, Sec. 4.1)."""
        self.has_cache = False
        self.last_refresh = 0
        self.g = np.float32(0.0)

    def needs_refresh(self, step):
        if not self.has_cache:
            return True
        return self.period > 0 and step - self.last_refresh >= self.period

    def freeze(self, g):
        """Hold the given reference from now on (calibrated-frozen policy)."""
        self.g = np.float32(g)
        self.has_cache = True
        self.period = 0

    def observe(self, x_bf16_bits, step):
        """Reference amax for optimizer step ``step``; returns (g, refreshed)."""
        return self.observe_amax(lambda: amax(x_bf16_bits), step)

    def observe_amax(self, amax_of, step):
        """``observe`` with the tensor amax supplied by ``amax_of()`` (called
        only on a refresh)."""
        if self.needs_refresh(step):
            self.g = np.float32(amax_of())
            self.last_refresh = int(step)
            self.has_cache = True
            return self.g, True
        return self.g, False
