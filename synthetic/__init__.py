"""Seeded synthetic inputs shared by the oracle-side tests, the GPU parity
tests and the benchmark.

This module holds no arithmetic of the quantization method: it only draws
random tensors and rounds them to bf16 (the input format of the linear's
operands).  The paper's training data, checkpoints and native GPU outputs are
not available; these tensors stand in for them with the shapes of the
Nemotron-H 8B linears (hidden 4096, FFN 21504, 8192-token sequences) and
distributions chosen to exercise the method: Gaussian bodies, sparse large
outliers in activations, small-magnitude gradients with a heavy per-row
spread, N(0, 0.02) weights.

Every generator uses NumPy's PCG64 seeded by SeedSequence([seed, role]) so a
given (seed, role) always yields the same bytes on every machine.
"""

import numpy as np

ROLE_X, ROLE_W, ROLE_DY, ROLE_OUTLIER, ROLE_ROWSCALE, ROLE_MISC, ROLE_DRIFT = range(7)


def rng_for(seed, role):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), int(role)])))


def f32_to_bf16_bits(x):
    """Round float32 to bf16 (nearest, ties to even) and return the uint16
    bit patterns.  Inputs must be finite."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal(seed, role, shape, std=1.0):
    r = rng_for(seed, role)
    x = r.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def add_outliers(x, seed, fraction, factor):
    """Multiply exactly round(fraction * numel) distinct, uniformly chosen
    entries by ``factor`` (sign kept)."""
    n = x.size
    k = int(round(fraction * n))
    if k:
        r = rng_for(seed, ROLE_OUTLIER)
        pos = r.choice(n, size=k, replace=False)
        flat = x.reshape(-1)
        flat[pos] *= np.float32(factor)
    return x


def lognormal_rows(x, seed, sigma):
    """Scale each row by exp(sigma * z_row), z_row ~ N(0, 1)."""
    r = rng_for(seed, ROLE_ROWSCALE)
    z = r.standard_normal(size=(x.shape[0], 1)).astype(np.float64)
    return (x * np.exp(sigma * z)).astype(np.float32)


# ----------------------------------------------------------- workloads ----
def activation(seed, rows, cols, outlier_fraction=1e-3, outlier_factor=100.0):
    x = normal(seed, ROLE_X, (rows, cols))
    return f32_to_bf16_bits(add_outliers(x, seed, outlier_fraction, outlier_factor))


def weight(seed, rows, cols, std=0.02):
    return f32_to_bf16_bits(normal(seed, ROLE_W, (rows, cols), std))


def gradient(seed, rows, cols, std=1e-5, row_sigma=0.0):
    g = normal(seed, ROLE_DY, (rows, cols), std)
    if row_sigma:
        g = lognormal_rows(g, seed, row_sigma)
    return f32_to_bf16_bits(g)


def linear_fprop_small(seed=0):
    """Single small linear: X [256, 512] N(0,1) with 1% of entries x50,
    W [256, 512] N(0, 0.02)."""
    return {"x": activation(seed, 256, 512, 0.01, 50.0), "w": weight(seed, 256, 512)}


def quantizer_bandwidth(seed=0, rows=8192, cols=4096, wdim=4096):
    """Activation [8192, 4096] N(0,1) with 0.1% x100 outliers; gradient of
    the same shape N(0, 1e-4) with a lognormal per-row scale (sigma 2);
    weight [4096, 4096] N(0, 0.02)."""
    return {"x": activation(seed, rows, cols, 1e-3, 100.0),
            "dy": gradient(seed, rows, cols, 1e-4, 2.0),
            "w": weight(seed, wdim, wdim)}


def ffn_step(seed=0, tokens=8192, k=4096, n=21504):
    """One linear training step Y = X W^T: X [T, K] N(0,1) with 0.1% x100
    outliers, W [N, K] N(0, 0.02), dY [T, N] N(0, 1e-5).  The default sizes
    are the Nemotron-H 8B FFN up-projection (hidden 4096, FFN 21504) on one
    8192-token sequence."""
    return {"x": activation(seed, tokens, k, 1e-3, 100.0),
            "w": weight(seed, n, k),
            "dy": gradient(seed, tokens, n, 1e-5)}


def qkv_formats(seed=0, tokens=16384, k=4096, n=6144):
    """The scale-format comparison workload (a QKV projection): X [T, K]
    N(0,1) with 0.1% x100 outliers, W [N, K] N(0, 0.02), dY [T, N]
    N(0, 1e-4) with a lognormal per-row scale (sigma 2)."""
    return {"x": activation(seed, tokens, k, 1e-3, 100.0),
            "w": weight(seed, n, k),
            "dy": gradient(seed, tokens, n, 1e-4, 2.0)}


def drift_factors(seed=0, steps=120, sigma=0.05, spike_prob=0.05, spike=20.0):
    """Per-step magnitude factors of the X, W and dY operands ([steps, 3]
    float32): a lognormal random walk (log step N(0, sigma)) per operand,
    times ``spike`` on steps drawn with probability ``spike_prob`` (a
    one-step spike).  Used to drive held tensor scales through drift,
    spikes and refreshes."""
    rng = rng_for(seed, ROLE_DRIFT)
    walk = np.exp(np.cumsum(rng.normal(0.0, sigma, (steps, 3)), axis=0))
    spikes = np.where(rng.random((steps, 3)) < spike_prob, spike, 1.0)
    walk[0] = 1.0
    return (walk * spikes).astype(np.float32)


def ffn_down_drift(seed=0, tokens=8192, k=21504, n=4096):
    """Base operands of the FFN down-projection drift workload: X [T, K]
    (the FFN activations) N(0,1) with 0.1% x100 outliers, W [N, K]
    N(0, 0.02), dY [T, N] N(0, 1e-5); each step multiplies them by
    ``drift_factors``."""
    return {"x": activation(seed, tokens, k, 1e-3, 100.0),
            "w": weight(seed, n, k),
            "dy": gradient(seed, tokens, n, 1e-5)}
