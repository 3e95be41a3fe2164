"""GPU parity of the amax and quantizer kernels against the oracle, through
the C ABI.  Payload nibbles, scale bytes and the decode multiplier must be
bit-exact, for RN and for SR with the same Philox counters."""

import numpy as np
import pytest
import torch

import paper_2609_02846_amd as ue
import synthetic
from oracle import quantize as oq
from oracle import scaling as osc
from tests.gpu_util import host, say, set_amax, to_dev

pytestmark = pytest.mark.gpu


def _gpu_amax(xd, period=1):
    st = ue.AmaxState(period=period)
    assert ue.amax_sample(st, xd, 0)
    torch.cuda.synchronize()
    return st, np.float32(st.amax.item())


# ---------------------------------------------------------------- amax ----
@pytest.mark.parametrize("shape", [(1, 1), (3, 5), (7, 9), (256, 512), (1000, 1000), (8192, 4096)])
def test_amax_matches_oracle(shape):
    say("amax", shape)
    bits = synthetic.activation(11, *shape, 1e-3, 100.0)
    _, g = _gpu_amax(to_dev(bits))
    assert g == osc.amax(bits)


def test_amax_empty_and_negative_max():
    say("amax empty / negative")
    st = ue.AmaxState(period=1)
    st.amax.fill_(5.0)
    assert ue.amax_sample(st, torch.empty(0, dtype=torch.bfloat16, device="cuda"), 0)
    torch.cuda.synchronize()
    assert st.amax.item() == 0.0
    x = synthetic.f32_to_bf16_bits(np.array([[0.5, -9.5, 3.0, -0.0]], np.float32))
    _, g = _gpu_amax(to_dev(x))
    assert g == 9.5


def test_amax_planted_maximum_positions():
    """The maximum in the first element, the last element of a grid-stride
    pass past the workgroup cap, the last full vector and the scalar tail;
    the running form (no clear) keeps a larger earlier value."""
    for shape in [(8192, 4104), (3, 1001)]:
        base = synthetic.activation(12, *shape, 0.0, 1.0)
        n = base.size
        for pos in sorted({0, n // 2 + 3, (n // 8) * 8 - 1, n - 1}):
            say("amax planted", shape, pos)
            bits = base.copy().ravel()
            bits[pos] = synthetic.f32_to_bf16_bits(np.array([-123.5], np.float32))[0]
            _, g = _gpu_amax(to_dev(bits.reshape(shape)))
            assert g == np.float32(123.5), (shape, pos)
    say("amax running maximum")
    a = torch.full((1,), 200.0, dtype=torch.float32, device="cuda")
    ue.amax_accumulate(to_dev(base), a, clear=False)
    torch.cuda.synchronize()
    assert a.item() == 200.0
    ue.amax_accumulate(to_dev(base), a, clear=True)
    torch.cuda.synchronize()
    assert np.float32(a.item()) == osc.amax(base)


def test_sample_and_hold_trace_on_gpu():
    """120 steps, D = 50: refreshes at 0, 50, 100 and the held amax is the one
    sampled at the last refresh (eq:delayed-amax)."""
    say("sample-and-hold trace")
    st = ue.AmaxState(period=50)
    ost = osc.AmaxState(period=50)
    refreshed = []
    for t in range(120):
        bits = synthetic.f32_to_bf16_bits(np.full((4, 16), float(t % 7 + 1), np.float32)
                                          * np.float32(1 + t))
        r = ue.amax_sample(st, to_dev(bits), t)
        g_o, r_o = ost.observe(bits, t)
        assert r == r_o
        if r:
            refreshed.append(t)
        torch.cuda.synchronize()
        assert np.float32(st.amax.item()) == g_o
    assert refreshed == [0, 50, 100]
    st.reset()
    assert ue.amax_sample(st, to_dev(bits), 120)


# ------------------------------------------------------------ 1D rows ----
ROW_CASES = [(1, 16), (3, 32), (37, 48), (64, 512), (100, 1040), (256, 512)]


@pytest.mark.parametrize("mode", ["rn", "sr"])
@pytest.mark.parametrize("shape", ROW_CASES)
@pytest.mark.parametrize("target", [448.0, 2048.0])
def test_quantize_rows(shape, mode, target):
    say("rows", shape, mode, target)
    bits = synthetic.gradient(5, *shape, 1e-4, 2.0) if mode == "sr" else \
        synthetic.activation(5, *shape, 0.01, 50.0)
    xd = to_dev(bits)
    st, g = _gpu_amax(xd)
    assert g == osc.amax(bits)
    p, s, d = ue.quantize_1d(xd, 1, st.amax, target, mode, seed=1, tensor_id=7)
    po, so, do = oq.quantize_1d(bits, 1, g, target, mode, 1, 7)
    assert np.array_equal(host(s), so)
    assert np.array_equal(host(p), po)
    assert np.float32(d.item()) == do


# ---------------------------------------------------------- 1D columns ----
COL_CASES = [(16, 2), (16, 4), (48, 38), (64, 100), (256, 512), (512, 300), (80, 1030)]


@pytest.mark.parametrize("mode", ["rn", "sr"])
@pytest.mark.parametrize("shape", COL_CASES)
def test_quantize_cols(shape, mode):
    say("cols", shape, mode)
    bits = synthetic.gradient(6, *shape, 1e-4, 2.0) if mode == "sr" else \
        synthetic.activation(6, *shape, 0.01, 50.0)
    xd = to_dev(bits)
    st, g = _gpu_amax(xd)
    p, s, d = ue.quantize_1d(xd, 0, st.amax, 448.0, mode, seed=3, tensor_id=2)
    po, so, do = oq.quantize_1d(bits, 0, g, 448.0, mode, 3, 2)
    assert np.array_equal(host(s), so)
    assert np.array_equal(host(p), po)
    assert np.float32(d.item()) == do


# ------------------------------------------------------------ 2D tiles ----
TILE_CASES = [(16, 16), (48, 80), (256, 512), (512, 1024), (208, 4096)]


@pytest.mark.parametrize("mode", ["rn", "sr"])
@pytest.mark.parametrize("shape", TILE_CASES)
def test_quantize_tiles(shape, mode):
    say("tiles", shape, mode)
    bits = synthetic.weight(7, *shape)
    xd = to_dev(bits)
    st, g = _gpu_amax(xd)
    p, s, pt, d, stt = ue.quantize_2d(xd, st.amax, 448.0, mode, seed=5, tensor_id=4)
    po, so, pto, do = oq.quantize_2d(bits, g, 448.0, mode, 5, 4)
    assert np.array_equal(host(s), so)
    assert np.array_equal(host(p), po)
    assert np.array_equal(host(pt), pto)
    assert np.array_equal(host(stt), so.T)
    assert np.float32(d.item()) == do
    # without the transposed copy
    p2, s2, pt2, _, st2 = ue.quantize_2d(xd, st.amax, 448.0, mode, seed=5, tensor_id=4,
                                         transposed=False)
    assert pt2 is None and st2 is None and np.array_equal(host(p2), po)


# ---------------------------------------------------- degenerate cases ----
def test_held_reference_saturation_and_underflow():
    """A stale held amax far below / above the tensor maximum drives blocks
    into UE5M3 saturation (Prop. 1) and into the zero-scale rule."""
    say("held reference regimes")
    bits = synthetic.activation(8, 64, 256, 0.01, 50.0)
    xd = to_dev(bits)
    amax = torch.zeros(1, dtype=torch.float32, device="cuda")
    # 1e-25: a tensor multiplier above 2^80, where the SR quantizers take
    # their unscaled conversion form
    for g in [1e-3, 0.05, 1.0, 1e4, 1e9, 0.0, 2.0 ** -100, 1e-25]:
        set_amax(amax, g)
        for axis in [0, 1]:
            for mode in ["rn", "sr"]:
                p, s, d = ue.quantize_1d(xd, axis, amax, 448.0, mode, seed=9, tensor_id=1)
                po, so, do = oq.quantize_1d(bits, axis, np.float32(g), 448.0, mode, 9, 1)
                assert np.array_equal(host(s), so), (g, axis, mode)
                assert np.array_equal(host(p), po), (g, axis, mode)
                assert np.float32(d.item()) == do
        sc = host(s)
        if g == 1e-3:
            assert (sc == 0xF7).any()
        if g == 1e9:
            assert (sc == 0x78).any()


def test_all_zero_and_special_values():
    say("zeros / signed zeros / worked blocks")
    z = np.zeros((32, 64), np.uint16)
    z[1, ::2] = 0x8000                                    # -0
    xd = to_dev(z)
    st, g = _gpu_amax(xd)
    assert g == 0.0
    p, s, d = ue.quantize_1d(xd, 1, st.amax, 448.0, "rn")
    po, so, do = oq.quantize_1d(z, 1, g, 448.0, "rn")
    assert np.array_equal(host(p), po) and np.array_equal(host(s), so)
    assert (so == 0x78).all()


def test_run_twice_bit_identical():
    say("determinism")
    bits = synthetic.gradient(12, 512, 1024, 1e-4, 2.0)
    xd = to_dev(bits)
    st, _ = _gpu_amax(xd)
    a = ue.quantize_1d(xd, 1, st.amax, 448.0, "sr", seed=77, tensor_id=1)
    b = ue.quantize_1d(xd, 1, st.amax, 448.0, "sr", seed=77, tensor_id=1)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


# ------------------------------------------------ full-size workloads ----
def test_quantizer_bandwidth_workload_whole_outputs():
    """8192 x 4096 activation (RN) and gradient (SR, seed 1), both 1D
    blockings, and the 4096 x 4096 weight (2D, with the transposed copy):
    every payload byte and scale code against the oracle."""
    say("quantizer workload 8192x4096")
    wl = synthetic.quantizer_bandwidth(0)
    for name, mode, seed, tid in [("x", "rn", 0, 0), ("dy", "sr", 1, 0)]:
        bits = wl[name]
        xd = to_dev(bits)
        st, g = _gpu_amax(xd)
        assert g == osc.amax(bits)
        for axis in (1, 0):
            say("quantizer workload", name, mode, "axis", axis)
            p, s, d = ue.quantize_1d(xd, axis, st.amax, 448.0, mode, seed, tid)
            po, so, do = oq.quantize_1d(bits, axis, g, 448.0, mode, seed, tid)
            assert np.array_equal(host(s), so), (name, axis)
            assert np.array_equal(host(p), po), (name, axis)
            assert np.float32(d.item()) == do
    say("quantizer workload w tiles")
    wb = wl["w"]
    wd = to_dev(wb)
    st, g = _gpu_amax(wd)
    p, s, pt, d, stt = ue.quantize_2d(wd, st.amax, 448.0, "rn")
    po, so, pto, do = oq.quantize_2d(wb, g, 448.0, "rn")
    assert np.array_equal(host(s), so) and np.array_equal(host(stt), so.T)
    assert np.array_equal(host(p), po) and np.array_equal(host(pt), pto)
    assert np.float32(d.item()) == do


# ------------------------------------------------ every bf16 bit pattern ----
def _all_bf16(rows, cols, seed):
    """Every non-NaN bf16 bit pattern (zeros, subnormals, +-inf included) in
    order of magnitude, shuffled only within runs of 16 so that row blocks
    hold neighbouring magnitudes (block scales then span the whole UE5M3
    range), tiled to [rows, cols]."""
    v = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = v[(v & 0x7FFF) <= 0x7F80]
    v = v[np.argsort(v & 0x7FFF, kind="stable")]
    v = v[: v.size - v.size % 16].reshape(-1, 16)
    v = np.random.default_rng(seed).permuted(v, axis=1).reshape(-1)
    n = rows * cols
    return np.ascontiguousarray(np.tile(v, -(-n // v.size))[:n].reshape(rows, cols))


@pytest.mark.parametrize("g", [1.0, 3.0e4, 2.0 ** -20, 1e-25])
@pytest.mark.parametrize("mode", ["rn", "sr"])
def test_every_bf16_value(g, mode):
    """All quantizers on inputs holding every non-NaN bf16 value, under held
    amax values that put most of them below, inside and above the E2M1 range
    of their blocks: payload and scales bit-exact with the oracle.  With
    g = 1e-25 the tensor multiplier exceeds 2^80 and the SR quantizers use
    their unscaled conversion form; the others use the scaled form."""
    say("every bf16 value", g, mode)
    amax = torch.zeros(1, dtype=torch.float32, device="cuda")
    set_amax(amax, g)
    bits = _all_bf16(256, 512, 21)
    xd = to_dev(bits)
    for axis in [1, 0]:
        p, s, d = ue.quantize_1d(xd, axis, amax, 448.0, mode, seed=11, tensor_id=3)
        po, so, do = oq.quantize_1d(bits, axis, np.float32(g), 448.0, mode, 11, 3)
        assert np.array_equal(host(s), so), axis
        assert np.array_equal(host(p), po), axis
        assert np.float32(d.item()) == do
    p, s, pt, d, st = ue.quantize_2d(xd, amax, 448.0, mode, seed=11, tensor_id=4)
    po, so, pto, do = oq.quantize_2d(bits, np.float32(g), 448.0, mode, 11, 4)
    assert np.array_equal(host(s), so)
    assert np.array_equal(host(p), po)
    assert np.array_equal(host(pt), pto)
    assert np.array_equal(host(st), so.T)
