"""Pins of the oracle's tensor-scale logic: amax (Sec. 4.1), sample-and-hold
(eq:delayed-amax), tensor multipliers and the Table 3 worked example,
Proposition 1 (eq:effective-range)."""

import os

import numpy as np
import pytest

import synthetic
from oracle import formats, quantize, scaling


def _pv(golden_dir):
    vals = {}
    for line in open(os.path.join(golden_dir, "paper_values.txt")):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()[:2]
            vals[k] = float(v)
    return vals


def _bits(vals):
    return synthetic.f32_to_bf16_bits(np.asarray(vals, np.float32))


def test_amax_exact():
    x = _bits([[0.5, -7.25, 3.0], [-0.0, 7.0, -1e-3]])
    assert scaling.amax(x) == np.float32(7.25)
    assert scaling.amax(np.zeros((0, 4), np.uint16)) == 0.0
    big = synthetic.activation(3, 64, 128)
    ref = max(abs(float(v)) for v in synthetic.bf16_bits_to_f32(big).ravel())
    assert scaling.amax(big) == np.float32(ref)


def test_sample_and_hold_trace(golden_dir):
    D = int(_pv(golden_dir)["refresh_period"])
    st = scaling.AmaxState(period=D)
    refreshed = []
    for t in range(120):
        x = _bits([[float(t + 1)]])              # amax at step t is t + 1
        g, r = st.observe(x, t)
        if r:
            refreshed.append(t)
        # held value is the amax of the most recent refresh step
        assert g == np.float32(max(s for s in refreshed) + 1)
    assert refreshed == [0, 50, 100]


def test_sample_and_hold_irregular_steps_reset_and_current():
    st = scaling.AmaxState(period=50)
    obs = [(0, 1.0), (30, 2.0), (49, 3.0), (50, 4.0), (99, 5.0), (120, 6.0), (169, 6.5), (170, 7.0)]
    got = [st.observe(_bits([[v]]), t) for t, v in obs]
    assert [bool(r) for _, r in got] == [True, False, False, True, False, True, False, True]
    assert [float(g) for g, _ in got] == [1.0, 1.0, 1.0, 4.0, 4.0, 6.0, 6.0, 7.0]
    st.reset()                                   # resume: cache not restored
    g, r = st.observe(_bits([[9.0]]), 171)
    assert r and g == 9.0
    cur = scaling.AmaxState(period=1)            # D = 1 is current scaling
    assert all(cur.observe(_bits([[float(t)]]), t)[1] for t in range(5))
    with pytest.raises(ValueError):
        scaling.AmaxState(period=-1)


def test_inference_policies():
    """Inference-scale policies (Table tab:inference-scale-summary): a held
    weight reference is measured on the first batch only, even across a
    huge step gap; a calibrated reference is the largest calibration amax
    and never refreshes; reset empties a held cache."""
    held = scaling.AmaxState(period=0)
    got = [held.observe(_bits([[float(v)]]), t) for t, v in [(0, 3.0), (1, 9.0), (10**12, 20.0)]]
    assert [(float(g), r) for g, r in got] == [(3.0, True), (3.0, False), (3.0, False)]
    held.reset()
    assert held.observe(_bits([[5.0]]), 10**12 + 1) == (5.0, True)
    cal = [_bits([[1.0, -4.5]]), _bits([[-7.0, 2.0]]), _bits([[6.0]])]
    assert scaling.calibrated_amax(cal) == np.float32(7.0)
    assert scaling.calibrated_amax([]) == 0.0
    st = scaling.AmaxState(period=50)
    st.observe(_bits([[100.0]]), 0)
    st.freeze(scaling.calibrated_amax(cal))
    assert all(st.observe(_bits([[1e3]]), t) == (7.0, False) for t in (0, 50, 500))


def test_multipliers_table3_example(golden_dir):
    pv = _pv(golden_dir)
    g = np.float32(pv["table3_g"])
    for T, code_key, mn, mx, room in [(448.0, "table3_code_T448", "table3_min_T448",
                                       "table3_max_T448", "table3_room_T448"),
                                      (2048.0, "table3_code_T2048", "table3_min_T2048",
                                       "table3_max_T2048", "table3_room_T2048")]:
        S, G, dec = scaling.tensor_multipliers(g, T)
        # a block as large as the held maximum lands on code T
        u = np.float32(g * S)
        c = formats.ue5m3_encode_rne_sat(u)
        assert formats.ue5m3_decode(c) == pv[code_key]
        # smallest nonzero block maximum: the one landing on 2**-17
        a_min = formats.ue5m3_decode(1) * float(g) / T
        assert float(f"{a_min:.1e}") == pv[mn]
        c_min = formats.ue5m3_encode_rne_sat(np.float32(np.float32(a_min) * S))
        assert c_min == 0x01
        # largest unsaturated block maximum: the one landing on 61440
        a_max = formats.UE5M3_MAX * float(g) / T
        assert int(a_max) == pv[mx]
        assert formats.ue5m3_encode_rne_sat(np.float32(np.float32(a_max) * S)) == 0xF7
        assert int(formats.UE5M3_MAX / T) == pv[room]
        assert G == np.float32(np.float32(T * 6) / g)
        assert dec == np.float32(g / np.float32(T * 6))


def test_multipliers_degenerate_reference():
    ref = scaling.tensor_multipliers(1.0, 448.0)
    for g in [0.0, -1.0, np.inf, np.nan, 1e-38]:
        assert scaling.tensor_multipliers(g, 448.0) == ref
    S, G, dec = scaling.tensor_multipliers(2.0 ** -90, 448.0)
    assert G < 2.0 ** 110 and np.isfinite(S)


def test_proposition1_saturation_boundary():
    """A block saturates (code 0xF7 with u_B above U) exactly when
    a_B > U g / T (eq:effective-range); checked away from the binary32
    rounding band around the boundary."""
    rng = np.random.default_rng(5)
    n = 20000
    g = np.exp(rng.uniform(np.log(1e-3), np.log(1e4), n)).astype(np.float32)
    T = rng.choice(np.array([448.0, 2048.0, 1000.0, 96.0], np.float32), n)
    ratio = np.exp(rng.uniform(np.log(1e-2), np.log(1e4), n))
    a = (ratio * g).astype(np.float32)
    bound = formats.UE5M3_MAX * g.astype(np.float64) / T
    far = np.abs(a / bound - 1.0) > 1e-5
    for i in np.nonzero(far)[0][:4000]:
        S, G, _ = scaling.tensor_multipliers(g[i], T[i])
        u = np.float32(a[i] * S)
        sat = bool(u > formats.UE5M3_MAX)
        assert sat == bool(a[i] > bound[i])
        if sat:
            assert formats.ue5m3_encode_rne_sat(u) == 0xF7


def test_stale_headroom_all_blocks_unsaturated():
    """eq:stale-headroom: if T * rho <= U (rho = current amax / held g), no
    block scale is clipped: every block's largest element maps to at most
    6 (1 + 2**-4) (the UE5M3 relative rounding), while T * rho = 2U clips."""
    rng = np.random.default_rng(9)
    x = rng.standard_normal((64, 256)).astype(np.float32)
    bits = synthetic.f32_to_bf16_bits(x)
    xf = synthetic.bf16_bits_to_f32(bits).astype(np.float64)
    a_t = float(scaling.amax(bits))
    a_B = np.abs(xf).reshape(64, 16, 16).max(axis=2)
    for T in [448.0, 2048.0]:
        for rho_T, clipped in [(0.999, False), (2.0, True)]:
            g = np.float32(a_t * T / (rho_T * formats.UE5M3_MAX))
            _, sc, _ = quantize.quantize_1d(bits, 1, g, T)
            _, G, _ = scaling.tensor_multipliers(g, T)
            y_max = a_B * float(G) / formats.ue5m3_decode(sc)
            if clipped:
                assert y_max.max() > 11.0
            else:
                assert y_max.max() <= 6.0 * (1 + 2.0 ** -4) * (1 + 1e-6)
