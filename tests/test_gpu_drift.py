"""FFN down-projection (T = 8192, K = 21504, N = 4096) over 120 optimizer
steps with the 50-step sample-and-hold reference (eq:delayed-amax) while the
operand magnitudes drift (lognormal walk, sigma 0.05 per step) and spike
(x20 on random steps): every step checks the refresh decisions and held
references of X, W and dY against the oracle's trace; at the refresh steps,
the spike steps between refreshes, the planted steps and the last step,
sampled rows of the quantized operands are bit-exact and sampled GEMM
outputs meet the GEMM bar.

Planted rows make the held reference's edge cases certain rather than
likely: one X row is zero on every step (all-zero blocks: the zero rule),
and on the planted steps (never refresh steps, so the held references do
not see them) one X row is scaled to 300 held references (its block scales
saturate, Proposition 1) and one dY row by 1e-10 (its blocks underflow to
code 0 and take the zero rule).  Those steps log the numbers of saturated,
underflowed and all-zero blocks in the sampled rows and require each to be
positive.

The operand of step t is bf16(base * f_t) (binary32 product, RNE), formed on
the device; the oracle forms the same bits for the rows it samples.  The
tensor amax of bf16(base * f) is bf16(max|base| * f) because both roundings
are monotone, which gives the oracle its references without materialising
each step's tensors on the host."""

import numpy as np
import pytest
import torch

import synthetic
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc
import paper_2609_02846_amd as ue
from tests.gpu_util import gemm_check, host, row_elem_index, say, to_dev

pytestmark = pytest.mark.gpu

STEPS, PERIOD = 120, 50
PLANTED = (10, 60, 119)
ZERO_ROW, SAT_ROW, UF_ROW = 5, 11, 13


def _scaled_bits(bits, f):
    return synthetic.f32_to_bf16_bits(synthetic.bf16_bits_to_f32(bits) * np.float32(f))


def _amax_scaled(base_max, f):
    return osc.amax(synthetic.f32_to_bf16_bits(np.array([[base_max * np.float32(f)]], np.float32)))


def _bf16_row_scaled(bits, factor):
    return synthetic.f32_to_bf16_bits(synthetic.bf16_bits_to_f32(bits) * np.float32(factor))


def _plant_x(bits, row_ids, t, sat_factor):
    """The planted X rows among ``row_ids`` (host copy of the device edit)."""
    out = bits.copy()
    for i, r in enumerate(row_ids):
        if r == ZERO_ROW:
            out[i] = 0
        elif r == SAT_ROW and t in PLANTED:
            out[i] = _bf16_row_scaled(out[i], sat_factor)
    return out


def _plant_dy(bits, row_ids, t):
    out = bits.copy()
    for i, r in enumerate(row_ids):
        if r == UF_ROW and t in PLANTED:
            out[i] = _bf16_row_scaled(out[i], 1e-10)
    return out


def test_down_projection_drift_120_steps():
    T, K, N = 8192, 21504, 4096
    say("down-projection drift", T, K, N, STEPS, "steps")
    wl = synthetic.ffn_down_drift(0, T, K, N)
    x0b, w0b, d0b = wl["x"], wl["w"], wl["dy"]
    fac = synthetic.drift_factors(0, STEPS)
    bmax = [np.float32(np.max(np.abs(synthetic.bf16_bits_to_f32(b)))) for b in (x0b, w0b, d0b)]
    # the zero row must not hold the tensor maximum (the references stay those of the bases)
    assert np.argmax(np.max(np.abs(synthetic.bf16_bits_to_f32(x0b)), axis=1)) != ZERO_ROW
    x0, w0, d0 = (to_dev(b).float() for b in (x0b, w0b, d0b))
    states = [ue.AmaxState(PERIOD) for _ in range(3)]
    ost = [osc.AmaxState(PERIOD) for _ in range(3)]
    spikes = {int(t) for t, j in np.argwhere(fac > 5.0)}
    refresh_steps = set(range(0, STEPS, PERIOD))
    assert not refresh_steps & set(PLANTED)
    checks = sorted((refresh_steps | {t for t in spikes if t % PERIOD}) | {STEPS - 1} | set(PLANTED))
    rng = np.random.default_rng(3)
    rows = np.sort(np.concatenate([[0, ZERO_ROW, SAT_ROW, UF_ROW, T - 1], rng.choice(np.arange(16, T - 1), 4,
                                                                                      replace=False)]))
    rdev = torch.from_numpy(rows).cuda()
    sat = 0
    for t in range(STEPS):
        f = fac[t]
        xt = (x0 * float(f[0])).to(torch.bfloat16)
        wt = (w0 * float(f[1])).to(torch.bfloat16)
        dt = (d0 * float(f[2])).to(torch.bfloat16)
        xt[ZERO_ROW] = 0
        sat_factor = None
        if t in PLANTED:
            # 300 held references over the row's maximum: u_B = 300 T > 61440 for its largest block
            arow = np.max(np.abs(synthetic.bf16_bits_to_f32(_scaled_bits(x0b[SAT_ROW], f[0]))))
            sat_factor = np.float32(300.0) * ost[0].g / arow
            xt[SAT_ROW] = (xt[SAT_ROW].float() * float(sat_factor)).to(torch.bfloat16)
            dt[UF_ROW] = (dt[UF_ROW].float() * float(np.float32(1e-10))).to(torch.bfloat16)
        for j, (st, tens) in enumerate(zip(states, (xt, wt, dt))):
            r = ue.amax_sample(st, tens, t)
            g_o, r_o = ost[j].observe_amax(lambda: _amax_scaled(bmax[j], f[j]), t)
            assert r == r_o, (t, j)
        torch.cuda.synchronize()
        for j in range(3):
            assert np.float32(states[j].amax.item()) == ost[j].g, (t, j)
        if t not in checks:
            continue
        say("drift check step", t, "factors", f.tolist())
        gx, gw, gd = (ost[j].g for j in range(3))
        xr = ue.quantize_1d(xt, 1, states[0].amax)
        xc = ue.quantize_1d(xt, 0, states[0].amax)
        wq = ue.quantize_2d(wt, states[1].amax)
        dr = ue.quantize_1d(dt, 1, states[2].amax, 448.0, "sr", 500 + t, 1)
        dc = ue.quantize_1d(dt, 0, states[2].amax, 448.0, "sr", 500 + t, 2)
        y = ue.gemm("nt", T, N, K, *xr, wq[0], wq[1], wq[3], out_dtype=torch.bfloat16)
        dx = ue.gemm("nn", T, K, N, *dr, wq[2], wq[4], wq[3], out_dtype=torch.bfloat16)
        dw = ue.gemm("tn", N, K, T, *dc, xc[0], xc[1], xc[2])
        torch.cuda.synchronize()
        # quantized rows of X and dY, bit-exact
        xs = _plant_x(_scaled_bits(x0b[rows], f[0]), rows, t, sat_factor)
        ds = _plant_dy(_scaled_bits(d0b[rows], f[2]), rows, t)
        xo = oq.quantize_1d(xs, 1, gx)
        do = oq.quantize_1d(ds, 1, gd, 448.0, "sr", 500 + t, 1, elem_index=row_elem_index(rows, N))
        assert np.array_equal(host(xr[0][rdev]), xo[0]) and np.array_equal(host(xr[1][rdev]), xo[1]), t
        assert np.array_equal(host(dr[0][rdev]), do[0]) and np.array_equal(host(dr[1][rdev]), do[1]), t
        sat += int(np.sum(xo[1] == 0xF7)) + int(np.sum(do[1] == 0xF7))
        zero_blocks = int(np.sum(np.max(np.abs(synthetic.bf16_bits_to_f32(xs)).reshape(len(rows), -1, 16),
                                        axis=2) == 0))
        assert zero_blocks >= K // 16 and np.all(xo[1][rows == ZERO_ROW] == 0x78), t
        if t in PLANTED:
            n_sat = int(np.sum(xo[1][rows == SAT_ROW] == 0xF7))
            # every block of the scaled dY row has u_B below half the smallest UE5M3 step
            uf = np.max(np.abs(synthetic.bf16_bits_to_f32(ds[rows == UF_ROW]))) * np.float32(448.0) / gd
            n_uf = int(np.sum(do[1][rows == UF_ROW] == 0x78))
            print(f"step {t}: saturated blocks {n_sat}, underflowed blocks {n_uf}, all-zero blocks "
                  f"{zero_blocks} (sampled rows)")
            assert n_sat > 0 and uf < 2.0 ** -18 and n_uf == N // 16, (t, n_sat, uf, n_uf)
        # fprop: sampled rows x one weight tile row (16 outputs each)
        wt16 = _scaled_bits(w0b[16 * 7:16 * 8], f[1])
        wo = oq.quantize_2d(wt16, gw)
        X, W = oq.decoded_1d(xo[0], xo[1], 1), oq.decoded_2d(wo[0], wo[1])
        al = ogemm.alpha(xo[2], wo[3])
        ref = ogemm.fprop(X, W, al)
        c16 = host(y[rdev][:, 16 * 7:16 * 8].float()).astype(np.float64)
        e = float(al) * K * 2.0 ** -23 * ogemm.abs_product(X, W)
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref) + e, 1e-30))) - 7)
        assert np.all(np.abs(c16 - ref) <= e + 1.01 * ulp + 1e-30), ("fprop", t)
        # dgrad: sampled rows x one 16-column weight tile column (all of N)
        wcol = _scaled_bits(np.ascontiguousarray(w0b[:, 16 * 3:16 * 4]), f[1])
        wco = oq.quantize_2d(wcol, gw)
        dY = oq.decoded_1d(do[0], do[1], 1)
        Wc = oq.decoded_2d(wco[0], wco[1])
        al = ogemm.alpha(do[2], wco[3])
        ref = ogemm.dgrad(dY, Wc, al)
        c16 = host(dx[rdev][:, 16 * 3:16 * 4].float()).astype(np.float64)
        e = float(al) * N * 2.0 ** -23 * ogemm.abs_product(dY, np.ascontiguousarray(Wc.T))
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref) + e, 1e-30))) - 7)
        assert np.all(np.abs(c16 - ref) <= e + 1.01 * ulp + 1e-30), ("dgrad", t)
        # wgrad: two dY columns x three X columns (all T rows, planted rows included)
        nc, kc = np.array([5, N - 1]), np.array([0, 999, K - 1])
        allr = np.arange(T)
        dsub = _plant_dy(_scaled_bits(np.ascontiguousarray(d0b[:, nc]), f[2]), allr, t)
        xsub = _plant_x(_scaled_bits(np.ascontiguousarray(x0b[:, kc]), f[0]), allr, t, sat_factor)
        dco = oq.quantize_1d(dsub, 0, gd, 448.0, "sr", 500 + t, 2,
                             elem_index=row_elem_index(np.arange(T), N, nc))
        xco = oq.quantize_1d(xsub, 0, gx)
        A = oq.decoded_1d(dco[0], dco[1], 0).T
        B = oq.decoded_1d(xco[0], xco[1], 0).T
        al = ogemm.alpha(dco[2], xco[2])
        ref = ogemm.fprop(A, B, al)
        got = host(dw)[np.ix_(nc, kc)]
        gemm_check(got, ref, al, ogemm.abs_product(A, B), T, f"wgrad step {t}")
    print("saturated block codes seen in the sampled rows:", sat)



FULL_STEPS = (0, 10, 50, 60, 100, 119)       # refresh steps and planted steps


@pytest.fixture(scope="module")
def drift_bases():
    T, K, N = 8192, 21504, 4096
    wl = synthetic.ffn_down_drift(0, T, K, N)
    return (T, K, N), wl, synthetic.drift_factors(0, STEPS)


def _held_references(bmax, fac, t):
    """The oracle's held references of X, W and dY at step t
    (eq:delayed-amax over steps 0..t)."""
    ost = [osc.AmaxState(PERIOD) for _ in range(3)]
    for s in range(t + 1):
        for j in range(3):
            ost[j].observe_amax(lambda: _amax_scaled(bmax[j], fac[s][j]), s)
    return [o.g for o in ost]


@pytest.mark.parametrize("t", FULL_STEPS)
def test_drift_whole_quantizer_outputs(drift_bases, t):
    """At the refresh steps (0, 50, 100) and the planted steps (10, 60, 119)
    of the drift run: every payload byte and scale code of X (both 1D
    blockings from one read, as the step runs them), W (tiles, the transposed
    copy and its scales) and dY (rows and columns, SR) against the oracle,
    with the references the sample-and-hold rule holds at that step
    (eq:delayed-amax; Proposition 1 and the zero-scale rule decide the
    planted rows).  The step's operands are formed on the device as in the
    drift run and must equal the host's bits."""
    (T, K, N), wl, fac = drift_bases
    x0b, w0b, d0b = wl["x"], wl["w"], wl["dy"]
    f = fac[t]
    bmax = [np.float32(np.max(np.abs(synthetic.bf16_bits_to_f32(b)))) for b in (x0b, w0b, d0b)]
    gx, gw, gd = _held_references(bmax, fac, t)
    say("drift whole outputs, step", t, "references", gx, gw, gd)
    # host bits of the step's operands, planted rows included
    xs = _scaled_bits(x0b, f[0])
    xs[ZERO_ROW] = 0
    ws = _scaled_bits(w0b, f[1])
    ds = _scaled_bits(d0b, f[2])
    sat_factor = None
    if t in PLANTED:
        arow = np.max(np.abs(synthetic.bf16_bits_to_f32(xs[SAT_ROW])))
        sat_factor = np.float32(300.0) * gx / arow
        xs[SAT_ROW] = _bf16_row_scaled(xs[SAT_ROW], sat_factor)
        ds[UF_ROW] = _bf16_row_scaled(ds[UF_ROW], 1e-10)
    # the same operands formed on the device
    xt = (to_dev(x0b).float() * float(f[0])).to(torch.bfloat16)
    wt = (to_dev(w0b).float() * float(f[1])).to(torch.bfloat16)
    dt = (to_dev(d0b).float() * float(f[2])).to(torch.bfloat16)
    xt[ZERO_ROW] = 0
    if t in PLANTED:
        xt[SAT_ROW] = (xt[SAT_ROW].float() * float(sat_factor)).to(torch.bfloat16)
        dt[UF_ROW] = (dt[UF_ROW].float() * float(np.float32(1e-10))).to(torch.bfloat16)
    for dev, hst, name in ((xt, xs, "X"), (wt, ws, "W"), (dt, ds, "dY")):
        assert np.array_equal(host(dev.view(torch.int16)).view(np.uint16), hst), (t, name)
    ax, aw, ad = (torch.tensor([float(g)], dtype=torch.float32, device="cuda") for g in (gx, gw, gd))
    xr, xc = ue.quantize_dual(xt, ax)
    wq = ue.quantize_2d(wt, aw)
    dr = ue.quantize_1d(dt, 1, ad, 448.0, "sr", 500 + t, 1)
    dc = ue.quantize_1d(dt, 0, ad, 448.0, "sr", 500 + t, 2)
    torch.cuda.synchronize()
    del xt, wt, dt

    say("drift whole outputs: X rows and columns, step", t)
    xro = oq.quantize_1d(xs, 1, gx)
    assert np.array_equal(host(xr[1]), xro[1]) and np.array_equal(host(xr[0]), xro[0]), t
    assert np.float32(xr[2].item()) == xro[2], t
    n_sat = int(np.sum(xro[1] == 0xF7))
    n_zero = int(np.sum(np.max(np.abs(synthetic.bf16_bits_to_f32(xs)).reshape(T, -1, 16), axis=2) == 0))
    assert n_zero >= K // 16 and np.all(xro[1][ZERO_ROW] == 0x78), t
    del xro
    xco = oq.quantize_1d(xs, 0, gx)
    assert np.array_equal(host(xc[1]), xco[1]) and np.array_equal(host(xc[0]), xco[0]), t
    del xco, xs

    say("drift whole outputs: W tiles and the transposed copy, step", t)
    wo = oq.quantize_2d(ws, gw)
    assert np.array_equal(host(wq[1]), wo[1]) and np.array_equal(host(wq[4]), wo[1].T), t
    assert np.array_equal(host(wq[0]), wo[0]) and np.array_equal(host(wq[2]), wo[2]), t
    assert np.float32(wq[3].item()) == wo[3], t
    del wo, ws

    say("drift whole outputs: dY rows and columns (SR), step", t)
    dro = oq.quantize_1d(ds, 1, gd, 448.0, "sr", 500 + t, 1)
    assert np.array_equal(host(dr[1]), dro[1]) and np.array_equal(host(dr[0]), dro[0]), t
    n_uf = int(np.sum(dro[1][UF_ROW] == 0x78))
    dco = oq.quantize_1d(ds, 0, gd, 448.0, "sr", 500 + t, 2)
    assert np.array_equal(host(dc[1]), dco[1]) and np.array_equal(host(dc[0]), dco[0]), t
    print(f"step {t}: saturated X blocks {n_sat}, underflowed dY-row blocks {n_uf}, all-zero X blocks {n_zero}")
    if t in PLANTED:
        # the planted rows: saturation (Proposition 1) and the zero-scale rule
        assert n_sat > 0 and n_uf == N // 16, (t, n_sat, n_uf)
