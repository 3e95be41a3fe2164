"""Teacher-student regression control on the GPU (Sec. "Optimizer-level
regression control", Table tab:grid-regression): the FP4 student (probe-
matched GEMMs in all three products of both layers) trains, is
deterministic run to run, and its final-evaluation error lies above the BF16
control's.  The grid-invariance counts of the table are reported by
``bench.py --control``; here one seed checks the no-snap vs 1/1024 pair."""

import numpy as np
import pytest

from paper_2609_02846_amd import control
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def test_control_trains_deterministically_and_trails_bf16():
    steps = 200
    say("control bf16", steps)
    bf = control.run(42, "bf16", steps=steps)
    say("control fp4 rn grid 1024")
    a = control.run(42, "fp4", "rn", grid=1024, steps=steps)
    say("control fp4 rn grid 1024 again")
    b = control.run(42, "fp4", "rn", grid=1024, steps=steps)
    assert control.same_trajectory(a, b) == (True, True)
    for r in (bf, a):
        assert np.all(np.isfinite(r["losses"]))
        assert r["losses"][-20:].mean() < 0.2 * r["losses"][:5].mean()
    assert bf["eval_mse"] < a["eval_mse"]
    say("control fp4 sr grid 0")
    s = control.run(42, "fp4", "sr", grid=0, steps=steps)
    assert s["losses"][-20:].mean() < 0.2 * s["losses"][:5].mean()
    print("eval mse bf16 %.6f fp4-rn-1024 %.6f fp4-sr-0 %.6f" % (bf["eval_mse"], a["eval_mse"], s["eval_mse"]))


def _pm_check(got_bf16, A, B, al, idx, what, d=1024):
    """Sampled outputs (m, n) of a bf16 probe-matched product against the
    oracle's model (oracle.accumulate: 64-product RNE partials, toward-zero
    group adds, 1/d snap, alpha), rounded to bf16: bit for bit."""
    import torch
    from oracle import accumulate as oacc
    ref = np.array([oacc.dot(A[m] * B[n], d, al)[0] for m, n in idx], np.float32)
    ref = torch.from_numpy(ref).to(torch.bfloat16).float().numpy()
    got = np.array([got_bf16[m, n] for m, n in idx], np.float32)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, f"{what}: {bad.size}/{len(idx)} differ, first {idx[bad[0]]}: {got[bad[0]]} vs {ref[bad[0]]}"


def _idx(M, N, seed, n=96):
    rng = np.random.default_rng(seed)
    idx = {(0, 0), (M - 1, N - 1), (0, N - 1), (M - 1, 0)}
    idx |= {(int(rng.integers(M)), int(rng.integers(N))) for _ in range(n)}
    return sorted(idx)


@pytest.mark.parametrize("rounding", ["rn", "sr"])
def test_control_first_step_matches_oracle(rounding):
    """The first training step of the control's FP4 student (seed 42, grid
    1/1024): both layers' outputs Y, input gradients dX and weight gradients
    dW equal the oracle's probe-matched model on sampled outputs, bit for bit
    (eq:issue-partial, eq:issue-rz, eq:final-grid), with operands the
    oracle quantizes from the same bits (references: each operand's current
    amax, the first sample-and-hold refresh; dY by RN or SR with each layer's
    Philox key and tensor ids)."""
    import torch
    from oracle import gemm as ogemm
    from oracle import quantize as oq
    from oracle import scaling as osc
    from paper_2609_02846_amd.linear import Linear
    from tests.gpu_util import host
    seed = 42
    say("control first step vs oracle", rounding)
    d = control._data(seed, "cuda")
    layers = [Linear(control.D_IN, control.D_HID, period=50, target=448.0, seed=1000 * seed + 1, layer_id=0,
                     device="cuda", grad_rounding=rounding, pm_grid=1024),
              Linear(control.D_HID, control.D_OUT, period=50, target=448.0, seed=1000 * seed + 2, layer_id=1,
                     device="cuda", grad_rounding=rounding, pm_grid=1024)]
    with torch.no_grad():
        for l, w in zip(layers, d["init"]):
            l.weight.copy_(w.to("cuda"))
    idx = d["order"][0].to("cuda")
    x = d["x_tr"][idx].clone().requires_grad_(True)
    for l in layers:
        l.step = 0
    y1 = layers[0](x)
    y1.retain_grad()
    y2 = layers[1](y1)
    y2.retain_grad()
    loss = torch.mean((y2.float() - d["y_tr"][idx]) ** 2)
    loss.backward()
    torch.cuda.synchronize()
    bits = lambda t: host(t.detach().contiguous().view(torch.int16)).view(np.uint16)
    hx, hy1, hdy2, hdy1 = bits(x), bits(y1), bits(y2.grad), bits(y1.grad)
    hw = [bits(l.weight) for l in layers]
    outs = {"y": [host(y1.float()), host(y2.float())], "dx": [host(x.grad.float()), host(y1.grad.float())],
            "dw": [host(l.weight.grad.float()) for l in layers]}
    ins = [hx, hy1]
    dys = [hdy1, hdy2]
    for li in range(2):
        xin, w, dy = ins[li], hw[li], dys[li]
        T, K = xin.shape
        N = w.shape[0]
        gx, gw, gd = osc.amax(xin), osc.amax(w), osc.amax(dy)
        xr, xc = oq.quantize_1d(xin, 1, gx), oq.quantize_1d(xin, 0, gx)
        wq = oq.quantize_2d(w, gw)
        key = 1000 * seed + 1 + li                            # first backward call: no offset
        dr = oq.quantize_1d(dy, 1, gd, 448.0, rounding, key, 2 * li + 1)
        dc = oq.quantize_1d(dy, 0, gd, 448.0, rounding, key, 2 * li + 2)
        X, W = oq.decoded_1d(xr[0], xr[1], 1), oq.decoded_2d(wq[0], wq[1])
        _pm_check(outs["y"][li], X, W, ogemm.alpha(xr[2], wq[3]), _idx(T, N, 1 + li), f"layer {li} Y")
        dY = oq.decoded_1d(dr[0], dr[1], 1)                   # [T, N]
        _pm_check(outs["dx"][li], dY, np.ascontiguousarray(W.T), ogemm.alpha(dr[2], wq[3]), _idx(T, K, 3 + li),
                  f"layer {li} dX")
        dYc = oq.decoded_1d(dc[0], dc[1], 0)                  # [T, N]
        Xc = oq.decoded_1d(xc[0], xc[1], 0)                   # [T, K]
        _pm_check(outs["dw"][li], np.ascontiguousarray(dYc.T), np.ascontiguousarray(Xc.T),
                  ogemm.alpha(dc[2], xc[2]), _idx(N, K, 5 + li), f"layer {li} dW")
