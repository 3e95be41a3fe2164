"""GPU parity of the FP4 Linear layer (autograd wrapper over the C ABI)
against the oracle's quantize-then-GEMM: forward Y, dX and dW of a training
step, sample-and-hold across optimizer steps (eq:delayed-amax), the SR key
schedule, and the inference-scale policies (Table
tab:inference-scale-summary).  Outputs are bf16; the bar is one bf16 ulp of
the exact product plus the fp32 accumulation bound."""

import numpy as np
import pytest
import torch

import synthetic
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc
from paper_2609_02846_amd.linear import Linear
from tests.gpu_util import host, say, to_dev

pytestmark = pytest.mark.gpu


def bf16_check(c, ref, al, absprod, K, what):
    """|C - C_ref| <= e + ulp_bf16(|C_ref| + e), e = the fp32 accumulation
    bound alpha K 2^-23 sum|A||B| (rounding the fp32 result to bf16 adds at
    most half an ulp of the value it rounds)."""
    c = np.asarray(host(c.float()), np.float64)
    e = float(al) * max(K, 1) * 2.0 ** -23 * absprod
    mag = np.abs(ref) + e
    ulp = np.exp2(np.floor(np.log2(np.maximum(mag, 1e-30))) - 7)
    bound = e + ulp * 1.01 + 1e-30
    err = np.abs(c - ref)
    assert np.all(err <= bound), f"{what}: {int((err > bound).sum())} elements out, worst {np.max(err / bound):.3g}"


def _inputs(seed, T, K, N):
    x = synthetic.activation(seed, T, K, 1e-2, 50.0)
    w = synthetic.weight(seed, N, K)
    dy = synthetic.gradient(seed, T, N, 1e-3, 1.0)
    return x, w, dy


def _scaled(bits, f):
    return synthetic.f32_to_bf16_bits(synthetic.bf16_bits_to_f32(bits) * np.float32(f))


def _ref_y(x, w, gx, gw, block=16):
    xr = oq.quantize_1d(x, 1, gx, block=block)
    wq = oq.quantize_2d(w, gw, tile=block)
    X, W = oq.decoded_1d(xr[0], xr[1], 1, block=block), oq.decoded_2d(wq[0], wq[1], tile=block)
    al = ogemm.alpha(xr[2], wq[3])
    return ogemm.fprop(X, W, al), ogemm.abs_product(X, W), al


def _ref_grads(x, w, dy, gx, gw, gd, seed, layer_id, block=16):
    xc = oq.quantize_1d(x, 0, gx, block=block)
    wq = oq.quantize_2d(w, gw, tile=block)
    dr = oq.quantize_1d(dy, 1, gd, 448.0, "sr", seed, 2 * layer_id + 1, block=block)
    dc = oq.quantize_1d(dy, 0, gd, 448.0, "sr", seed, 2 * layer_id + 2, block=block)
    W = oq.decoded_2d(wq[0], wq[1], tile=block)
    dY = oq.decoded_1d(dr[0], dr[1], 1, block=block)
    dYc = oq.decoded_1d(dc[0], dc[1], 0, block=block)
    Xc = oq.decoded_1d(xc[0], xc[1], 0, block=block)
    al_d, al_w = ogemm.alpha(dr[2], wq[3]), ogemm.alpha(dc[2], xc[2])
    return ((ogemm.dgrad(dY, W, al_d), ogemm.abs_product(dY, W.T), al_d),
            (ogemm.wgrad(dYc, Xc, al_w), ogemm.abs_product(dYc.T, Xc.T), al_w))


def _layer(K, N, w, **kw):
    layer = Linear(K, N, **kw)
    with torch.no_grad():
        layer.weight.copy_(to_dev(w))
    return layer


def test_training_step_matches_oracle():
    """One training step on several GEMM tiles with ragged tails: Y, dX and
    dW equal the oracle's products of exactly quantized operands (X, W RN;
    dY SR with the layer's Philox key and tensor ids); a second backward
    draws new SR words (key seed + 1)."""
    T, K, N = 528, 400, 272
    say("linear training step", T, K, N)
    x, w, dy = _inputs(11, T, K, N)
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    layer = _layer(K, N, w, period=50, seed=5, layer_id=3)
    yref, yabs, yal = _ref_y(x, w, gx, gw)
    grads = []
    for call in range(2):
        xd = to_dev(x).requires_grad_(True)
        layer.weight.grad = None
        y = layer(xd)
        y.backward(to_dev(dy))
        torch.cuda.synchronize()
        bf16_check(y, yref, yal, yabs, K, f"fprop call {call}")
        (dxr, dxa, dxl), (dwr, dwa, dwl) = _ref_grads(x, w, dy, gx, gw, gd, 5 + call, 3)
        bf16_check(xd.grad, dxr, dxl, dxa, N, f"dgrad call {call}")
        bf16_check(layer.weight.grad, dwr, dwl, dwa, T, f"wgrad call {call}")
        assert xd.grad.dtype == torch.bfloat16 and layer.weight.grad.dtype == torch.bfloat16
        grads.append((host(xd.grad.float()), host(layer.weight.grad.float())))
    assert layer.sr_calls == 2
    assert not np.array_equal(grads[0][0], grads[1][0])      # fresh SR words per call
    for st, g in [(layer.amax_x, gx), (layer.amax_w, gw), (layer.amax_dy, gd)]:
        assert np.float32(st.amax.item()) == g and st.last_refresh == 0


def test_batched_input_shape_and_inference_ragged_tokens():
    """[B, S, K] inputs keep their leading dimensions; without gradients
    the token count need not be a multiple of 16."""
    K, N = 64, 48
    x, w, _ = _inputs(2, 40, K, N)
    say("linear shapes", x.shape)
    layer = _layer(K, N, w, period=1)
    xd = to_dev(x).reshape(2, 20, K)
    with torch.no_grad():
        y = layer(xd)
    assert y.shape == (2, 20, N)
    yref, yabs, yal = _ref_y(x, w, osc.amax(x), osc.amax(w))
    bf16_check(y.reshape(40, N), yref, yal, yabs, K, "batched fprop")
    x37 = np.ascontiguousarray(x[:37])
    layer.step = 1                                      # D = 1: a new step refreshes
    with torch.no_grad():
        y37 = layer(to_dev(x37))
    yref, yabs, yal = _ref_y(x37, w, osc.amax(x37), osc.amax(w))
    bf16_check(y37, yref, yal, yabs, K, "37 tokens")
    with pytest.raises(ValueError):
        layer(to_dev(x37).requires_grad_(True))


def test_sample_and_hold_across_steps():
    """Period 2 over optimizer steps 0..3 with X and W changing every step:
    the layer's references follow the oracle's sample-and-hold trace, and Y
    at each step equals the oracle's with the held references."""
    T, K, N = 64, 128, 96
    x0, w0, _ = _inputs(4, T, K, N)
    layer = _layer(K, N, w0, period=2)
    ox, ow = osc.AmaxState(2), osc.AmaxState(2)
    for t in range(4):
        say("sample-and-hold step", t)
        xt, wt = _scaled(x0, t + 1), _scaled(w0, 1.0 / (t + 1))
        with torch.no_grad():
            layer.weight.copy_(to_dev(wt))
        layer.step = t
        with torch.no_grad():
            y = layer(to_dev(xt))
        gx, rx = ox.observe(xt, t)
        gw, rw = ow.observe(wt, t)
        torch.cuda.synchronize()
        assert layer.amax_x.last_refresh == ox.last_refresh and layer.amax_w.last_refresh == ow.last_refresh
        assert np.float32(layer.amax_x.amax.item()) == gx and np.float32(layer.amax_w.amax.item()) == gw
        yref, yabs, yal = _ref_y(xt, wt, gx, gw)
        bf16_check(y, yref, yal, yabs, K, f"step {t}")


def test_inference_policies():
    """Delayed: the weight reference is measured on the first batch and
    held (even after the weight changes), activations refresh every 50
    batches.  Current: every batch.  Calibrated: the largest calibration
    amax, held for every later batch."""
    T, K, N = 48, 96, 64
    x0, w0, _ = _inputs(6, T, K, N)
    batches = [_scaled(x0, f) for f in (1.0, 3.0, 0.5)]

    say("inference delayed")
    layer = _layer(K, N, w0, period=50).inference_policy("delayed")
    gw0 = osc.amax(w0)
    w1 = _scaled(w0, 4.0)
    for i, xb in enumerate(batches):
        with torch.no_grad():
            y = layer(to_dev(xb))
            if i == 0:
                layer.weight.copy_(to_dev(w1))       # held weight reference stays gw0
        wcur = w0 if i == 0 else w1
        yref, yabs, yal = _ref_y(xb, wcur, osc.amax(batches[0]), gw0)
        bf16_check(y, yref, yal, yabs, K, f"delayed batch {i}")
    assert layer.batches == 3 and layer.amax_w.last_refresh == 0

    say("inference current")
    layer = _layer(K, N, w0).inference_policy("current")
    for i, xb in enumerate(batches):
        with torch.no_grad():
            y = layer(to_dev(xb))
        yref, yabs, yal = _ref_y(xb, w0, osc.amax(xb), gw0)
        bf16_check(y, yref, yal, yabs, K, f"current batch {i}")

    say("inference calibrated")
    layer = _layer(K, N, w0)
    layer.inference_policy("calibrated", calibration=[to_dev(b) for b in batches])
    gcal = osc.calibrated_amax(batches)
    torch.cuda.synchronize()
    assert np.float32(layer.amax_x.amax.item()) == gcal
    big = _scaled(x0, 10.0)
    for xb in (big, batches[2]):
        with torch.no_grad():
            y = layer(to_dev(xb))
        yref, yabs, yal = _ref_y(xb, w0, gcal, gw0)
        bf16_check(y, yref, yal, yabs, K, "calibrated")
    assert np.float32(layer.amax_x.amax.item()) == gcal


def test_amax_accumulate_running_max():
    """ue5m3_amax_accumulate: clear on the first batch, then the running
    maximum, equal to the oracle's calibrated reference; an empty batch
    leaves the value unchanged."""
    from paper_2609_02846_amd import amax_accumulate
    say("amax accumulate")
    bs = [synthetic.activation(s, 33, 48) for s in range(4)]
    acc = torch.full((1,), 123.0, device="cuda")
    for i, b in enumerate(bs):
        amax_accumulate(to_dev(b), acc, clear=(i == 0))
    amax_accumulate(torch.empty(0, dtype=torch.bfloat16, device="cuda"), acc)
    torch.cuda.synchronize()
    assert np.float32(acc.item()) == osc.calibrated_amax(bs)


@pytest.mark.parametrize("pm_grid", [None, 1024])
def test_training_step_block32(pm_grid):
    """The block-size control through the layer: X, W, dY quantized with
    blocks of 32 (32 x 32 weight tiles); Y, dX and dW equal the oracle's
    block-32 products (decoded-operand GEMM bar, or the probe-matched model
    exactly, up to the bf16 rounding of Y and dX)."""
    from oracle import accumulate as oacc
    T, K, N = 544, 416, 288
    say("linear training step block 32", T, K, N, "pm", pm_grid)
    x, w, dy = _inputs(13, T, K, N)
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    layer = _layer(K, N, w, period=50, seed=9, layer_id=2, block=32, pm_grid=pm_grid)
    xd = to_dev(x).requires_grad_(True)
    y = layer(xd)
    y.backward(to_dev(dy))
    torch.cuda.synchronize()
    yref, yabs, yal = _ref_y(x, w, gx, gw, block=32)
    (dref, dabs, dal), (wref, wabs, wal) = _ref_grads(x, w, dy, gx, gw, gd, 9, 2, block=32)
    if pm_grid is None:
        bf16_check(y, yref, yal, yabs, K, "Y")
        bf16_check(xd.grad, dref, dal, dabs, N, "dX")
        bf16_check(layer.weight.grad, wref, wal, wabs, T, "dW")
        return
    # probe-matched: exact model at sampled outputs, then the bf16 rounding
    xr = oq.quantize_1d(x, 1, gx, block=32)
    wq = oq.quantize_2d(w, gw, tile=32)
    X, W = oq.decoded_1d(xr[0], xr[1], 1, block=32), oq.decoded_2d(wq[0], wq[1], tile=32)
    al = ogemm.alpha(xr[2], wq[3])
    rng = np.random.default_rng(1)
    got = host(y.float())
    for m, n in [(0, 0), (T - 1, N - 1)] + [(int(rng.integers(T)), int(rng.integers(N))) for _ in range(60)]:
        want = np.float32(oacc.dot(X[m] * W[n], 1024, al)[0])
        want = torch.tensor([want]).to(torch.bfloat16).float().item()
        assert got[m, n] == want, (m, n, got[m, n], want)
