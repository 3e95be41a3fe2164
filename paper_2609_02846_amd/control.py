"""Teacher-student regression control (paper App. "Statistical Consequences
of the Probe-Matched Emulator", Sec. "Optimizer-level regression control",
Table tab:grid-regression).

A two-layer student 256 -> 256 -> 64 without biases (81,920 weights) learns
a fixed teacher of the same shape from 2,048 fixed training examples,
evaluated on 1,024 fixed examples, with minibatches of 128 and 500 AdamW
updates.  The quantized student runs the forward, data-gradient and
weight-gradient products of both layers through the FP4 ``Linear`` (UE5M3
block scales, scale target 448, sample-and-hold period 50, no Hadamard
transform) with the probe-matched GEMM and a final-grid denominator d; the
control is the same student with plain BF16 products.  For one seed every
variant shares the teacher, the data, the initial weights, the minibatch
order and the SR key.

Readings where the paper gives no detail (this module's choices): no
activation between the two layers of teacher and student (a two-layer
linear network: with a ReLU, tanh or GELU the 81,920-weight student does
not fit the 2,048 examples, and its evaluation error of 0.05-0.17, not
quantization, dominates); inputs N(0, 1); teacher and initial student
weights N(0, 1/fan_in) from independent streams; training labels carry
Gaussian noise of standard deviation 0.1 (evaluation targets are the clean
teacher outputs), which puts the BF16 control's final evaluation error at
the paper's magnitude; mean squared error; AdamW (lr 1e-3, betas
0.9/0.999, weight decay 0.01) on fp32 master weights that are rounded to
the bf16 layer weights after every update.  The final evaluation runs the
trained student as it trains (FP4 products for the FP4 student);
``eval_mse_bf16`` evaluates the same final weights with BF16 products.
"""

import numpy as np
import torch

from .linear import Linear

D_IN, D_HID, D_OUT = 256, 256, 64
N_TRAIN, N_EVAL, BATCH, STEPS = 2048, 1024, 128, 500


LABEL_NOISE = 0.1


def _data(seed, device, label_noise=LABEL_NOISE):
    g = torch.Generator(device="cpu").manual_seed(seed)
    w1 = torch.randn(D_HID, D_IN, generator=g) / D_IN ** 0.5
    w2 = torch.randn(D_OUT, D_HID, generator=g) / D_HID ** 0.5
    x_tr = torch.randn(N_TRAIN, D_IN, generator=g)
    x_ev = torch.randn(N_EVAL, D_IN, generator=g)
    teach = lambda x: (x @ w1.T) @ w2.T
    s1 = torch.randn(D_HID, D_IN, generator=g) / D_IN ** 0.5
    s2 = torch.randn(D_OUT, D_HID, generator=g) / D_HID ** 0.5
    order = torch.stack([torch.randperm(N_TRAIN, generator=g)[:BATCH] for _ in range(STEPS)])
    y_tr = teach(x_tr)
    if label_noise:
        # noisy teacher labels for training; evaluation targets stay clean
        y_tr = y_tr + label_noise * torch.randn(y_tr.shape, generator=g)
    dev = lambda t: t.to(device)
    return dict(x_tr=dev(x_tr.bfloat16()), y_tr=dev(y_tr), x_ev=dev(x_ev.bfloat16()),
                y_ev=dev(teach(x_ev)), init=(s1, s2), order=order)


def run(seed=42, mode="fp4", grad_rounding="rn", grid=1024, steps=STEPS, device="cuda",
        label_noise=LABEL_NOISE):
    """One training run.  mode "fp4" (FP4 Linear, probe-matched GEMM with
    final-grid denominator ``grid``) or "bf16" (control).  Returns a dict
    with per-step losses, master-gradient norms and zero-gradient rates,
    the final evaluation MSE (of the trained model as it runs: FP4 products
    for "fp4"), the same final weights evaluated with plain BF16 products
    (``eval_mse_bf16``) and the final fp32 master weights."""
    d = _data(seed, device, label_noise)
    masters = [torch.nn.Parameter(w.clone().to(device)) for w in d["init"]]
    opt = torch.optim.AdamW(masters, lr=1e-3, betas=(0.9, 0.999), weight_decay=0.01)
    if mode == "fp4":
        layers = [Linear(D_IN, D_HID, period=50, target=448.0, seed=1000 * seed + 1, layer_id=0,
                         device=device, grad_rounding=grad_rounding, pm_grid=grid),
                  Linear(D_HID, D_OUT, period=50, target=448.0, seed=1000 * seed + 2, layer_id=1,
                         device=device, grad_rounding=grad_rounding, pm_grid=grid)]
        weights = [l.weight for l in layers]
    elif mode == "bf16":
        layers = None
        weights = [torch.nn.Parameter(torch.empty(m.shape, dtype=torch.bfloat16, device=device)) for m in masters]
    else:
        raise ValueError(mode)

    def sync_weights():
        with torch.no_grad():
            for w, m in zip(weights, masters):
                w.copy_(m)

    def forward(x, step):
        if layers is None:
            return torch.nn.functional.linear(torch.nn.functional.linear(x, weights[0]), weights[1])
        for l in layers:
            l.step = step
        return layers[1](layers[0](x))

    def eval_mse(step):
        with torch.no_grad():
            y = forward(d["x_ev"], step)
            return float(torch.mean((y.float() - d["y_ev"]) ** 2))

    sync_weights()
    losses, gnorms, zeros = [], [], []
    for t in range(steps):
        idx = d["order"][t].to(device)
        for w in weights:
            w.grad = None
        y = forward(d["x_tr"][idx], t)
        loss = torch.mean((y.float() - d["y_tr"][idx]) ** 2)
        loss.backward()
        for w, m in zip(weights, masters):
            m.grad = w.grad.float()
        flat = torch.cat([m.grad.flatten() for m in masters])
        losses.append(float(loss.detach()))
        gnorms.append(float(flat.norm()))
        zeros.append(float((flat == 0).float().mean()))
        opt.step()
        sync_weights()
    with torch.no_grad():
        wb = [m.to(torch.bfloat16) for m in masters]
        yb = torch.nn.functional.linear(torch.nn.functional.linear(d["x_ev"], wb[0]), wb[1])
        mse_bf16 = float(torch.mean((yb.float() - d["y_ev"]) ** 2))
    return dict(losses=np.array(losses), grad_norms=np.array(gnorms), zero_grad=np.array(zeros),
                eval_mse=eval_mse(steps), eval_mse_bf16=mse_bf16, masters=[m.detach().clone() for m in masters])


def same_trajectory(a, b):
    """Exact equality of two runs' records and final weights."""
    rec = all(np.array_equal(a[k], b[k]) for k in ("losses", "grad_norms", "zero_grad"))
    state = all(torch.equal(x, y) for x, y in zip(a["masters"], b["masters"]))
    return rec, state
