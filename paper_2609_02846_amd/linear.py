"""FP4 linear layer: Y = X W^T with the UE5M3 recipe in all three GEMMs.

A ``torch.autograd.Function`` over the library's calls (argument marshalling
only; every quantization and product runs in the HIP kernels):

forward (Sec. 2.3, Table 5; eq:delayed-amax)
  * sample-and-hold amax of X and W at the layer's step;
  * X row blocks RN (the fprop operand) and, when W needs a gradient, X
    column blocks RN (the wgrad operand, blocked along tokens) from one
    read;
  * W 16x16 tiles RN, plus the transposed payload when X needs a gradient;
  * fprop GEMM, bf16 Y.

backward (eq:sr: stochastic rounding on the upstream gradient only; RN on
request)
  * sample-and-hold amax of dY;
  * dY row blocks SR -> dgrad GEMM dX = dY W (bf16);
  * dY column blocks SR -> wgrad GEMM dW = dY^T X (in the weight's dtype).

Policies (Table tab:inference-scale-summary):
  * training: every operand refreshes every ``period`` optimizer steps
    (50 in the recipe, 1 = current scaling); the caller sets ``step`` to the
    optimizer-step index;
  * inference (``inference_policy``): the weight amax is measured on the
    first batch and held; activations refresh every 50 batches ("delayed"),
    every batch ("current"), or use a calibrated reference held fixed
    ("calibrated", after ``calibrate``); the batch index is the layer's own
    forward count.

SR randomness: each backward call draws from Philox with key ``seed`` +
(number of earlier backward calls of this layer), counter block
(element index, tensor id); the tensor ids are 2 * layer_id + 1 (dgrad
operand) and 2 * layer_id + 2 (wgrad operand), so layers and the two dY
blockings never share words.

Block-size control (Sec. "Recipe comparison", Table tab:results):
``block=32`` runs every 1D block and weight tile at 32 (one scale code per
32 elements, 32 x 32 weight tiles) with the rest of the recipe unchanged.

Shapes: in_features and out_features multiples of the block (16 or 32);
with W trainable the token count (X's leading dimensions flattened) must
be a multiple of the block too.  Weights are bf16.  There is no bias term.
"""

import torch

from . import (AmaxState, amax_accumulate, amax_sample, amax_sample_rht, gemm, gemm_pm, quantize_1d,
               quantize_2d, quantize_cols_rht, quantize_dual)


class _FP4LinearFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x2d, weight, layer, need_dx, need_dw):
        # need_dx / need_dw are decided by the caller: autograd runs this
        # method with gradients disabled.
        T, K = x2d.shape
        N = weight.shape[0]
        step = layer._forward_step()
        amax_sample(layer.amax_x, x2d, step)
        amax_sample(layer.amax_w, weight, step)
        tx = layer.target
        B = layer.block
        dec_xc = None
        if B == 32:
            xr, sxr, dec_x = quantize_1d(x2d, 1, layer.amax_x.amax, tx, "rn", block=32)
            xc = sxc = None
            if need_dw:
                xc, sxc, dec_xc = quantize_1d(x2d, 0, layer.amax_x.amax, tx, "rn", block=32)
        elif need_dw and layer.rht_wgrad:
            xr, sxr, dec_x = quantize_1d(x2d, 1, layer.amax_x.amax, tx, "rn")
            amax_sample_rht(layer.amax_xt, x2d, layer.rht_mask, step)
            xc, sxc, dec_xc = quantize_cols_rht(x2d, layer.amax_xt.amax, layer.rht_mask, tx, "rn")
        elif need_dw:
            (xr, sxr, dec_x), (xc, sxc, _) = quantize_dual(x2d, layer.amax_x.amax, tx, "rn")
            dec_xc = dec_x
        else:
            xr, sxr, dec_x = quantize_1d(x2d, 1, layer.amax_x.amax, tx, "rn")
            xc = sxc = None
        pw, sw, pwt, dec_w, swt = quantize_2d(weight, layer.amax_w.amax, tx, "rn", transposed=need_dx, tile=B)
        y = layer._gemm("nt", T, N, K, xr, sxr, dec_x, pw, sw, dec_w, out_dtype=torch.bfloat16)
        ctx.layer = layer
        ctx.step = step
        ctx.shape = (T, K, N)
        ctx.wdtype = weight.dtype
        ctx.save_for_backward(xc, sxc, dec_xc, pwt, swt, dec_w)
        return y

    @staticmethod
    def backward(ctx, dy):
        layer = ctx.layer
        T, K, N = ctx.shape
        xc, sxc, dec_xc, pwt, swt, dec_w = ctx.saved_tensors
        dy = dy.to(torch.bfloat16).contiguous()
        amax_sample(layer.amax_dy, dy, ctx.step)
        seed = layer._next_sr_seed()
        dx = dw = None
        mode = layer.grad_rounding
        if ctx.needs_input_grad[0]:
            dr = quantize_1d(dy, 1, layer.amax_dy.amax, layer.target, mode, seed, 2 * layer.layer_id + 1,
                             block=layer.block)
            dx = layer._gemm("nn", T, K, N, *dr, pwt, swt, dec_w, out_dtype=torch.bfloat16)
        if ctx.needs_input_grad[1]:
            tid = 2 * layer.layer_id + 2
            if layer.rht_wgrad:
                amax_sample_rht(layer.amax_dyt, dy, layer.rht_mask, ctx.step)
                dc = quantize_cols_rht(dy, layer.amax_dyt.amax, layer.rht_mask, layer.target_dy_wgrad, mode,
                                       seed, tid)
            else:
                dc = quantize_1d(dy, 0, layer.amax_dy.amax, layer.target_dy_wgrad, mode, seed, tid,
                                 block=layer.block)
            dw = layer._gemm("tn", N, K, T, *dc, xc, sxc, dec_xc, out_dtype=ctx.wdtype)
        return dx, dw, None, None, None


class Linear(torch.nn.Module):
    """FP4 (E2M1 + UE5M3 block scales) linear layer without bias.

    ``period``: sample-and-hold period D in optimizer steps (50 in the
    recipe).  ``target``: scale target T (448); ``target_dy_wgrad``: T of the
    wgrad dY operand (448, or 2048 for the paper's override).  The weight is
    bf16 and so is its gradient (the wgrad GEMM writes it directly).
    ``grad_rounding``: "sr" (the recipe) or "rn" for the dY quantizers.
    ``pm_grid``: None runs the decoded-operand GEMMs (fp32 accumulation);
    an integer d runs all three products through the probe-matched output
    model with final-grid denominator d (0 = no snap, the paper's 1024).
    ``rht_wgrad``: quantize the two wgrad operands (X and dY blocked along
    tokens) after a 16-point randomized Hadamard transform with one sign mask
    per layer (drawn from ``seed``), each with the amax of its transformed
    tensor as reference (the "UE5M3 with Transformer Engine settings"
    recipe, with ``period`` 1 and ``pm_grid`` 1024).  ``block``: 16 (the
    recipe) or 32 (the block-size control; not with ``rht_wgrad``)."""

    def __init__(self, in_features, out_features, period=50, target=448.0, target_dy_wgrad=448.0,
                 seed=0, layer_id=0, device="cuda", grad_rounding="sr", pm_grid=None, rht_wgrad=False,
                 block=16):
        super().__init__()
        if grad_rounding not in ("sr", "rn"):
            raise ValueError("grad_rounding must be 'sr' or 'rn'")
        if block not in (16, 32):
            raise ValueError("block must be 16 or 32")
        if block == 32 and rht_wgrad:
            raise ValueError("the Hadamard transform works on blocks of 16")
        self.block = int(block)
        self.grad_rounding, self.pm_grid = grad_rounding, pm_grid
        self.rht_wgrad = bool(rht_wgrad)
        self.rht_mask = (((int(seed) * 0x9E3779B97F4A7C15 + 0x632BE59BD9B4E019) % 2 ** 64) >> 48) & 0xFFFF
        if in_features % block or out_features % block or in_features <= 0 or out_features <= 0:
            raise ValueError(f"in_features and out_features must be positive multiples of {block}")
        self.in_features, self.out_features = int(in_features), int(out_features)
        self.weight = torch.nn.Parameter(
            torch.empty(out_features, in_features, dtype=torch.bfloat16, device=device))
        torch.nn.init.normal_(self.weight, std=in_features ** -0.5)
        self.target, self.target_dy_wgrad = float(target), float(target_dy_wgrad)
        self.seed, self.layer_id = int(seed), int(layer_id)
        self.amax_x = AmaxState(period, device)
        self.amax_w = AmaxState(period, device)
        self.amax_dy = AmaxState(period, device)
        self.amax_xt = AmaxState(period, device)     # transformed wgrad operands
        self.amax_dyt = AmaxState(period, device)
        self.step = 0               # optimizer-step index, set by the training loop
        self.sr_calls = 0           # backward calls so far (SR key offset)
        self.batches = 0            # forward calls under an inference policy
        self.policy = None          # None = training

    # -- scale policies -------------------------------------------------
    def inference_policy(self, policy="delayed", calibration=None):
        """Switch to an inference-scale policy: "delayed" (D = 50),
        "current" (D = 1) or "calibrated" (the largest amax over the
        ``calibration`` batches, held fixed).  Caches start empty; the weight
        reference is measured on the first batch and held."""
        if policy not in ("delayed", "current", "calibrated"):
            raise ValueError(policy)
        self.amax_w.set_period(0)
        self.amax_x.set_period(50 if policy == "delayed" else 1)
        if policy == "calibrated":
            if not calibration:
                raise ValueError("the calibrated policy needs calibration batches")
            self.calibrate(calibration)
        self.policy, self.batches = policy, 0
        return self

    def calibrate(self, batches):
        """Hold the largest activation amax over ``batches`` (bf16 tensors of
        [..., in_features]) as X's reference from now on."""
        for i, b in enumerate(batches):
            amax_accumulate(self._flat(b), self.amax_x.amax, clear=(i == 0))
        self.amax_x.freeze()

    def training_policy(self, period=50):
        """Back to training: every operand refreshes every ``period`` steps,
        from empty caches."""
        for st in (self.amax_x, self.amax_w, self.amax_dy, self.amax_xt, self.amax_dyt):
            st.set_period(period)
        self.policy = None
        return self

    # -- internals ------------------------------------------------------
    def _gemm(self, *args, **kw):
        if self.pm_grid is None:
            return gemm(*args, block=self.block, **kw)
        return gemm_pm(*args, grid=self.pm_grid, block=self.block, **kw)

    def _forward_step(self):
        if self.policy is None:
            return self.step
        b = self.batches
        self.batches += 1
        return b

    def _next_sr_seed(self):
        s = (self.seed + self.sr_calls) & (2 ** 64 - 1)
        self.sr_calls += 1
        return s

    def _flat(self, x):
        if x.dtype != torch.bfloat16 or x.shape[-1] != self.in_features:
            raise ValueError(f"input must be bf16 with last dimension {self.in_features}")
        return x.reshape(-1, self.in_features).contiguous()

    def forward(self, x):
        x2d = self._flat(x)
        grad = torch.is_grad_enabled()
        need_dx = grad and x.requires_grad
        need_dw = grad and self.weight.requires_grad
        if need_dw and x2d.shape[0] % self.block:
            raise ValueError("the wgrad operand is blocked along tokens: token count must be a "
                             f"multiple of {self.block}")
        y = _FP4LinearFn.apply(x2d, self.weight, self, need_dx, need_dw)
        return y.reshape(*x.shape[:-1], self.out_features)

    def extra_repr(self):
        return (f"in_features={self.in_features}, out_features={self.out_features}, target={self.target}, "
                f"block={self.block}")
