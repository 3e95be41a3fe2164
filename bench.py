#!/usr/bin/env python3
"""Benchmark of one UE5M3 FP4 linear training step on one MI355X.

A step is the whole per-linear hot path on the Nemotron-H-8B FFN
up-projection (T = 8192 tokens, K = 4096, N = 21504):
  sample-and-hold amax (D = 50; a refresh launches the amax kernels),
  X rows and columns RN (re-blocked along tokens) from one read, W 16x16
  tiles RN (+ the transposed payload), dY rows SR, dY columns SR,
  fprop Y = X W^T (bf16 out), dgrad dX = dY W (bf16 out),
  wgrad dW = dY^T X (fp32 out).
Inputs are seeded synthetic bf16 tensors resident in HBM before timing; the
step cycles through four input and output sets (over 2 GB) so that no step
reads what the previous one left in the 256 MB Infinity Cache.  The
refresh-step amax is timed on its own and charged at its 1/D rate.

Prints ONE JSON line.  ``value`` = emulated-FP4 GEMM TFLOP/s of the whole
step (3 x 2TNK flops / step time, quantizers and amax included).  Beside it:
per-kernel HIP-event times inside the timed region, each quantizer alone on
the rotating sets, the quantizer-only workload (activation / gradient /
weight), the single small linear's latency, the roofline of the fprop GEMM
and the oracle's CPU baseline (timed first, on the host cores).
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, TFLOP/s
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12   # 32-bit (and binary64 add) VALU lane ops/s
PM_VALU_PER_GROUP = 9          # probe-matched output model: VALU ops per output per 64-product group
PM_VALU_MEASURED = 11.1        # the same, as issued (SQ_INSTS_VALU of the fprop launch): model + decode, span check, addressing
METRIC = "quantize GB/s + emulated FP4 GEMM TFLOP/s (fprop+dgrad+wgrad), % roofline"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--tokens", type=int, default=8192)
    p.add_argument("--k", type=int, default=4096)
    p.add_argument("--n", type=int, default=21504)
    p.add_argument("--period", type=int, default=50)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--step-only", action="store_true",
                   help="profiling aid: only the step (warm-up, refresh timing, timed steps); no isolated "
                        "quantizer runs, quantizer workload or small-linear lines, so that every launch of a "
                        "kernel in a trace has the step's shape")
    p.add_argument("--valu", default=os.path.join(ROOT, "profiles", "quantizer_valu.json"),
                   help="VALU instructions per element of the SR quantizers from rocprofv3 counters (JSON)")
    p.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "gemm_traffic.json"),
                   help="HBM traffic per launch measured with rocprofv3 counters (JSON)")
    p.add_argument("--kernel", default=None,
                   help="profiling aid: after setup run only this step kernel (e.g. gemm_fprop) "
                        "--steps times and exit without a JSON line")
    p.add_argument("--pm", type=int, default=None, metavar="GRID",
                   help="run the step with the probe-matched GEMMs (64-product RNE partials, "
                        "toward-zero cross-group adds, 1/GRID snap; 0 = no snap)")
    p.add_argument("--rht", action="store_true",
                   help="quantize the wgrad operands (X and dY blocked along tokens) after the 16-point "
                        "randomized Hadamard transform, each with its transformed amax")
    p.add_argument("--control", action="store_true",
                   help="teacher-student regression control: BF16 vs FP4 (probe-matched GEMM) final-eval MSE "
                        "and grid invariance over seeds 41-43, RN and SR gradients")
    p.add_argument("--drift", action="store_true",
                   help="the FFN down-projection drift run (T=8192, K=21504, N=4096): 120 steps with the "
                        "sample-and-hold reference (--period) while operand magnitudes drift and spike; "
                        "prints its own JSON line")
    p.add_argument("--formats", action="store_true",
                   help="scale-format comparison instead of the headline step: UE5M3 (delayed "
                        "amax; blocks of 16 and the block-32 control), E4M3 (current amax) and "
                        "E8M0 (blocks of 32) on the QKV workload "
                        "X [16384, 4096], W [6144, 4096], dY [16384, 6144]; one JSON line")
    p.add_argument("--copy-ref", type=int, default=0, metavar="BYTES",
                   help="profiling aid: time a plain device copy of BYTES bytes (the reference "
                        "that scales the HBM byte counters) and exit")
    p.add_argument("--matmul-ref", action="store_true",
                   help="ceiling reference only (not the product path): time a plain bf16 "
                        "torch.matmul for each of the step's three GEMM shapes and exit")
    p.add_argument("--gemm-shapes", action="store_true",
                   help="profiling aid: the fprop-layout GEMM at the step's flops (2 x 8192 x 21504 x "
                        "4096) split into fewer, longer tiles (K = 4096, 8192, 16384, 21504), bf16 and "
                        "fp32 outputs, one line per shape, then exit")
    return p.parse_args()


def gemm_source_hash():
    """Hash of the GEMM kernel source with comments and blank lines removed:
    the stored HBM traffic figure is valid only for the code it was measured
    on, and a comment edit does not change that code."""
    import hashlib
    h = hashlib.sha256()
    for f in ("gemm.hip", "fp4_decode.hpp", "codec.hpp"):
        text = open(os.path.join(ROOT, "paper_2609_02846_amd", "csrc", f), encoding="utf-8").read()
        lines = (ln.split("//")[0].rstrip() for ln in text.splitlines())
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()[:16]


def quantize_source_hash():
    """Hash of the quantizer kernel source with comments and blank lines
    removed (the stored VALU counts are valid only for that code)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("quantize.hip", "codec.hpp"):
        text = open(os.path.join(ROOT, "paper_2609_02846_amd", "csrc", f), encoding="utf-8").read()
        lines = (ln.split("//")[0].rstrip() for ln in text.splitlines())
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()[:16]


def quant_bytes_1d(rows, cols):
    return rows * cols * 2 + rows * cols // 2 + rows * cols // 16


def quant_bytes_dual(rows, cols):
    return rows * cols * 2 + 2 * (rows * cols // 2 + rows * cols // 16)


def quant_bytes_2d(rows, cols, transposed):
    return rows * cols * 2 + rows * cols // 2 * (2 if transposed else 1) + rows * cols // 256


# ------------------------------------------------------------ CPU leg ----
_POOL = {}


def _pool_quantize(job):
    """One worker's row shard of an oracle quantization (forked worker; the
    tensors come from _POOL)."""
    from oracle import quantize as oq
    kind, r0, r1 = job
    x = _POOL[kind]
    g = _POOL["g_" + kind]
    if kind == "w":
        oq.quantize_2d(x[r0:r1], g)
    elif kind == "x":
        oq.quantize_1d(x[r0:r1], 1, g)
    else:
        rows = np.arange(r0, r1, dtype=np.int64)
        idx = rows[:, None] * x.shape[1] + np.arange(x.shape[1], dtype=np.int64)[None, :]
        oq.quantize_1d(x[r0:r1], 1, g, 448.0, "sr", 1, 0, elem_index=idx)
    return r1 - r0


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(T, K, N):
    """The oracle, as it stands, timed on this host's cores (run before the
    GPU is touched, so the worker pool forks a GPU-free process):
      * the quantizer workload (activation [8192, 4096] rows RN, gradient
        [8192, 4096] rows SR with Philox seed 1, weight [4096, 4096] 16 x 16
        tiles RN) on the whole tensors, in one process and row-sharded over a
        pool of all cores;
      * the fprop product of the FFN up-projection shape (T x K by K x N) as a
        float32 BLAS matmul on all cores, with decoded FP4 operands (the
        weight's rows tiled from the decoded 4096 x 4096 weight).
    The step estimate takes the pool's per-element quantizer cost for the
    step's five quantizations and three fprop-sized products.  Returns the
    cpu_baseline object (value in the metric's unit, TFLOP/s of GEMM work
    per step)."""
    import multiprocessing as mp
    import synthetic
    from oracle import gemm as og
    from oracle import quantize as oq
    from oracle import scaling as osc
    t_all = time.perf_counter()
    wl = synthetic.quantizer_bandwidth(0)
    x, dy, w = wl["x"], wl["dy"], wl["w"]
    cores = min(len(os.sched_getaffinity(0)), 16)
    res = {}
    nbytes = {"x": quant_bytes_1d(*x.shape), "dy": quant_bytes_1d(*dy.shape), "w": quant_bytes_2d(*w.shape, False)}
    _POOL.update({"x": x, "dy": dy, "w": w, "g_x": osc.amax(x), "g_dy": osc.amax(dy), "g_w": osc.amax(w)})
    for kind in ("x", "dy", "w"):
        t0 = time.perf_counter()
        _pool_quantize((kind, 0, _POOL[kind].shape[0]))
        res[kind] = {"single_s": round(time.perf_counter() - t0, 3)}
    with mp.get_context("fork").Pool(cores) as pool:
        for kind in ("x", "dy", "w"):
            R = _POOL[kind].shape[0]
            step = (R // (4 * cores)) // 16 * 16 or 16
            jobs = [(kind, r, min(R, r + step)) for r in range(0, R, step)]
            t0 = time.perf_counter()
            assert sum(pool.map(_pool_quantize, jobs)) == R
            res[kind]["pool_s"] = round(time.perf_counter() - t0, 3)
    for kind in ("x", "dy", "w"):
        res[kind]["single_GBps"] = round(nbytes[kind] / res[kind]["single_s"] / 1e9, 4)
        res[kind]["pool_GBps"] = round(nbytes[kind] / res[kind]["pool_s"] / 1e9, 4)
    _POOL.clear()
    # fp32 BLAS fprop at the step's shape on decoded operands
    xq = oq.quantize_1d(x, 1, osc.amax(x))
    wq = oq.quantize_2d(w, osc.amax(w))
    X = oq.decoded_1d(xq[0], xq[1], 1).astype(np.float32)[:T, :K]
    Wd = oq.decoded_2d(wq[0], wq[1]).astype(np.float32)
    W = np.ascontiguousarray(np.tile(Wd, ((N + Wd.shape[0] - 1) // Wd.shape[0], 1))[:N, :K])
    al = og.alpha(xq[2], wq[3])
    t0 = time.perf_counter()
    og.fprop(X, W, al, accumulate="fp32")
    t_gemm = time.perf_counter() - t0
    del X, W, Wd
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = None
    # step estimate: per-element quantizer cost of the pool run (1D RN and SR
    # rows, 2D tiles) for the step's quantizations, plus three products
    per_el = {k: res[k]["pool_s"] / (nbytes[k] / (2.5625 if k != "w" else 2.50390625)) for k in res}
    t_quant = (2 * T * K * per_el["x"] + N * K * per_el["w"] + 2 * T * N * per_el["dy"])
    flop_step = 3 * 2.0 * T * N * K
    t_step = t_quant + 3 * t_gemm
    return {"value": flop_step / t_step / 1e12, "unit": "TFLOP/s", "cores": max(cores, blas_threads or 1),
            "kind": "oracle",
            "sample": (f"oracle quantizers on the whole quantizer-workload tensors (activation 8192x4096 rows RN, "
                       f"gradient 8192x4096 rows SR, weight 4096x4096 tiles RN), one process and a pool of "
                       f"{cores} processes; float32 BLAS fprop {T}x{K} by {K}x{N} on {blas_threads} threads; "
                       f"step estimate {t_step:.1f} s from the pool rates"),
            "pool_processes": cores, "blas_threads": blas_threads, "host_cpus": len(os.sched_getaffinity(0)),
            "cpu_model": _cpu_model(), "quantizers": res,
            "gemm_fp32_blas": {"s": round(t_gemm, 3), "TFLOP/s": round(2.0 * T * N * K / t_gemm / 1e12, 4)},
            "seconds": round(time.perf_counter() - t_all, 1)}


def _decode_rows(payload, scales, fmt):
    """Host decode of sampled quantized rows (measurement only): E2M1 value
    times its block scale, float64."""
    mag = np.array([0, .5, 1, 1.5, 2, 3, 4, 6], np.float64)
    p = payload.astype(np.uint8)
    nib = np.empty((p.shape[0], p.shape[1] * 2), np.uint8)
    nib[:, 0::2], nib[:, 1::2] = p & 15, p >> 4
    q = np.where(nib & 8, -1.0, 1.0) * mag[nib & 7]
    c = scales.astype(np.int64)
    if fmt == "e8m0":
        s = np.exp2(c - 127.0)
    else:
        bias, sub = (15, 2.0 ** -17) if fmt == "ue5m3" else (7, 2.0 ** -9)
        e, m = c >> 3, c & 7
        s = np.where(e == 0, m * sub, (1 + m / 8.0) * np.exp2(e - float(bias)))
    return q * np.repeat(s, q.shape[1] // s.shape[1], axis=1)


def control_bench(args):
    """Table tab:grid-regression structure: per gradient rounding, the mean
    BF16 and FP4 (d = 1024) final-eval MSE over seeds 41-43, and how many of
    the 15 (seed, nonzero d) runs reproduce the d = 0 run exactly (records:
    every loss, gradient norm and zero-gradient rate; states: final
    weights)."""
    from paper_2609_02846_amd import control
    grids = (256, 512, 1024, 2048, 4096)
    res = {}
    t0 = time.time()
    bf = {s: control.run(s, "bf16") for s in (41, 42, 43)}
    for rnd in ("rn", "sr"):
        mse_q, mse_qb, rec, st = [], [], 0, 0
        for s in (41, 42, 43):
            base = control.run(s, "fp4", rnd, grid=0)
            for d in grids:
                r = control.run(s, "fp4", rnd, grid=d)
                a, b = control.same_trajectory(base, r)
                rec += int(a)
                st += int(b)
                if d == 1024:
                    mse_q.append(r["eval_mse"])
                    mse_qb.append(r["eval_mse_bf16"])
            print(f"control {rnd} seed {s} done ({time.time() - t0:.0f} s)", flush=True)
        res[rnd] = {"bf16_eval_mse": round(float(np.mean([bf[s]["eval_mse"] for s in bf])), 6),
                    "fp4_eval_mse": round(float(np.mean(mse_q)), 6),
                    "fp4_weights_bf16_eval_mse": round(float(np.mean(mse_qb)), 6),
                    "exact_records": f"{rec}/15", "exact_states": f"{st}/15"}
    print(json.dumps({"metric": "teacher-student regression control (256-256-64, 500 AdamW steps, "
                                f"label noise {control.LABEL_NOISE})",
                      "unit": "final-eval MSE", "seeds": [41, 42, 43], "grids": list(grids),
                      "results": res, "paper": {"rn": {"bf16_eval_mse": 0.001956, "fp4_eval_mse": 0.027130,
                                                        "exact_records": "15/15", "exact_states": "15/15"},
                                                 "sr": {"bf16_eval_mse": 0.001956, "fp4_eval_mse": 0.027578,
                                                        "exact_records": "15/15", "exact_states": "15/15"}},
                      "seconds": round(time.time() - t0, 1)}), flush=True)


def formats_bench(args):
    """Config-5 comparison: per encoding, the step time of the quantizers and
    the three GEMMs, and the quantization error on sampled rows."""
    import torch
    import paper_2609_02846_amd as ue
    import synthetic
    T, K, N = 16384, 4096, 6144
    dev = torch.device("cuda:0")
    wl = synthetic.qkv_formats(0, T, K, N)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    x, w, dy = up(wl["x"]), up(wl["w"]), up(wl["dy"])
    flop = 3 * 2.0 * T * N * K
    rows = np.random.default_rng(0).choice(T, 256, replace=False)
    res = {}
    for name, fmt, B in [("ue5m3", "ue5m3", 16), ("ue5m3_b32", "ue5m3", 32), ("e4m3", "e4m3", 16),
                         ("e8m0", "e8m0", 32)]:
        period = 50 if fmt == "ue5m3" else 1
        kb = {} if fmt == "e8m0" else {"block": B}
        st = {n: ue.AmaxState(period) for n in "xwd"}
        y = torch.empty(T, N, dtype=torch.float32, device=dev)
        dx = torch.empty(T, K, dtype=torch.bfloat16, device=dev)
        dw = torch.empty(N, K, dtype=torch.float32, device=dev)
        out = {}

        def step(t):
            if fmt != "e8m0":
                ue.amax_sample(st["x"], x, t)
                ue.amax_sample(st["w"], w, t)
                ue.amax_sample(st["d"], dy, t)
            a = (lambda n: None) if fmt == "e8m0" else (lambda n: st[n].amax)
            out["xr"] = ue.quantize_1d(x, 1, a("x"), fmt=fmt, **kb)
            out["xc"] = ue.quantize_1d(x, 0, a("x"), fmt=fmt, **kb)
            out["dr"] = ue.quantize_1d(dy, 1, a("d"), 448.0, "sr", 1000 + t, 1, fmt=fmt, **kb)
            out["dc"] = ue.quantize_1d(dy, 0, a("d"), 448.0, "sr", 1000 + t, 2, fmt=fmt, **kb)
            if fmt == "e8m0":
                wr = ue.quantize_1d(w, 1, None, fmt=fmt)
                wc = ue.quantize_1d(w, 0, None, fmt=fmt)
                out["bf"], out["bd"] = (wr[0], wr[1], wr[2]), (wc[0], wc[1], wc[2])
            else:
                wq = ue.quantize_2d(w, a("w"), fmt=fmt, tile=B)
                out["bf"], out["bd"] = (wq[0], wq[1], wq[3]), (wq[2], wq[4], wq[3])
            ue.gemm("nt", T, N, K, *out["xr"], *out["bf"], out=y, fmt=fmt, **kb)
            ue.gemm("nn", T, K, N, *out["dr"], *out["bd"], out=dx, fmt=fmt, **kb)
            ue.gemm("tn", N, K, T, *out["dc"], *out["xc"], out=dw, fmt=fmt, **kb)

        for t in range(args.warmup):
            step(t)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for t in range(args.warmup, args.warmup + args.steps):
            step(t)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        # quantization error on 256 sampled rows (X, dY rows) and the fprop
        # output against fp32 products of the bf16 inputs
        xs = torch.from_numpy(synthetic.bf16_bits_to_f32(wl["x"][rows])).double().numpy()
        ds = torch.from_numpy(synthetic.bf16_bits_to_f32(wl["dy"][rows])).double().numpy()
        dec = lambda r, sel: _decode_rows(r[0].cpu().numpy()[sel], r[1].cpu().numpy()[sel], fmt) * \
            float(r[2].item())
        xq, dq = dec(out["xr"], rows), dec(out["dr"], rows)
        rel = lambda a, b: float(np.sqrt(np.mean((a - b) ** 2)) / np.sqrt(np.mean(b ** 2)))
        wf = synthetic.bf16_bits_to_f32(wl["w"])
        yref = (torch.from_numpy(synthetic.bf16_bits_to_f32(wl["x"][rows])).to(dev) @
                torch.from_numpy(wf).to(dev).t()).double().cpu().numpy()
        res[name] = {"ms_per_step": round(ms, 4), "gemm_TFLOPs_step": round(flop / ms / 1e9, 1),
                     "rel_rmse_x": round(rel(xq, xs), 5), "rel_rmse_dy": round(rel(dq, ds), 5),
                     "rel_rmse_y": round(rel(y[torch.from_numpy(rows).to(dev)].double().cpu().numpy(), yref), 5),
                     "amax_period": period if fmt != "e8m0" else None,
                     "blocks": B}
    print(json.dumps({"metric": "scale-format comparison (QKV workload)", "unit": "TFLOP/s",
                      "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "data": "synthetic",
                      "dtype": "fp4-e2m1 operands, fp32 accumulate",
                      "config": {"workload": "QKV projection T=16384 K=4096 N=6144, SR dY"},
                      "formats": res}), flush=True)


def drift_bench(args):
    """The drift run: FFN down-projection (T = 8192, K = 21504, N = 4096)
    for 120 steps with the sample-and-hold reference (eq:delayed-amax, period
    --period) while the operand magnitudes drift (lognormal walk, sigma 0.05
    per step) and spike (x20 on random steps).  Step t's operands are
    bf16(base x f_t), formed on the device between two timed intervals; each
    interval holds the step's whole path: the three sample-and-hold calls
    (amax kernels on refresh steps), X rows and columns from one read, W
    tiles, dY rows and columns (SR), fprop, dgrad and wgrad.  Reports the
    mean path time per step, the refresh steps and how many of the steps ran
    on a held reference that the current operand exceeds (saturating
    blocks) or undershoots by more than 2^10."""
    import torch
    import paper_2609_02846_amd as ue
    import synthetic
    T, K, N, STEPS = 8192, 21504, 4096, 120
    dev = torch.device("cuda:0")
    wl = synthetic.ffn_down_drift(0, T, K, N)
    f = synthetic.drift_factors(0, STEPS)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    base = [up(wl["x"]), up(wl["w"]), up(wl["dy"])]
    del wl
    bmax = [float(b.float().abs().max()) for b in base]
    cur = [torch.empty_like(b) for b in base]
    u8 = lambda *sh: torch.empty(sh, dtype=torch.uint8, device=dev)
    f32 = lambda *sh: torch.empty(sh, dtype=torch.float32, device=dev)
    xr, xc = (u8(T, K // 2), u8(T, K // 16), f32(1)), (u8(K, T // 2), u8(K, T // 16))
    wq = (u8(N, K // 2), u8(N // 16, K // 16), u8(K, N // 2), f32(1), u8(K // 16, N // 16))
    dr, dc = (u8(T, N // 2), u8(T, N // 16), f32(1)), (u8(N, T // 2), u8(N, T // 16), f32(1))
    y = torch.empty(T, N, dtype=torch.bfloat16, device=dev)
    dx = torch.empty(T, K, dtype=torch.bfloat16, device=dev)
    dw = torch.empty(N, K, dtype=torch.float32, device=dev)

    def run(st, t, ev=None):
        for j in range(3):
            torch.mul(base[j], float(f[t, j]), out=cur[j])
        if ev is not None:
            ev[0].record()
        n = [int(ue.amax_sample(st[r], cur[j], t)) for j, r in enumerate("xwd")]
        ue.quantize_dual(cur[0], st["x"].amax, 448.0, "rn", 0, 0, 0, xr[:2], xc, xr[2])
        ue.quantize_2d(cur[1], st["w"].amax, 448.0, "rn", 0, 0, True, *wq)
        ue.quantize_1d(cur[2], 1, st["d"].amax, 448.0, "sr", 5000 + t, 1, *dr)
        ue.quantize_1d(cur[2], 0, st["d"].amax, 448.0, "sr", 5000 + t, 2, *dc)
        ue.gemm("nt", T, N, K, xr[0], xr[1], xr[2], wq[0], wq[1], wq[3], out=y)
        ue.gemm("nn", T, K, N, dr[0], dr[1], dr[2], wq[2], wq[4], wq[3], out=dx)
        ue.gemm("tn", N, K, T, dc[0], dc[1], dc[2], xc[0], xc[1], xr[2], out=dw)
        if ev is not None:
            ev[1].record()
        return n

    warm = {r: ue.AmaxState(args.period) for r in "xwd"}
    for t in range(3):
        run(warm, t)
    torch.cuda.synchronize()
    st = {r: ue.AmaxState(args.period) for r in "xwd"}
    evs = [_events(2) for _ in range(STEPS)]
    refreshed = []
    for t in range(STEPS):
        refreshed.append(run(st, t, evs[t]))
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in evs])
    # held reference vs the operand's own amax, per role and step (from the
    # known base maxima and factors: bf16 rounding is monotone)
    held = np.zeros((STEPS, 3))
    last = [0.0, 0.0, 0.0]
    for t in range(STEPS):
        for j in range(3):
            if refreshed[t][j]:
                last[j] = bmax[j] * float(f[t, j])
            held[t, j] = last[j]
    ratio = np.array([[bmax[j] * float(f[t, j]) / held[t, j] for j in range(3)] for t in range(STEPS)])
    flop = 3 * 2.0 * T * N * K
    print(json.dumps({
        "metric": "drift run: quantize + emulated FP4 GEMM step time under sample-and-hold scaling",
        "unit": "ms", "value": round(float(ms.mean()), 4), "higher_is_better": False, "n_gpus": 1,
        "steps": STEPS, "warmup": 3, "data": "synthetic", "dtype": "fp16",
        "config": {"workload": "FFN down-projection drift run T=8192 K=21504 N=4096", "period": args.period,
                   "drift_sigma": 0.05, "spike": 20.0},
        "ms_per_step_p10_p50_p90": [round(float(q), 4) for q in np.percentile(ms, [10, 50, 90])],
        "gemm_TFLOPs": round(flop / (float(ms.mean()) * 1e-3) / 1e12, 1),
        "refresh_steps": [t for t in range(STEPS) if any(refreshed[t])],
        "refreshes_per_role": {r: int(sum(refreshed[t][j] for t in range(STEPS))) for j, r in enumerate("xwd")},
        "steps_above_held_reference": {r: int((ratio[:, j] > 1.0).sum()) for j, r in enumerate("xwd")},
        "steps_below_held_reference_by_2e10": {r: int((ratio[:, j] < 2.0 ** -10).sum()) for j, r in enumerate("xwd")},
        "max_operand_over_held": {r: round(float(ratio[:, j].max()), 2) for j, r in enumerate("xwd")},
    }), flush=True)


def matmul_ref(T, K, N, dev, verbose=True):
    """bf16 inputs, library GEMM (hipBLASLt through torch.matmul): what a plain
    dense bf16 product of the step's three shapes reaches on this GPU, as a
    ceiling reference for the FP4 GEMMs.  Operands are contiguous (the
    transposes are materialised before timing)."""
    import torch
    g = torch.Generator(device=dev).manual_seed(0)
    shapes = {"fprop": (T, K, N), "dgrad": (T, N, K), "wgrad": (N, T, K)}
    out = {}
    for name, (m, k, n) in shapes.items():
        a = torch.randn(m, k, device=dev, dtype=torch.bfloat16, generator=g)
        b = torch.randn(k, n, device=dev, dtype=torch.bfloat16, generator=g)
        c = torch.empty(m, n, device=dev, dtype=torch.bfloat16)
        for _ in range(5):
            torch.matmul(a, b, out=c)
        torch.cuda.synchronize()
        reps = 30
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.matmul(a, b, out=c)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        tf = 2.0 * m * n * k / (ms * 1e-3) / 1e12
        out[name] = {"m": m, "k": k, "n": n, "ms": round(ms, 4), "TFLOP/s": round(tf, 1),
                     "frac_bf16": round(tf / BF16_PEAK_TFLOPS, 4)}
        if verbose:
            print(f"[matmul-ref] {name} {m}x{k}x{n}: {ms:.3f} ms {tf:.1f} TFLOP/s", flush=True)
        del a, b, c
    return out


def copy_ceiling(dev, nbytes=352 * 2 ** 20, nsets=4):
    """A plain device copy (torch) of nbytes over nsets rotating buffer pairs:
    the HBM rate a streaming kernel reaches on this GPU (bytes read plus
    bytes written, per second), as a ceiling reference for the quantizers."""
    import torch
    n = nbytes // 4
    src = [torch.full((n,), 1.0 + i, dtype=torch.float32, device=dev) for i in range(nsets)]
    dst = [torch.empty(n, dtype=torch.float32, device=dev) for _ in range(nsets)]
    med, _, p = _time_kernel(lambda i: dst[i].copy_(src[i]), nsets, reps=20, warm=4)
    del src, dst
    gbs = 2 * nbytes / (med * 1e-3) / 1e9
    return {"bytes_moved": 2 * nbytes, "ms": round(med, 5), "GB/s": round(gbs, 1),
            "frac_hbm": round(gbs / HBM_PEAK_GBS, 4), "ms_p10_p50_p90": p}


def gemm_shapes(dev):
    """Equal-flop fprop GEMMs with 10.5, 5.25, 2.6 and 2 output tiles per CU:
    how the per-tile cost (epilogue, pipeline refill) shows at the step's
    K = 4096.  Operands are N(0,1) activations and N(0,0.02) weights,
    quantized by the library (RN, current amax)."""
    import torch
    import paper_2609_02846_amd as ue
    g = torch.Generator(device=dev).manual_seed(0)
    out = []
    for (M, N, K) in [(8192, 21504, 4096), (8192, 10752, 8192), (8192, 5376, 16384), (8192, 4096, 21504)]:
        x = torch.randn(M, K, device=dev, dtype=torch.float32, generator=g).to(torch.bfloat16)
        w = (0.02 * torch.randn(N, K, device=dev, dtype=torch.float32, generator=g)).to(torch.bfloat16)
        sx, sw = ue.AmaxState(50), ue.AmaxState(50)
        ue.amax_sample(sx, x, 0)
        ue.amax_sample(sw, w, 0)
        xp, xs, xd = ue.quantize_1d(x, 1, sx.amax)
        wp, ws, _, wd, _ = ue.quantize_2d(w, sw.amax, transposed=False)
        del x, w
        rec = {"M": M, "N": N, "K": K, "tiles_per_cu": round(((M + 255) // 256) * ((N + 255) // 256) / 256, 2)}
        for od in (torch.bfloat16, torch.float32):
            c = torch.empty(M, N, device=dev, dtype=od)
            # warm-up long enough for the clock to settle under load (the
            # first launches of a process run slower)
            for _ in range(15):
                ue.gemm("nt", M, N, K, xp, xs, xd, wp, ws, wd, out=c, out_dtype=od)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(20):
                ue.gemm("nt", M, N, K, xp, xs, xd, wp, ws, wd, out=c, out_dtype=od)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / 20
            name = "bf16" if od == torch.bfloat16 else "f32"
            rec[name + "_ms"] = round(ms, 4)
            rec[name + "_TFLOPs"] = round(2.0 * M * N * K / (ms * 1e-3) / 1e12, 1)
            del c
        print(f"[gemm-shapes] {rec}", flush=True)
        out.append(rec)
    print(json.dumps({"gemm_shapes": out}), flush=True)


NSETS = 4      # rotating input / output sets: > 512 MB, past the 256 MB Infinity Cache


class _HipEvent:
    """A HIP timing event recorded on torch's current stream, created
    without the system-scope memory fence that torch's events carry (the
    step's kernels exchange data only through device memory; measured: the
    fenced events lengthen the timed step by about 0.8%, these by 0.3%)."""
    _hip = None
    kDisableSystemFence = 0x20000000

    def __init__(self):
        import ctypes
        if _HipEvent._hip is None:
            _HipEvent._hip = ctypes.CDLL("libamdhip64.so")
        self.h = ctypes.c_void_p()
        if _HipEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.h),
                                                  ctypes.c_uint(self.kDisableSystemFence)) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self):
        import ctypes
        import torch
        if _HipEvent._hip.hipEventRecord(self.h, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, other):
        import ctypes
        ms = ctypes.c_float()
        if _HipEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self.h, other.h) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value


def _events(n):
    return [_HipEvent() for _ in range(n)]


def _time_kernel(fn, nsets, reps=30, warm=4):
    """Median / mean device time of fn(i) over reps launches, fn cycling
    through nsets buffer sets; HIP events on the current stream."""
    import torch
    for i in range(warm):
        fn(i % nsets)
    torch.cuda.synchronize()
    evs = [(_events(2)) for _ in range(reps)]
    for i in range(reps):
        evs[i][0].record()
        fn(i % nsets)
        evs[i][1].record()
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in evs])
    return float(np.median(ms)), float(ms.mean()), [round(float(q), 5) for q in np.percentile(ms, [10, 50, 90])]


def quantizer_workload(dev):
    """The quantizer-only workload: activation [8192, 4096] N(0,1) with 0.1% x100
    outliers, rows RN; gradient [8192, 4096] N(0, 1e-4) with a lognormal row
    scale, rows SR (Philox seed 1); weight [4096, 4096] N(0, 0.02), 16 x 16
    tiles RN; current amax.  Each quantizer alone over NSETS rotating input
    and output sets (640 MB of inputs), HIP events."""
    import torch
    import paper_2609_02846_amd as ue
    import synthetic
    wl = synthetic.quantizer_bandwidth(0)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    base = {k: up(wl[k]) for k in ("x", "dy", "w")}
    # sets 1.. are the same tensors scaled by 1 + i/128 (bf16): same distributions
    sets = [{k: (v.float() * (1.0 + i / 128.0)).to(torch.bfloat16) if i else v for k, v in base.items()}
            for i in range(NSETS)]
    am = [{k: torch.empty(1, device=dev) for k in base} for _ in range(NSETS)]
    for i in range(NSETS):
        for k in base:
            ue.amax_accumulate(sets[i][k], am[i][k], clear=True)
    R, C = base["x"].shape
    W = base["w"].shape[0]
    u8 = lambda *sh: torch.empty(sh, dtype=torch.uint8, device=dev)
    outs = [{"x": (u8(R, C // 2), u8(R, C // 16)), "dy": (u8(R, C // 2), u8(R, C // 16)),
             "w": (u8(W, W // 2), u8(W // 16, W // 16))} for _ in range(NSETS)]
    dec = torch.empty(1, device=dev)
    fns = {"activation_rows_rn": (lambda i: ue.quantize_1d(sets[i]["x"], 1, am[i]["x"], 448.0, "rn", 0, 0,
                                                          *outs[i]["x"], dec), quant_bytes_1d(R, C)),
           "gradient_rows_sr": (lambda i: ue.quantize_1d(sets[i]["dy"], 1, am[i]["dy"], 448.0, "sr", 1, 0,
                                                         *outs[i]["dy"], dec), quant_bytes_1d(R, C)),
           "weight_tiles_rn": (lambda i: ue.quantize_2d(sets[i]["w"], am[i]["w"], 448.0, "rn", 0, 0, False,
                                                        outs[i]["w"][0], outs[i]["w"][1], None, dec),
                               quant_bytes_2d(W, W, False))}
    res = {}
    for name, (fn, nb) in fns.items():
        med, mean, pct = _time_kernel(fn, NSETS)
        gbs = nb / (med * 1e-3) / 1e9
        res[name] = {"us": round(med * 1e3, 2), "GB/s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
                     "us_mean": round(mean * 1e3, 2)}
    return res


def small_linear_latency(dev):
    """The single small linear (X [256, 512] with 1% x50 outliers, W [256,
    512]; X rows RN, W 16 x 16 tiles RN, NT GEMM to fp32): device time per
    launch of each kernel and of the whole forward, HIP events."""
    import torch
    import paper_2609_02846_amd as ue
    import synthetic
    wl = synthetic.linear_fprop_small(0)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    x, w = up(wl["x"]), up(wl["w"])
    ax, aw = torch.empty(1, device=dev), torch.empty(1, device=dev)
    u8 = lambda *sh: torch.empty(sh, dtype=torch.uint8, device=dev)
    xo = (u8(256, 256), u8(256, 32), torch.empty(1, device=dev))
    wo = (u8(256, 256), u8(16, 32))
    wd = torch.empty(1, device=dev)
    y = torch.empty(256, 256, device=dev)

    def fwd(_i=0):
        ue.amax_accumulate(x, ax, clear=True)
        ue.amax_accumulate(w, aw, clear=True)
        ue.quantize_1d(x, 1, ax, 448.0, "rn", 0, 0, *xo)
        ue.quantize_2d(w, aw, 448.0, "rn", 0, 0, False, wo[0], wo[1], None, wd)
        ue.gemm("nt", 256, 256, 512, *xo, wo[0], wo[1], wd, out=y)
    parts = {"amax_x_and_w": lambda i: (ue.amax_accumulate(x, ax, clear=True), ue.amax_accumulate(w, aw, clear=True)),
             "quant_x_rows": lambda i: ue.quantize_1d(x, 1, ax, 448.0, "rn", 0, 0, *xo),
             "quant_w_tiles": lambda i: ue.quantize_2d(w, aw, 448.0, "rn", 0, 0, False, wo[0], wo[1], None, wd),
             "gemm_nt": lambda i: ue.gemm("nt", 256, 256, 512, *xo, wo[0], wo[1], wd, out=y),
             "forward_total": fwd}
    res = {}
    for name, fn in parts.items():
        med, mean, _ = _time_kernel(fn, 1, reps=200, warm=20)
        res[name + "_us"] = round(med * 1e3, 2)
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU (got --gpus {args.gpus}): the step has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    if args.control:
        control_bench(args)
        return
    if args.formats:
        formats_bench(args)
        return
    if args.drift:
        drift_bench(args)
        return
    T, K, N = args.tokens, args.k, args.n
    want_cpu = (not args.no_cpu_baseline and args.pm is None and not args.rht and args.kernel is None
                and not (args.copy_ref or args.matmul_ref or args.gemm_shapes))
    # the oracle leg first: its worker pool forks this process before any GPU use
    cpu = cpu_baseline(T, K, N) if want_cpu else None
    import torch
    import paper_2609_02846_amd as ue
    import synthetic

    dev = torch.device("cuda:0")
    if args.copy_ref:
        src = torch.empty(args.copy_ref // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"copied {args.copy_ref} bytes 5 times", flush=True)
        return
    if args.matmul_ref:
        print(json.dumps({"matmul_ref_bf16": matmul_ref(T, K, N, dev)}), flush=True)
        return
    if args.gemm_shapes:
        gemm_shapes(dev)
        return
    wl = synthetic.ffn_step(0, T, K, N)

    def up(bits):
        return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)
    # input sets: set 0 is the seeded workload; sets 1.. are it scaled by
    # 1 + i/128 (bf16), same distributions, so that no step reads inputs the
    # previous step left in the 256 MB Infinity Cache
    base = (up(wl["x"]), up(wl["w"]), up(wl["dy"]))
    ins = [base] + [tuple((t.float() * (1.0 + i / 128.0)).to(torch.bfloat16) for t in base)
                    for i in range(1, NSETS)]
    del wl
    u8 = lambda *s: torch.empty(s, dtype=torch.uint8, device=dev)
    f32 = lambda *s: torch.empty(s, dtype=torch.float32, device=dev)
    sets = []
    for i in range(NSETS):
        sets.append({
            "xr": (u8(T, K // 2), u8(T, K // 16), f32(1)),
            "xc": (u8(K, T // 2), u8(K, T // 16), f32(1)),
            "w": (u8(N, K // 2), u8(N // 16, K // 16), u8(K, N // 2), f32(1), u8(K // 16, N // 16)),
            "dr": (u8(T, N // 2), u8(T, N // 16), f32(1)),
            "dc": (u8(N, T // 2), u8(N, T // 16), f32(1)),
            "y": torch.empty(T, N, dtype=torch.bfloat16, device=dev),
            "dx": torch.empty(T, K, dtype=torch.bfloat16, device=dev),
            "dw": torch.empty(N, K, dtype=torch.float32, device=dev)})
    # one sample-and-hold state per operand role, as in training: a refresh
    # measures the current set's tensor (the sets differ by at most 2.3%)
    roles = {n: ue.AmaxState(args.period) for n in ("x", "w", "d", "xt", "dt")}
    st = [roles] * NSETS

    names = ["amax", "quant_x_dual", "quant_w_tiles", "quant_dy_rows", "quant_dy_cols", "gemm_fprop",
             "gemm_dgrad", "gemm_wgrad"]
    MASK = 0x3C5A

    if args.pm is None:
        G = ue.gemm
    else:
        def G(*a, **kw):
            return ue.gemm_pm(*a, grid=args.pm, **kw)

    def kernel_fns(i, seed):
        x, w, dy = ins[i]
        b, s = sets[i], st[i]
        xc_dec = b["xc"][2] if args.rht else b["xr"][2]     # one-read X quantizer: one decode factor
        pw, sw_, pwt, dw_, swt = b["w"]

        def quant_x():
            if args.rht:
                ue.quantize_1d(x, 1, s["x"].amax, 448.0, "rn", 0, 0, *b["xr"])
                ue.quantize_cols_rht(x, s["xt"].amax, MASK, 448.0, "rn", 0, 0, *b["xc"])
            else:
                ue.quantize_dual(x, s["x"].amax, 448.0, "rn", 0, 0, 0, b["xr"][:2], b["xc"][:2], b["xr"][2])

        def quant_dy_cols():
            if args.rht:
                ue.quantize_cols_rht(dy, s["dt"].amax, MASK, 448.0, "sr", seed, 2, *b["dc"])
            else:
                ue.quantize_1d(dy, 0, s["d"].amax, 448.0, "sr", seed, 2, *b["dc"])
        xr, xc, dr, dc = b["xr"], b["xc"], b["dr"], b["dc"]
        return {
            "quant_x_dual": quant_x,
            "quant_w_tiles": lambda: ue.quantize_2d(w, s["w"].amax, 448.0, "rn", 0, 0, True, pw, sw_, pwt, dw_, swt),
            "quant_dy_rows": lambda: ue.quantize_1d(dy, 1, s["d"].amax, 448.0, "sr", seed, 1, *dr),
            "quant_dy_cols": quant_dy_cols,
            "gemm_fprop": lambda: G("nt", T, N, K, xr[0], xr[1], xr[2], pw, sw_, dw_, out=b["y"]),
            "gemm_dgrad": lambda: G("nn", T, K, N, dr[0], dr[1], dr[2], pwt, swt, dw_, out=b["dx"]),
            "gemm_wgrad": lambda: G("tn", N, K, T, dc[0], dc[1], dc[2], xc[0], xc[1], xc_dec, out=b["dw"]),
        }

    def sample(i, t):
        """The step's sample-and-hold calls; returns how many refreshed."""
        x, w, dy = ins[i]
        s = st[i]
        n = int(ue.amax_sample(s["x"], x, t)) + int(ue.amax_sample(s["w"], w, t)) + int(ue.amax_sample(s["d"], dy, t))
        if args.rht:
            n += int(ue.amax_sample_rht(s["xt"], x, MASK, t)) + int(ue.amax_sample_rht(s["dt"], dy, MASK, t))
        return n

    def step(t, ev=None):
        i = t % NSETS
        if ev is not None:
            ev[0].record()
        refreshed = sample(i, t)
        fns = kernel_fns(i, 1000 + t)
        for j, n in enumerate(names[1:]):
            if ev is not None:
                ev[j + 1].record()
            fns[n]()
        if ev is not None:
            ev[len(names)].record()
        return refreshed

    # warm-up: the first NSETS steps refresh every set's references
    for t in range(max(args.warmup, NSETS)):
        step(t)
    torch.cuda.synchronize()
    if args.kernel is not None:
        for r in range(args.steps):
            kernel_fns(r % NSETS, 7)[args.kernel]()
        torch.cuda.synchronize()
        print(f"ran {args.kernel} {args.steps} times", flush=True)
        return
    # --- refresh-step amax, timed alone (three tensor amax launches) ---------
    def refresh_all(i):
        x, w, dy = ins[i]
        for s_, tns in ((roles["x"], x), (roles["w"], w), (roles["d"], dy)):
            ue.amax_accumulate(tns, s_.amax, clear=True)
        if args.rht:
            # the transformed operands' amax passes
            for key, tns in (("xt", x), ("dt", dy)):
                s_ = roles[key]
                s_.reset()
                ue.amax_sample_rht(s_, tns, MASK, 0)
    refresh_ms, _, _ = _time_kernel(refresh_all, NSETS, reps=20, warm=2)
    for key in roles:               # the warm-up schedule again, from empty caches
        roles[key].reset()
    t0 = max(args.warmup, NSETS)
    for t in range(t0):
        step(t)
    torch.cuda.synchronize()
    # --- timed region: exactly `steps` steps, per-kernel events inside -------
    evs = [_events(len(names) + 1) for _ in range(args.steps)]
    start, stop = _events(2)
    torch.cuda.synchronize()
    start.record()
    refreshed = []
    for r in range(args.steps):
        refreshed.append(step(t0 + r, evs[r]) > 0)
    stop.record()
    torch.cuda.synchronize()
    window_ms = start.elapsed_time(stop)
    n_refresh = int(sum(refreshed))
    per = {n: [] for n in names}
    for ev in evs:
        for j, n in enumerate(names):
            per[n].append(ev[j].elapsed_time(ev[j + 1]))
    # the refresh-step amax at its 1/D rate: the window's own refresh-step
    # amax time is replaced by the timed refresh cost once every D steps
    refresh_in_window = sum(v for v, f in zip(per["amax"], refreshed) if f)
    D = max(args.period, 1)
    ms = (window_ms - refresh_in_window + refresh_ms * args.steps / D) / args.steps
    avg = {n: float(np.mean(v)) for n, v in per.items()}
    pct = {n: [round(float(q), 5) for q in np.percentile(v, [10, 50, 90])] for n, v in per.items()}

    flop_gemm = 2.0 * T * N * K
    qbytes = {"quant_x_dual": 2 * quant_bytes_1d(T, K) if args.rht else quant_bytes_dual(T, K),
              "quant_w_tiles": quant_bytes_2d(N, K, True),
              "quant_dy_rows": quant_bytes_1d(T, N), "quant_dy_cols": quant_bytes_1d(T, N)}
    kernels = {}
    for n, b in qbytes.items():
        gbs = b / (avg[n] * 1e-3) / 1e9
        kernels[n] = {"ms": round(avg[n], 5), "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
                      "ms_p10_p50_p90": pct[n], "alg_bytes": b}
    for n in ["gemm_fprop", "gemm_dgrad", "gemm_wgrad"]:
        tf = flop_gemm / (avg[n] * 1e-3) / 1e12
        kernels[n] = {"ms": round(avg[n], 5), "TFLOP/s": round(tf, 1), "frac": round(tf / BF16_PEAK_TFLOPS, 4),
                      "ms_p10_p50_p90": pct[n]}
    amax_bytes = 2 * (T * K + N * K + T * N)
    kernels["amax_refresh"] = {"ms": round(refresh_ms, 5), "GB/s": round(amax_bytes / (refresh_ms * 1e-3) / 1e9, 1),
                               "per_step_share_ms": round(refresh_ms / D, 5),
                               "note": f"X, W and dY amax, launched on 1 step in {D}"}
    # SR quantizers are bound by VALU issue: instructions per element (rocprofv3
    # SQ_INSTS_VALU, stored with the source hash) against 1024 SIMDs issuing
    # one wave64 instruction per 4 cycles at 2.4 GHz
    if os.path.exists(args.valu):
        try:
            vj = json.load(open(args.valu))
            if vj.get("source_sha256_16") == quantize_source_hash() and vj.get("config") == [T, K, N]:
                for n, ipe in vj["instr_per_element"].items():
                    if n in kernels:
                        el = T * N if n.startswith("quant_dy") else (T * K if n == "quant_x_dual" else N * K)
                        frac = ipe * el * 4 / 64 / (1024 * 2.4e9 * avg[n] * 1e-3)
                        kernels[n]["valu_instr_per_element"] = ipe
                        kernels[n]["valu_frac"] = round(frac, 4)
        except Exception:
            pass
    iso = {}
    for n in (qbytes if not args.step_only else []):
        # each quantizer alone over the rotating sets (no input of the
        # previous launch in the Infinity Cache)
        med, mean, p = _time_kernel(lambda i, n=n: kernel_fns(i, 7)[n](), NSETS, reps=20, warm=4)
        gbs = qbytes[n] / (med * 1e-3) / 1e9
        iso[n] = {"ms": round(med, 5), "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
    qtime = sum(avg[n] for n in qbytes)
    quant_gbs = sum(qbytes.values()) / (qtime * 1e-3) / 1e9
    gtime = sum(avg[n] for n in ["gemm_fprop", "gemm_dgrad", "gemm_wgrad"])
    gemm_tf = 3 * flop_gemm / (gtime * 1e-3) / 1e12

    dom = "gemm_fprop"
    traffic = None
    if os.path.exists(args.traffic):
        # HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE (scaled by a
        # plain copy of known size); void once the kernel source has changed.
        try:
            tr = json.load(open(args.traffic))
            fresh = gemm_source_hash() == tr.get("source_sha256_16")
            if fresh and tr.get("kernel") == dom and tr.get("config") == [T, K, N]:
                traffic = round(float(tr["bytes_per_launch"]))
        except Exception:
            traffic = None
    achieved = flop_gemm / (avg[dom] * 1e-3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": traffic,
                "peak_note": "dense fp16 MFMA (the bf16 peak), the instruction the GEMM issues"}
    if args.pm is not None:
        # probe-matched GEMM: bound by the per-output VALU work of each
        # 64-product group (4 widenings, 3 binary64 adds, 1 narrowing, 1
        # toward-zero add), against 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
        groups = T * N * ((K + 63) // 64)
        ach = PM_VALU_MEASURED * groups / (avg[dom] * 1e-3) / 1e12
        roofline = {"bound": "alu", "kernel": dom + " (probe-matched)", "achieved": round(ach, 2),
                    "peak": VALU_PEAK_TOPS, "unit": "Tops/s (VALU lane ops)",
                    "frac": round(ach / VALU_PEAK_TOPS, 4), "traffic": None,
                    "ops_per_output_group": {"issued": PM_VALU_MEASURED, "output_model": PM_VALU_PER_GROUP},
                    "model_only_frac": round(PM_VALU_PER_GROUP * groups / (avg[dom] * 1e-3) / 1e12 / VALU_PEAK_TOPS, 4)}

    value = 3 * flop_gemm / (ms * 1e-3) / 1e12
    out = {"metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp16",
           "operands": ("E2M1 payloads x UE5M3 block scales, decoded exactly to fp16 for the matrix "
                        "cores; fp32 accumulation"),
           "data": "synthetic",
           "config": {"workload": f"FFN up-projection linear training step T={T} K={K} N={N}",
                      "tokens": T, "k": K, "n": N, "refresh_period": args.period,
                      "target": 448.0, "wgrad_operand_rht": bool(args.rht), "input_sets": NSETS,
                      "gemm": ("decoded-operand, fp32 accumulation" if args.pm is None else
                               f"probe-matched, grid 1/{args.pm}" if args.pm else "probe-matched, no snap")},
           "window_ms_per_step": round(window_ms / args.steps, 4), "refresh_steps_in_window": n_refresh,
           "quantize_GBps": round(quant_gbs, 1), "quantize_frac_hbm": round(quant_gbs / HBM_PEAK_GBS, 4),
           "gemm_TFLOPs": round(gemm_tf, 1), "gemm_frac_bf16": round(gemm_tf / BF16_PEAK_TFLOPS, 4),
           "kernels": kernels, "quantizers_isolated": iso, "roofline": roofline}
    if args.pm is None and not args.rht and not args.step_only:
        out["quantizer_workload"] = quantizer_workload(dev)
        out["small_linear"] = small_linear_latency(dev)
        # measured ceilings on this GPU (references only, not the product
        # path): a plain device copy for the quantizers, a bf16 library GEMM
        # of the same shapes for the FP4 GEMMs
        cp = copy_ceiling(dev)
        mm = matmul_ref(T, K, N, dev, verbose=False)
        for n in qbytes:
            kernels[n]["frac_copy"] = round(kernels[n]["GB/s"] / cp["GB/s"], 4)
        for n in ["gemm_fprop", "gemm_dgrad", "gemm_wgrad"]:
            kernels[n]["frac_matmul_ref"] = round(kernels[n]["TFLOP/s"] / mm[n[5:]]["TFLOP/s"], 4)
        out["ceilings"] = {"device_copy": cp, "bf16_matmul": mm}
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
