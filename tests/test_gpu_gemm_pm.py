"""GPU parity of the probe-matched GEMM (ue5m3_gemm_pm) with the oracle's
exact output model (oracle.accumulate: eq:issue-partial, eq:issue-rz,
eq:final-grid, eq:grid-denominator).  The model is a deterministic function
of the decoded operands, so the bar is equality of every compared output
(binary32 value; -0 and +0 compare equal).  Operands come from the oracle's
quantizers, from raw codes built to force the wide-span path, or (full
size) from the GPU quantizers with the expected values from the oracle's
quantization of the sampled rows."""

import numpy as np
import pytest
import torch

import synthetic
from oracle import accumulate as oacc
from oracle import gemm as ogemm
from oracle import quantize as oq
from oracle import scaling as osc
import paper_2609_02846_amd as ue
from tests.gpu_util import (f32_scalar_dev, host, oracle_cols, oracle_rows, say, to_dev,
                            u8_to_dev)

pytestmark = pytest.mark.gpu


def _ref(A, B, al, d, idx):
    """Oracle outputs at the (m, n) pairs of idx."""
    return np.array([oacc.dot(A[m] * B[n], d, al)[0] for m, n in idx], np.float32)


def _sample(M, N, n, seed, tile=128):
    """Tile corners and edges plus random positions."""
    rng = np.random.default_rng(seed)
    ms = sorted({0, M - 1, *[v for t in range(0, M, tile) for v in (t, min(t + tile, M) - 1)]})
    ns = sorted({0, N - 1, *[v for t in range(0, N, tile) for v in (t, min(t + tile, N) - 1)]})
    idx = {(m, q) for m in ms for q in ns}
    idx |= {(int(rng.integers(M)), int(rng.integers(N))) for _ in range(n)}
    return sorted(idx)


def _check(c, A, B, al, d, idx, what, bf16=False):
    got = host(c.float()) if bf16 else host(c)
    ref = _ref(A, B, al, d, idx)
    if bf16:
        ref = torch.from_numpy(ref).to(torch.bfloat16).float().numpy()
    g = np.array([got[m, n] for m, n in idx], np.float32)
    bad = np.nonzero(g != ref)[0]
    assert bad.size == 0, (f"{what}: {bad.size}/{len(idx)} outputs differ, first {idx[bad[0]]}: "
                           f"{g[bad[0]]!r} vs {ref[bad[0]]!r}")


def _operands(seed, T, K, N, fmt="ue5m3"):
    x = synthetic.activation(seed, T, K, 1e-2, 50.0)
    w = synthetic.weight(seed, N, K)
    dy = synthetic.gradient(seed, T, N, 1e-3, 1.0)
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    return dict(xr=oq.quantize_1d(x, 1, gx, fmt=fmt), xc=oq.quantize_1d(x, 0, gx, fmt=fmt),
                wq=oq.quantize_2d(w, gw, fmt=fmt),
                dr=oq.quantize_1d(dy, 1, gd, 448.0, "sr", 3, 1, fmt=fmt),
                dc=oq.quantize_1d(dy, 0, gd, 448.0, "sr", 3, 2, fmt=fmt))


def _run_layouts(T, K, N, seed, grids, n_samples, fmt="ue5m3"):
    op = _operands(seed, T, K, N, fmt)
    xr, xc, wq, dr, dc = op["xr"], op["xc"], op["wq"], op["dr"], op["dc"]
    D, U = f32_scalar_dev, u8_to_dev
    X = oq.decoded_1d(xr[0], xr[1], 1, fmt)
    W = oq.decoded_2d(wq[0], wq[1], fmt)
    dY = oq.decoded_1d(dr[0], dr[1], 1, fmt)
    dYc, Xc = oq.decoded_1d(dc[0], dc[1], 0, fmt), oq.decoded_1d(xc[0], xc[1], 0, fmt)
    cases = [
        ("nt", T, N, K, (U(xr[0]), U(xr[1]), D(xr[2]), U(wq[0]), U(wq[1]), D(wq[3])), X, W,
         ogemm.alpha(xr[2], wq[3])),
        ("nn", T, K, N, (U(dr[0]), U(dr[1]), D(dr[2]), U(wq[2]), U(np.ascontiguousarray(wq[1].T)), D(wq[3])),
         dY, np.ascontiguousarray(W.T), ogemm.alpha(dr[2], wq[3])),
        ("tn", N, K, T, (U(dc[0]), U(dc[1]), D(dc[2]), U(xc[0]), U(xc[1]), D(xc[2])),
         np.ascontiguousarray(dYc.T), np.ascontiguousarray(Xc.T), ogemm.alpha(dc[2], xc[2])),
    ]
    for lay, M_, N_, K_, args, A, B, al in cases:
        idx = _sample(M_, N_, n_samples, seed)
        for d in grids:
            say("gemm_pm", fmt, lay, M_, N_, K_, "grid", d)
            c = ue.gemm_pm(lay, M_, N_, K_, *args, grid=d, fmt=fmt)
            torch.cuda.synchronize()
            _check(c, A, B, al, d, idx, f"{fmt} {lay} {M_}x{N_}x{K_} d={d}")
        if lay == "nt":
            c = ue.gemm_pm(lay, M_, N_, K_, *args, grid=1024, out_dtype=torch.bfloat16, fmt=fmt)
            torch.cuda.synchronize()
            _check(c, A, B, al, 1024, idx, f"{fmt} {lay} bf16", bf16=True)


def test_pm_three_layouts_ragged_tiles():
    """Several 128x128 tiles with 16-row/column tails and K with a partial
    last group (336 = 5 x 64 + 16, 144 = 2 x 64 + 16, 272 = 4 x 64 + 16)."""
    _run_layouts(272, 336, 144, 0, (1024, 0, 256), 700)


def test_pm_small_every_output():
    """Every output of a one-tile case, four grids."""
    T, K, N = 48, 208, 48
    op = _operands(5, T, K, N)
    xr, wq = op["xr"], op["wq"]
    X, W = oq.decoded_1d(xr[0], xr[1], 1), oq.decoded_2d(wq[0], wq[1])
    al = ogemm.alpha(xr[2], wq[3])
    idx = [(m, n) for m in range(T) for n in range(N)]
    for d in (0, 256, 1024, 4096):
        say("gemm_pm small every output grid", d)
        c = ue.gemm_pm("nt", T, N, K, u8_to_dev(xr[0]), u8_to_dev(xr[1]), f32_scalar_dev(xr[2]),
                       u8_to_dev(wq[0]), u8_to_dev(wq[1]), f32_scalar_dev(wq[3]), grid=d)
        torch.cuda.synchronize()
        _check(c, X, W, al, d, idx, f"small d={d}")


def test_pm_e4m3_operands():
    _run_layouts(144, 208, 160, 2, (1024,), 300, fmt="e4m3")


def test_pm_wide_span_groups():
    """Raw scale codes far apart inside 64-k groups (2^-14 next to 2^15 and
    subnormal codes) force the exact 128-bit path for some groups, while
    other groups of the same launch stay on the binary64 path."""
    M, N, K = 96, 64, 320
    rng = np.random.default_rng(11)
    pay_a = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    pay_b = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    wide = np.array([0x08, 0xF0, 0x03, 0x77], np.uint8)            # L = -17, 12, -17, -3
    narrow = rng.integers(0x70, 0x80, (M, K // 16), dtype=np.uint8)
    sa = narrow.copy()
    sa[:, 4:8] = wide[None, :]                                      # group 1 wide for every row
    sa[::3, 12:16] = rng.choice(wide, (len(range(0, M, 3)), 4))     # group 3 wide for some rows
    sb = rng.integers(0x60, 0x90, (N // 16, K // 16), dtype=np.uint8)
    sb[:, 8:12] = np.array([0xE8, 0x10, 0x02, 0xB0], np.uint8)      # group 2 wide on B
    sb[::2, 4:8] = wide[None, :]     # group 1 wide on both: block sums span ~80 bits
    A = oq.decoded_1d(pay_a, sa, 1)
    B = oq.decoded_2d(pay_b, sb)
    al = np.float32(0.75)
    idx = [(m, n) for m in range(M) for n in range(N)]
    for d in (0, 1024):
        say("gemm_pm wide span grid", d)
        c = ue.gemm_pm("nt", M, N, K, u8_to_dev(pay_a), u8_to_dev(sa), f32_scalar_dev(1.0),
                       u8_to_dev(pay_b), u8_to_dev(sb), f32_scalar_dev(0.75), grid=d)
        torch.cuda.synchronize()
        _check(c, A, B, al, d, idx, f"wide span d={d}")


def _pair_bound_operands(M, N, K, span_a, span_b, seed):
    """Raw operands whose groups put the block pairs (0, 1) and (2, 3) at the
    edge of exact binary32 addition: blocks 0, 2, 3 at the largest block sum
    (every nibble 6, scale integer 15: 518400 x 2^E), block 1 of odd products (nibbles
    0.5, 1.5 and 6 with both signs) with its scale exponent span_a lower on
    A and span_b lower on B, so that block 1's sums sit 2^(span_a + span_b)
    below block 0's; blocks 2 and 3 at block 0's exponent, so that adding
    the two pair sums usually rounds.  Every fourth A row and every second
    B tile keep all four exponents equal (span 0), so the group's span is a
    maximum over rows."""
    rng = np.random.default_rng(seed)
    nb = K // 16

    def payload(rows):
        big = np.full((rows, nb, 16), 0x7, np.uint8)
        odd = rng.choice(np.array([0x1, 0x3, 0x7, 0x9, 0xB, 0xF], np.uint8), (rows, nb, 16))
        nib = np.where((np.arange(nb) % 4 == 1)[None, :, None], odd, big)
        nib = nib.reshape(rows, K)
        return (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)

    def codes(rows, e_top, span, flat_every):
        e = np.full((rows, nb), e_top, np.int64)
        e[:, 1::4] = e_top - span
        e[::flat_every, :] = e_top
        return ((e << 3) | 7).astype(np.uint8)

    return payload(M), codes(M, 12, span_a, 4), payload(N), codes(N // 16, 10, span_b, 2)


@pytest.mark.parametrize("K", [128, 144])
def test_pm_pair_path_at_its_bound(K):
    """Spans adding up to 4 take the binary32 pair path (its bound: block
    sums up to 518400 x 2^E, pairs 2^4 apart), 5 the binary64 path; every
    output of each launch against the oracle, with and without the snap.
    K = 144 has a partial last group (the per-block span check)."""
    M, N = 64, 64
    for span_a, span_b in ((3, 1), (4, 0), (0, 4), (2, 2), (3, 2), (5, 0)):
        pay_a, sa, pay_b, sb = _pair_bound_operands(M, N, K, span_a, span_b, 10 * span_a + span_b)
        A = oq.decoded_1d(pay_a, sa, 1)
        B = oq.decoded_2d(pay_b, sb)
        idx = [(m, n) for m in range(M) for n in range(N)]
        for d in (0, 1024):
            say("gemm_pm pair bound", K, span_a, span_b, "grid", d)
            c = ue.gemm_pm("nt", M, N, K, u8_to_dev(pay_a), u8_to_dev(sa), f32_scalar_dev(1.0),
                           u8_to_dev(pay_b), u8_to_dev(sb), f32_scalar_dev(1.0), grid=d)
            torch.cuda.synchronize()
            _check(c, A, B, np.float32(1.0), d, idx, f"pair bound K={K} spans {span_a}+{span_b} d={d}")


def test_pm_tie_broken_by_tiny_block():
    """One group whose block sums are 2^24, 1 and +-2^-30: the exact sum sits
    2^-30 off the binary32 tie 2^24 + 1, so RNE gives 2^24 + 2 (or 2^24);
    a binary64 sum would drop the 2^-30 and round the tie to even (2^24)
    either way.  Scale codes 2^12, 1, 2^-14 in one group take the exact
    path."""
    M, N, K = 32, 32, 64
    pay = np.zeros((M, K // 2), np.uint8)
    pay[:, 0] = 0x02                   # block 0, element 0: 1.0
    pay[:, 8] = 0x02                   # block 1, element 0: 1.0
    pay[:, 16] = 0x01                  # block 2, element 0: 0.5
    codes = np.array([0xD8, 0x78, 0x08, 0x78], np.uint8)           # 2^12, 1, 2^-14, 1
    sa = np.tile(codes, (M, 1))
    sb = np.tile(codes, (N // 16, 1))
    payb = pay.copy()
    payb[1::2, 16] = 0x09              # odd B rows: -0.5 in block 2
    A = oq.decoded_1d(pay, sa, 1)
    B = oq.decoded_2d(payb, sb)
    for n, want in [(0, 2.0 ** 24 + 2), (1, 2.0 ** 24)]:
        assert float(oacc.dot(A[0] * B[n], 0, 1.0)[0]) == want
    say("gemm_pm tie broken by a tiny block")
    c = ue.gemm_pm("nt", M, N, K, u8_to_dev(pay), u8_to_dev(sa), f32_scalar_dev(1.0),
                   u8_to_dev(payb), u8_to_dev(sb), f32_scalar_dev(1.0), grid=0)
    torch.cuda.synchronize()
    got = host(c)
    assert (got[:, 0::2] == 2.0 ** 24 + 2).all() and (got[:, 1::2] == 2.0 ** 24).all()


def test_pm_k_zero_and_empty():
    say("gemm_pm K=0")
    c = torch.full((8, 16), 7.0, device="cuda")
    one = f32_scalar_dev(1.0)
    dummy = torch.zeros(16, dtype=torch.uint8, device="cuda")
    ue.gemm_pm("nt", 8, 16, 0, dummy, dummy, one, dummy, dummy, one, out=c)
    torch.cuda.synchronize()
    assert (host(c) == 0).all()
    ue.gemm_pm("nt", 0, 16, 64, dummy, dummy, one, dummy, dummy, one, out=torch.empty(0, device="cuda"))


def test_pm_ffn_up_projection_sampled():
    """Nemotron-H-8B FFN up-projection (T=8192, K=4096, N=21504), GPU
    quantizers then the three probe-matched GEMMs, sampled outputs against
    the oracle's model on the oracle's quantization of those rows."""
    T, K, N = 8192, 4096, 21504
    say("gemm_pm ffn full size", T, K, N)
    wl = synthetic.ffn_step(0, T, K, N)
    x, w, dy = wl["x"], wl["w"], wl["dy"]
    xd, wd, dyd = to_dev(x), to_dev(w), to_dev(dy)
    sx, sw, sd = ue.AmaxState(50), ue.AmaxState(50), ue.AmaxState(50)
    for st, t in [(sx, xd), (sw, wd), (sd, dyd)]:
        ue.amax_sample(st, t, 0)
    (xr, xc) = ue.quantize_dual(xd, sx.amax)
    wq = ue.quantize_2d(wd, sw.amax)
    dr = ue.quantize_1d(dyd, 1, sd.amax, 448.0, "sr", 1, 1)
    dc = ue.quantize_1d(dyd, 0, sd.amax, 448.0, "sr", 1, 2)
    y = ue.gemm_pm("nt", T, N, K, *xr, wq[0], wq[1], wq[3], out_dtype=torch.bfloat16)
    dx = ue.gemm_pm("nn", T, K, N, *dr, wq[2], wq[4], wq[3], out_dtype=torch.bfloat16)
    dw = ue.gemm_pm("tn", N, K, T, *dc, xc[0], xc[1], xr[2])
    torch.cuda.synchronize()
    gx, gw, gd = osc.amax(x), osc.amax(w), osc.amax(dy)
    rng = np.random.default_rng(4)
    rows = np.sort(rng.choice(T, 6, replace=False))
    # fprop: sampled token rows x sampled weight rows (their 16-row tiles)
    xo = oracle_rows(x, rows, gx, 448.0, "rn", 0, 0)
    Xs = oq.decoded_1d(xo[0], xo[1], 1)
    wt = np.sort(rng.choice(N // 16, 2, replace=False))
    wrows = (wt[:, None] * 16 + np.arange(16)).ravel()
    Ws = np.concatenate([oq.decoded_2d(*oq.quantize_2d(w[16 * t:16 * t + 16], gw)[:2]) for t in wt])
    al = ogemm.alpha(xo[2], oq.quantize_2d(w[:16], gw)[3])
    idx = [(i, j) for i in range(len(rows)) for j in range(0, len(wrows), 5)]
    ref = torch.from_numpy(_ref(Xs, Ws, al, 1024, idx)).to(torch.bfloat16).float().numpy()
    got = host(y.float())
    g = np.array([got[rows[i], wrows[j]] for i, j in idx], np.float32)
    assert np.array_equal(g, ref), "fprop sampled"
    # wgrad: sampled dW rows (dY columns) x sampled columns (X columns)
    ncols = np.sort(rng.choice(N, 3, replace=False))
    kcols = np.sort(rng.choice(K, 3, replace=False))
    dco = oracle_cols(dy, ncols, gd, 448.0, "sr", 1, 2)
    xco = oracle_cols(x, kcols, gx, 448.0, "rn", 0, 0)
    A = np.ascontiguousarray(oq.decoded_1d(dco[0], dco[1], 0).T)      # [3, T]
    Bm = np.ascontiguousarray(oq.decoded_1d(xco[0], xco[1], 0).T)     # [3, T]
    al = ogemm.alpha(dco[2], xco[2])
    idx = [(i, j) for i in range(3) for j in range(3)]
    ref = _ref(A, Bm, al, 1024, idx)
    got = host(dw)
    g = np.array([got[ncols[i], kcols[j]] for i, j in idx], np.float32)
    assert np.array_equal(g, ref), "wgrad sampled"
    # dgrad: one sampled row against all of W's K columns would need all of
    # W decoded; check two output columns through their 16-column tiles
    kt = np.sort(rng.choice(K // 16, 1, replace=False))
    kc = (kt[:, None] * 16 + np.arange(16)).ravel()
    dro = oracle_rows(dy, rows[:2], gd, 448.0, "sr", 1, 1)
    dYs = oq.decoded_1d(dro[0], dro[1], 1)
    Wk = oq.decoded_2d(*oq.quantize_2d(np.ascontiguousarray(w[:, kc]), gw)[:2])     # [N, 16]
    al = ogemm.alpha(dro[2], oq.quantize_2d(w[:16], gw)[3])
    idx = [(i, j) for i in range(2) for j in (0, 9)]
    ref = torch.from_numpy(_ref(dYs, np.ascontiguousarray(Wk.T), al, 1024, idx)).to(torch.bfloat16).float().numpy()
    got = host(dx.float())
    g = np.array([got[rows[i], kc[j]] for i, j in idx], np.float32)
    assert np.array_equal(g, ref), "dgrad sampled"
