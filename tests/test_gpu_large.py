"""Maximum-size cases: 64-bit offsets and counters.

* GEMM with an A payload beyond 2^31 bytes (the persistent kernel's buffer
  resources cover 2^31 bytes, so the general kernel runs): sampled rows on
  both sides of the 2 GiB offset against the oracle.
* amax and the row, column (SR: Philox counters past 2^31) and tile
  quantizers on a bf16 tensor of more than 2^31 elements, with a planted
  maximum past element 2^31; sampled rows, columns and the last tile row
  bit-exact against the oracle.
Inputs are seeded device-side fills (payload bytes, scale codes, uniform
values); expected values come from the oracle on copies of the sampled
parts."""

import numpy as np
import pytest
import torch

from oracle import gemm as ogemm
from oracle import quantize as oq
import paper_2609_02846_amd as ue
from tests.gpu_util import f32_scalar_dev, gemm_check, host, row_elem_index, say

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def test_gemm_operand_beyond_2gib():
    M, N, K = (1 << 20) + 128, 256, 4096           # A payload 2,147,745,792 bytes
    say("gemm A payload > 2 GiB", M, N, K)
    g = torch.Generator(device="cuda").manual_seed(5)
    a = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device="cuda", generator=g)
    sa = torch.randint(0x68, 0x88, (M, K // 16), dtype=torch.uint8, device="cuda", generator=g)
    b = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device="cuda", generator=g)
    sb = torch.randint(0x68, 0x88, (N // 16, K // 16), dtype=torch.uint8, device="cuda", generator=g)
    one = f32_scalar_dev(1.0)
    c = ue.gemm("nt", M, N, K, a, sa, one, b, sb, one)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 777, M // 2, (1 << 20) - 1, 1 << 20, (1 << 20) + 1, (1 << 20) + 64, M - 2, M - 1])
    ridx = torch.from_numpy(rows).cuda()
    A = oq.decoded_1d(host(a[ridx]), host(sa[ridx]), 1)
    B = oq.decoded_2d(host(b), host(sb))
    al = ogemm.alpha(1.0, 1.0)
    gemm_check(host(c[ridx]), ogemm.fprop(A, B, al), al, ogemm.abs_product(A, B), K, "A > 2 GiB")
    del a, sa, c


def test_quantizers_beyond_2g_elements():
    R, C = (1 << 19) + 16, 4096                    # 2,147,549,184 elements
    say("quantizers on", R, "x", C)
    g = torch.Generator(device="cuda").manual_seed(6)
    x = torch.empty(R, C, dtype=torch.bfloat16, device="cuda")
    for r0 in range(0, R, 1 << 16):                # fill in chunks (bounded fp32 temporary)
        r1 = min(R, r0 + (1 << 16))
        x[r0:r1] = (torch.rand(r1 - r0, C, generator=g, device="cuda") * 2 - 1).to(torch.bfloat16)
    x[R - 1, C - 3] = 7.5                          # element index > 2^31
    st = ue.AmaxState(1)
    ue.amax_sample(st, x, 0)
    torch.cuda.synchronize()
    assert st.amax.item() == 7.5
    G = np.float32(7.5)

    say("rows RN beyond 2^31")
    p, s, d = ue.quantize_1d(x, 1, st.amax, 448.0, "rn")
    torch.cuda.synchronize()
    rows = np.array([0, 3, R // 2, (1 << 19) - 1, 1 << 19, R - 1])
    xr = _bits(x[torch.from_numpy(rows).cuda()])
    rp, rs, rd = oq.quantize_1d(xr, 1, G, 448.0, "rn")
    assert np.array_equal(host(p[torch.from_numpy(rows).cuda()]), rp)
    assert np.array_equal(host(s[torch.from_numpy(rows).cuda()]), rs)
    assert np.float32(d.item()) == rd
    del p, s

    say("columns SR beyond 2^31 (64-bit Philox counters)")
    pc, sc, _ = ue.quantize_1d(x, 0, st.amax, 448.0, "sr", 3, 4)
    torch.cuda.synchronize()
    cols = np.array([0, 1, C // 2, C - 3, C - 1])
    sub = _bits(x[:, torch.from_numpy(cols).cuda()])
    idx = row_elem_index(np.arange(R), C, cols)
    cp_, cs_, _ = oq.quantize_1d(sub, 0, G, 448.0, "sr", 3, 4, elem_index=idx)
    assert np.array_equal(host(pc[torch.from_numpy(cols).cuda()]), cp_)
    assert np.array_equal(host(sc[torch.from_numpy(cols).cuda()]), cs_)
    del pc, sc

    say("tiles RN, last tile row beyond 2^31")
    pw, sw, pwt, _, swt = ue.quantize_2d(x, st.amax, 448.0, "rn")
    torch.cuda.synchronize()
    last = _bits(x[R - 16:])
    tp, ts, tpt, _ = oq.quantize_2d(last, G, 448.0, "rn")
    assert np.array_equal(host(pw[R - 16:]), tp)
    assert np.array_equal(host(sw[R // 16 - 1]), ts[0])
    assert np.array_equal(host(pwt[:, (R - 16) // 2:]), tpt)
    assert np.array_equal(host(swt[:, R // 16 - 1]), ts[0])
