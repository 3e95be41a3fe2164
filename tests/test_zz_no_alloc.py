"""The allocation-free GEMM entry point (ue5m3_gemm_noalloc) against
ue5m3_gemm: same kernels and split plan, so the outputs must be equal bit
for bit.  Two calls in a row on shapes whose last wave of tiles is split
along K (so the partials go through the static scratch array), the second
smaller than the first, for each layout and both output types; the
reference calls run on the same stream before the allocation-free ones."""

import pytest
import torch

import paper_2609_02846_amd as ue
import synthetic
from tests.gpu_util import say, to_dev

pytestmark = pytest.mark.gpu

# 16 x 17 = 272 tiles on 256 CUs: the 16 tiles of the last wave are split
# along K, in 4 parts for K = 2048 and in 2 parts for K = 1024.
M, N = 4096, 4352


def _operands(layout, k, seed):
    """Quantized operands of one product of the given layout with
    contraction length k, as the recipe's quantizers produce them."""
    if layout == "tn":
        # wgrad: sources [k, M] and [k, N], blocked down their columns
        a_src = to_dev(synthetic.gradient(seed, k, M, 1e-5))
        b_src = to_dev(synthetic.activation(seed, k, N, 1e-3, 100.0))
    else:
        a_src = to_dev(synthetic.activation(seed, M, k, 1e-3, 100.0))
        b_src = to_dev(synthetic.weight(seed, N, k) if layout == "nt" else synthetic.weight(seed, k, N))
    aa, ab = torch.empty(1, device="cuda"), torch.empty(1, device="cuda")
    ue.amax_accumulate(a_src, aa, clear=True)
    ue.amax_accumulate(b_src, ab, clear=True)
    if layout == "tn":
        a = ue.quantize_1d(a_src, 0, aa, 448.0, "sr", seed, 2)
        b = ue.quantize_1d(b_src, 0, ab)
        return a, (b[0], b[1], b[2])
    a = ue.quantize_1d(a_src, 1, aa, 448.0, "sr" if layout == "nn" else "rn", seed, 1)
    wq = ue.quantize_2d(b_src, ab)
    if layout == "nt":
        return a, (wq[0], wq[1], wq[3])
    return a, (wq[2], wq[4], wq[3])


@pytest.mark.parametrize("layout", ["nt", "nn", "tn"])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_noalloc_equals_gemm_two_calls(layout, out_dtype):
    outs = {}
    for k in (2048, 1024):                    # the second call is the smaller one
        say("gemm_noalloc", layout, out_dtype, M, N, k)
        a, b = _operands(layout, k, 20 + k // 1024)
        ref = ue.gemm(layout, M, N, k, *a, *b, out_dtype=out_dtype)
        got = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
        ue.gemm_noalloc(layout, M, N, k, *a, *b, out=got)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), (layout, out_dtype, k)
        outs[k] = got
    assert not torch.equal(outs[2048][:16], outs[1024][:16])


def test_noalloc_checks_match_gemm():
    """Argument errors are the same as ue5m3_gemm's and are reported
    before anything is enqueued."""
    a, b = _operands("nt", 1024, 3)
    out = torch.empty(M, N, device="cuda")
    with pytest.raises(ue.UE5M3Error) as e:
        ue.gemm_noalloc("tn", M, N, 1024, *a, *b, out=out, a_blk="row", b_blk="tile")
    assert e.value.status == ue.UE5M3_ELAYOUT
    with pytest.raises(ValueError):
        ue.gemm_noalloc("nt", M, N, 1024, *a, *b, out=None)
