"""Host-side argument checks of the FP4 Linear layer (no GPU: the layer is
built on the CPU and never run)."""

import pytest

from paper_2609_02846_amd.linear import Linear


def test_block_size_and_shape_checks():
    assert Linear(64, 96, device="cpu", block=32).block == 32
    assert Linear(48, 80, device="cpu").block == 16
    with pytest.raises(ValueError):
        Linear(48, 64, device="cpu", block=32)            # 48 is not a multiple of 32
    with pytest.raises(ValueError):
        Linear(64, 64, device="cpu", block=8)
    with pytest.raises(ValueError):
        Linear(64, 64, device="cpu", block=32, rht_wgrad=True)
    with pytest.raises(ValueError):
        Linear(40, 64, device="cpu")
    with pytest.raises(ValueError):
        Linear(64, 64, device="cpu", grad_rounding="stochastic")
