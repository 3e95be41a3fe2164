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
