"""CPU oracle of the UE5M3 FP4 quantize-and-GEMM step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library under ``paper_2609_02846_amd/csrc`` and never imports it.

The oracle is written from the paper "UE5M3 FP4 Block Scaling for Stable
Language Model Pretraining" (arXiv 2609.02846):

* ``formats``  -- E2M1 payload and UE5M3 block-scale codebooks (Sec. 2.1-2.2,
  Sec. 3, eq:ue5m3max, Table 2) and the E4M3 / E8M0 comparison formats
  (Table 1, Table 2).
* ``philox``   -- Philox4x32-10 (Salmon et al., SC'11), the counter-based
  stream that draws the stochastic-rounding words.
* ``scaling``  -- tensor amax, the periodic sample-and-hold refresh
  (eq:delayed-amax, Sec. 4.1) and the tensor multipliers (Sec. 4.2).
* ``quantize`` -- block quantizers (eq:microscaling, eq:scale-target,
  eq:sr, Table 5) and dequantization.
* ``gemm``     -- the decoded-operand GEMM model (Sec. 5.1) for the fprop,
  dgrad and wgrad products of Sec. 4.3.
* ``rht``      -- the 16-point randomized Hadamard transform of the wgrad
  operands (the "UE5M3 with Transformer Engine settings" recipe) and the
  quantizer on transformed values.
* ``accumulate`` -- the probe-matched output model (eq:issue-partial,
  eq:issue-rz, eq:final-grid, eq:grid-denominator): 64-product RNE
  partials, toward-zero cross-group adds, optional 1/d product-lattice snap.

Floating point: every decision that yields a code (block-scale byte, payload
nibble) is taken in IEEE binary32 with round-to-nearest-even, one rounding
per operation, in the order documented in ``quantize``; the paper gives real
formulas only, so the binary32 sequence is this implementation's reading.
GEMM references accumulate in float64.

Parity status: every function here is pinned by a CPU test (``tests/``)
except the binary32 operation order of the block quantizer, which the paper
does not fix ("parity unpinned" against the paper for that choice; the
worked blocks in ``tests/golden`` pin it against hand derivation).
"""

from . import formats, philox, scaling, quantize, gemm, accumulate, rht  # noqa: F401
