"""Oracle for the Scale-QLoRA frozen-code linear layer.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct CPU
statement of what the GPU library computes.  Only the test suite, the smoke
entry and the CPU-baseline leg of the benchmark may import it; the product
path (the HIP library and its Python binding) never does, and the two share
no code.

Arithmetic conventions
----------------------
* Contractions (forward, dX, the dW that feeds dS) are taken in float64 on the
  exact values of the bf16 inputs and of the dequantised weight.
* Steps the method defines on 32-bit floats (scale merge, round-to-grid,
  round-to-nearest re-quantisation) are emulated with numpy float32
  elementwise operations, which are IEEE-754 correctly rounded and are never
  contracted into fused multiply-adds.
* Codecs (E2M1, E8M0, E4M3) are written from their bit-field definitions and
  their encoders by exact comparison against the enumerated value grids.

Modules
-------
codec   element formats: E2M1 codes, E8M0 and E4M3 block scales (paper §2,
        "Native FP4 microscaling storage").
linear  dequantisation, forward, dX and the per-block scale gradient dS
        (paper §2 storage equation; §3 "Scale-QLoRA forward").
merge   scale-plane merge / swap on the deployment grid (§3 "QAST makes merge
        exact by construction", stability recipe items (ii)-(iii); App. B.2
        hot-swap).
rtn     round-to-nearest re-quantisation of a bf16 weight, the naive merge
        baseline (§2 "The naive re-quantized merge"; App. "Why the naive merge
        returns the base" for the amax/6 rule; App. "Calibrated PTQ on a sparse
        MoE" for the MXFP4 ceil-log2 rule).
audit   merge rollback with the applied on-grid delta and byte / nibble diff
        counts (App. B "Payoff 3: invertible merges and rollback", "Payoff 5:
        verifiability and provenance").
qast    one QAST low-rank scale step: Delta_S = (alpha/r) B A, the on-grid
        scale bytes through the merge's grid-and-clamp path, the clamp mask,
        and the factor gradients dB, dA (§3 "Scale-QLoRA forward", "QAST
        makes merge exact by construction", stability recipe (ii)-(iii)).
qat     the QAT-LoRA weight-space STE comparator: W = base + (alpha/r) B A
        fake-quantised by the nearest rule, and the factor gradients through
        the straight-through estimator (§2 related work, "Merge-aware
        weight-space"; App. "Training cost per step").
philox  Philox4x64-10, the counter-based generator behind the stochastic
        deploy rule (rtn.quantize_rule; App. B threat model (a), the
        deployment-quantizer sweep).
"""

from . import audit, codec, linear, merge, philox, qast, qat, rtn  # noqa: F401
