"""CPU oracle for OmniQuant's block-wise calibration step -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct numpy restatement of what one
calibration step computes (OmniQuant, arXiv 2308.13137: Eq.1 block objective,
Eq.2 learnable weight clipping, Eq.3/Eq.4 learnable equivalent transformation,
Algorithm 1's inner loop body, and the AdamW update of the training settings in
Sec. 4.1).  It exists only to check the HIP path.  Only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may import
it; the product package never does, and it imports nothing from the product.

Precision.  Where a floating-point value decides an integer (a quantisation
code, an argmax/argmin) the oracle takes that decision in fp32 with a fixed
operation order ("fp32-spec mode", the precision the kernels use), so integer
codes can be compared bit for bit.  Everything else (dot products, sums,
gradients) is evaluated in fp64 and rounded once.  bf16 rounding is applied
only where the kernels hand a bf16 operand to a matrix product.  Every
function also runs with ``ft=np.float64`` and ``bf16=False`` (pure fp64 mode),
used by the finite-difference checks.

Modules
  quant      Eq.2 quantiser (LWC) and the per-token MinMax quantiser, fwd + STE bwd
  let        Eq.3 LET transform, bias fold, SmoothQuant/OS+ initialisation
  block      one block step over the block's linear sub-graph (Eq.1, Eq.4, Alg.1)
  adamw      the AdamW update (Sec. 4.1 training settings)
  surrogate  fp64 frozen-selection surrogate of the step, for finite differences
  packed     low-bit code storage and the weight-only quantised linear of
             the deployed model (Sec. 4.5)
"""
