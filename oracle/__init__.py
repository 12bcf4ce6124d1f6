"""fp64 CPU oracle for the JoLT / FlashJoLT compression path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, deliberately
obvious restatement of the method of "A JoLT for the KV Cache" (arXiv
2607.12550) in float64 numpy.  It exists to check the GPU library, and only
the test suite, the smoke entry point and the benchmark's CPU-baseline leg may
import it.  It shares no code with the GPU library and imports nothing from it.

Module map (paper passages in brackets):

* :mod:`oracle.rounding`  - fp16 / bf16 round-to-nearest-even used by the
  stored formats (fp16 factor serialisation, section 9 Conclusion).
* :mod:`oracle.philox`    - Philox4x32-10 counter-based generator (Salmon et
  al. 2011), Box-Muller Gaussians, Rademacher signs.
* :mod:`oracle.residual`  - random orthogonal rotation and uniform b-bit
  residual quantiser (section 4, "Rotated residual").
* :mod:`oracle.tucker`    - mode spectra, exact and randomized token-mode
  SVD with tail-mass accounting (sections 4 and 5), ST-HOSVD truncation,
  serialisation and reconstruction.
* :mod:`oracle.alloc`     - byte model eq. (1), error model eq. (2),
  budgeted problem eq. (3), Lagrangian bisection eq. (4), FlashJoLT cap
  policy (section 5, "Cap selection"), epsilon^2(b) calibration.
* :mod:`oracle.pipeline`  - one cell end to end, budgeted whole-cache
  compression, the blob byte format, metrics.
* :mod:`oracle.rope`      - rotary position embedding re-applied to decoded
  keys (appendix B: keys are compressed before RoPE).
* :mod:`oracle.diagnostics` - singular values of the three mode unfoldings and
  their appendix-A summary (section 3, appendix A).
* :mod:`oracle.attention` - decode-time softmax attention over the decompressed
  cache (the result a fused attention-on-factors kernel must reproduce; section 8).

Parity-unpinned items (no value in the paper can be reproduced on synthetic
data): the absolute reconstruction errors, the epsilon^2(b) values, the chosen
ranks and the speedups.
"""
from . import rounding, philox, residual, tucker, alloc, pipeline, rope, diagnostics, attention  # noqa: F401,E402
