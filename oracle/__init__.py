"""CPU oracle for the chunk-wise Gated DeltaNet inverse path (fp64 / exact ints).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import, call or run anything here.  It shares no code with
the HIP library (no kernels, headers, helpers or constant tables); the only
module both sides use is the seeded input generator ``workloads``.

Every function is a plain, slow statement of what the paper defines, in
float64 (or exact integers for the low-bit path), written so that it can be
checked against the paper by eye.  Stacks of tiles are processed with numpy's
batched matmul as a library primitive; nothing is blocked, fused or
reordered beyond what the definitions state.

Sign convention: the paper inverts (I - A) with A strictly lower triangular
(Section 2.1).  Gated DeltaNet inverts (I + A) with
A = strict_tril(diag(beta) (K K^T) * exp(g_i - g_j)); every paper formula is
applied here to Lm := -A, so (I + A)^-1 = (I - Lm)^-1.

Modules:
  gdn   float64 oracle: build A, exact inverse (forward substitution),
        masked truncated Neumann + residual correction (Algorithm 1),
        Newton form, block-wise inverse (Appendix E), WY application,
        accuracy metrics.
  int8  exact-integer oracle of the low-bit (INT8) pipeline.
  gdn_forward  float64 oracle of the whole chunk-wise Gated DeltaNet forward
        (token recurrence, and the chunk-wise form around the inverse).
  varlen  the chunk path over packed variable-length sequences (partial last
        chunks).
"""

from . import gdn  # noqa: F401
from . import int8  # noqa: F401
from . import gdn_forward  # noqa: F401
from . import varlen  # noqa: F401
