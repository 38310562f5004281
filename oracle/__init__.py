"""CPU oracle for the Gated Delta Rule-2 (GDR-2) operator -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct fp64 numpy restatement of what
the paper (Gated DeltaNet-2, arXiv 2605.22791) defines.  It exists so that the
GPU path can be checked against something written directly from the paper.

Rules of use:
  * Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
    ``bench.py`` may import it.  The product path (``paper_2605_22791_amd``)
    never imports, calls or links anything here, and nothing here imports the
    product path.  The two share no code.
  * Everything is computed in float64 regardless of the input dtype; callers
    hand in the very same (already bf16-rounded, if applicable) input values
    the GPU path consumes.

Modules:
  recurrent  -- the token-by-token recurrence (Sec. 3.1, eqs. eq_gdn2_e_z,
                eq_gdn2_residual, eq_gdn2_recurrence) and its hand-derived
                reverse-time adjoint (the definition the method reaches);
                packed variable-length batches (App. C.6) as their sequences
                run one by one; grouped value heads (Sec. 3.5) as the key-side
                tensors repeated over each group.
  chunkwise  -- the chunk algebra of App. A (WY form) and App. B (backward),
                exposing every intermediate for per-kernel debugging.
  limits     -- independent textbook recurrences the paper reduces to:
                linear attention, Mamba-2 decay, KDA and Gated DeltaNet (Sec. 2).
  brute      -- dense products of explicit per-token transition matrices.
  fd         -- central finite differences of a scalar loss.
  layer      -- the input stage around the operator: per-head L2 normalisation
                of q and k (App. D.2) and the fp32 log-decay activation
                g = -exp(a) softplus(f + delta) (App. C.1), their adjoints, and
                the fused operator (stage, then the recurrence) with its backward.

Parity pins (tests/test_oracle_*.py) tie each function to something other than
itself: closed forms, tied-gate reductions, brute force and finite differences.
"""

from .recurrent import gdr2_recurrent_fwd, gdr2_recurrent_bwd, gdr2_step_states  # noqa: F401
from .recurrent import gdr2_packed_fwd, gdr2_packed_bwd, gdr2_grouped_fwd, gdr2_grouped_bwd  # noqa: F401
from .chunkwise import gdr2_chunk_fwd_ref, gdr2_chunk_bwd_ref  # noqa: F401
from .layer import gdr2_fused_fwd, gdr2_fused_bwd  # noqa: F401
from . import limits, brute, fd, layer  # noqa: F401
