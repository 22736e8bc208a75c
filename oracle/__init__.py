"""CPU fp64 oracle of one DC-Leap denoising iteration — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg
may import this package. The product (the HIP library and its Python binding)
never calls it, and this package imports nothing from the product; the only
shared code is the seeded input generator ``synth``.

Every function is the plain definition from the paper (DC-Leap, "Draft-guided
Contiguous Leaping"), written out in numpy float64:

* ``numerics``  — bfloat16 rounding, RMSNorm, RoPE, SiLU (architecture of the
  LLaDA / Dream base models of Section 4 setup);
* ``forward``   — the bidirectional transformer forward, ``Forward(p_theta, x)``
  of Algorithm 1 (Appendix A);
* ``scores``    — per-position softmax over the vocabulary (Section 2.1, Eq. 2),
  top-1 confidence (Eq. threshold_pd), top-1/top-2 gap (Section 2.2);
* ``select``    — Dynamic Contiguous Verification (Section 3.2, Eq. compute_k),
  commit, draft update (Section 3.3, Eq. draft_update) and draft invalidation
  (Eq. remasking);
* ``loop``      — the full decode loop of Algorithm 1 and the brute-force
  sequential (chain-rule, Section 2.2) and non-contiguous threshold (Eq.
  threshold_pd) reference decoders used as pins.

Parity status: the selection rules and the vocabulary reduction are pinned by
closed forms, exhaustive enumeration and library routines (``tests/``). The
transformer forward has no published numeric value to match: it is pinned by
library routines (torch.nn.functional in fp64) and invariants only — "parity
unpinned" against the paper itself.
"""
from .numerics import bf16_round, rmsnorm, rope_tables, apply_rope, silu  # noqa: F401
from .forward import forward, lm_logits  # noqa: F401
from .scores import row_entropy, row_stats, SENTINEL_ID, SENTINEL_CONF  # noqa: F401
from .select import compute_k, select_contiguous, select_noncontiguous, scored_mask  # noqa: F401
from .step import step, step_from_weights  # noqa: F401
from .loop import generate, sequential_greedy, noncontiguous_commit_set  # noqa: F401
