"""Plain CPU oracle of DAVET's per-step hot path.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything here.  The product path (the HIP library and
its Python binding) never calls into this package, and this package never
imports the product.  The two share no code; only the seeded input generators
in ``synth`` serve both sides.

Contents (each function cites the passage of the paper it follows):
  views   -- evidence hierarchy by per-crop average pooling + index maps
             (Sec. 4.3 "Ordered evidence hierarchy", v^(K) = v)
  realizers -- nested pruning and hierarchical similarity merging through
             the same index maps (Sec. 4.3 "Compatible evidence realizers")
  policy  -- phase profile, normalisation N(p; beta), evidence envelope,
             trajectory risk, envelope allocation, K-level quantisation
             (Sec. 4.2, Eqs. 6-9; Appendix A Table A for the demand prior)
  model   -- bidirectional masked-diffusion denoiser step over
             [view | prompt | response] (Sec. 3.1, Eq. 1)
  decode  -- argmax and max-softmax confidence on masked rows, confidence-
             ranked commitment (Eq. 2; Sec. 5.1 decoding settings)
  stats   -- mean confidence and prediction churn for the risk (Sec. 4.2)
  loop    -- the full schedule loop (Sec. 3.1 and Fig. 2's procedure)

Precision: the denoiser runs in float64 on bf16-rounded (or fp32) inputs;
the policy runs in IEEE double with the operation order printed in the
equations.  Readings of silent or ambiguous passages are listed in the
design notes of the repository and restated where each is used.
"""

from . import views, realizers, policy, model, decode, stats, loop  # noqa: F401
