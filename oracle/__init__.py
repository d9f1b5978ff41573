"""CPU oracle for the Archer cached-prompt decoding path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its Python
binding) never imports, links or runs anything from here, and this package
imports nothing from the product path.

The oracle is plain, slow and written for checking by eye against the paper
("Archer: Adaptive Reuse of Cached Hidden States for Efficient Rollback in
Diffusion Language Models", arXiv 2608.08086):

* :mod:`oracle.model`      -- the bidirectional DLM forward Phi_theta in its two
  modes, FullForward(p, g) (Sec. 4.1 Eq. archer-fresh; App. A.1 Eq. app-eager)
  and CachedForward(g; C_r) (Sec. 4.1 Eq. archer-cached / archer-attention;
  App. A.1 Eq. app-cached).
* :mod:`oracle.decoder`    -- the confidence unmask / threshold remask decoder D
  and a computable lower bound on its decision margin (Sec. 5.2
  Eq. theory-margin; App. A.5 Prop. app-decision).
* :mod:`oracle.controller` -- the anchor distance D_t = d_H(g_t, g_r)
  (Sec. 4.2 Eq. archer-distance) and the refresh rules (Eq. archer-controller;
  the cache-age signal A_t = t - r of Sec. 6.4).
* :mod:`oracle.decode`     -- Algorithm 1 (state-anchored rollback decoding).

Arithmetic is float64 (NumPy).  For bf16 models the oracle rounds to bf16
(round-to-nearest-even) at exactly the points where the HIP path stores bf16
operands (see :mod:`oracle.numerics`); everything else stays float64.

Parity status: the paper prints no numeric worked example, so absolute
logits and trajectories are not pinned by printed values.  Every function is
pinned instead by brute force on tiny inputs, library routines, closed forms
and the paper's invariants (tests/test_oracle_*.py).
"""

from . import numerics, model, decoder, controller, decode  # noqa: F401
