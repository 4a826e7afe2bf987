"""CPU oracle for one blockwise masked-diffusion denoising step and gated block decode.

TEST INFRASTRUCTURE ONLY.  Plain, slow, obviously correct numpy code (fp64 by
default).  Only ``tests/``, ``__graft_entry__.smoke()`` and the bench's CPU
baseline leg may import it; the GPU library never does, and this package
imports nothing from the library.

Contents
--------
forward  : the dense bidirectional Transformer pass (backbone of Section 3,
           one dense pass per executed step) -> logits of chosen rows.
decode   : Eq. (1) top-1 and confidence; Eq. (2) persistence counter; the
           original low-confidence transfer rule; Eq. (3) residual gate;
           Eq. (4) commit; block termination; the gated block decode loop.
theory   : Proposition 1 (margin condition and its confidence bound),
           g(delta_p), the step ratio and the disagreement losses
           (Eqs. 7 and 12).

Every function cites the passage it follows.  Parity pins live in
``tests/test_oracle_*.py``.  Readings of points the paper leaves open are
stated where they are applied: the decision rules' readings, numbered R1-R27,
in the ``decode`` docstring; the backbone the paper does not spell out in the
``forward`` docstring.
"""
from . import forward, decode, theory  # noqa: F401
