"""CPU oracle for the Subspace Networks stage-boundary codec.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path (the
HIP library and its Python binding) never does, and shares no code with it.

The oracle is the plain definition of each operation, written in numpy with
float64 arithmetic on exactly up-converted inputs, rounded once at the end to
the output dtype with round-to-nearest-even:

* ``compress``       C = (X - P[pos] - T_fixed[tok]) U          (Sec. 4.3.1, Eq. "subtract")
* ``decompress``     X_rec = C U^T + P[pos] + T_fixed[tok]       (Sec. 4.3.1, recovery)
* ``grad_compress``  C_g = G U                                    (Sec. 4.4, Eq. "grad_compress")
* ``grad_decompress`` G_rec = C_g U^T                             (Sec. 4.4, recovery)
* ``project_weights`` W' = U (U^T W)                              (Sec. 4.3 / Sec. 5: rows of the
  projection matrices confined to S = Col(U); Appendix E's projection Pi_S)

The subspace update of Section 4.5 (off-subspace loss, accumulation matrix,
Riemannian gradient, QR retraction) is in ``grassmann``; the modified AdamW
step of Section 5 in ``adamw``; the trainable low-rank token table of
Section 4.3.1 in ``embed``.

``exact`` holds the same operations in exact rational arithmetic
(``fractions.Fraction``) for brute-force checks on tiny inputs.
"""
from .bf16 import decode_bf16, encode_bf16, round_bf16, round_f32, round_to
from .codec import (compress, decompress, grad_compress, grad_decompress,
                    project_weights, default_positions)
from . import adamw, embed, grassmann

__all__ = ["decode_bf16", "encode_bf16", "round_bf16", "round_f32", "round_to",
           "compress", "decompress", "grad_compress", "grad_decompress",
           "project_weights", "default_positions", "grassmann", "adamw", "embed"]
