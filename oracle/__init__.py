"""Plain fp64 CPU oracle for the symmetric InfoNCE (CLIP) loss.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) imports, links or calls this package; only the tests, the
round-end smoke check and the benchmark's CPU-baseline leg do.  It shares no
code, constants or helpers with the GPU path.

The oracle computes the loss of Eq. 1 (image->text) and its symmetric
text->image counterpart (Sec. 2.2, "the implementation of text-to-image loss is
symmetric"), averaged, together with the exact gradients of the chain rule of
Eq. 6, completed for the temperature/scale, the text side and the column half.
It deliberately does NOT follow the paper's tiling (Eq. 3-5, Alg. 2/4): the
method is an exact rewrite of this definition, so the definition itself is the
oracle.  See ``oracle.infonce`` for the per-function citations.
"""

from .infonce import (  # noqa: F401
    forward,
    backward,
    forward_backward,
    sampled_rows,
    sampled_cols,
    softplus,
)
