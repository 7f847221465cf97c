"""Plain CPU oracle of SPIDER's pruned-and-skipped multimodal prefill.

TEST INFRASTRUCTURE ONLY.  This package is the slow, obviously-correct
reference that the GPU library is checked against.  Only the test suite, the
smoke entry point and the benchmark's CPU-baseline leg may import it; the
product path (the HIP library and its Python binding) never imports, calls or
links anything here, and nothing here imports the product path.

Modules (each function cites the passage of the paper it follows):

* ``bf16``       - round-to-nearest-even to bfloat16 (the rounding recipe of
                   the bf16 workloads).
* ``msv_prune``  - Sec. 4.1: CLS-attention anchors (Eq. 1), K-means
                   clustering, quota allocation (Eq. 2), multi-layer
                   similarity (Eq. 3), per-cluster selection, spatial-order
                   union and sequence assembly.
* ``asl_skip``   - Sec. 4.2-4.3 and Algorithm 1: skippability (Eq. 4),
                   SLC normalisation (Eq. 5), per-layer target, fused score
                   accumulation and admission (Eq. 6).
* ``decoder``    - the LLaMA-style decoder prefill with per-row sub-layer
                   bypass (VSkip-Attn / VSkip-FFN of Sec. 3.2), computed
                   densely and then masked.

Parity status of each function is stated in its module docstring.
"""
from . import bf16, msv_prune, asl_skip, decoder  # noqa: F401
