"""Seeded synthetic inputs shared by the GPU path's tests/bench and the oracle.

This package only *draws* inputs (random tensors with the shapes and value
structure of the paper's LLaVA workloads); it holds none of SPIDER's
arithmetic.  Two generators are used:

* ``numpy.random.Generator(PCG64(SeedSequence([seed, tensor_id])))`` for the
  small vision-side tensors (CLS attention, ViT features, skip scores), and
* a counter-based SplitMix64 generator (``counter_rng``) for the large decoder
  tensors (weights, visual source rows, text rows), which produces identical
  bits on the CPU and on the GPU so multi-GB weight sets need not be copied.
"""
from .configs import WORKLOADS, Workload, ScoreCfg, DecoderCfg, get_workload  # noqa: F401
from .counter_rng import normal_bf16, normal_f32  # noqa: F401
from . import vision, decoder_inputs, skip_inputs  # noqa: F401
