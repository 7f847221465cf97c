"""MI355X (gfx950) implementation of SPIDER's pruned-and-skipped multimodal prefill.

The work happens in libspider.so (hand-written HIP kernels behind the C ABI of
include/spider.h); this package only loads it and marshals torch tensors.
"""
from ._lib import (  # noqa: F401
    BF16, F32, SpiderError, budget, decoder_cfg, layer_weights, lib, plan_skips, prefill,
    prefill_workspace_size, profile_enable, profile_read, score, select, slc_policy,
)
from .pipeline import Pipeline  # noqa: F401
