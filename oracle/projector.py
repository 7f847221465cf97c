"""Multimodal projector applied to the kept visual rows only (the appendix's
reading of MSV-Prune for LLaVA: pruning happens in the ViT feature space,
before the projector).

Test infrastructure (the oracle), not part of the product path.

The projector is LLaVA's two-layer MLP: y = W2 GELU(W1 x + b1) + b2 with the
exact GELU(t) = t Phi(t) = t (1 + erf(t / sqrt 2)) / 2.  Rows are independent,
so projecting only the kept rows equals projecting every row and keeping the
same rows (pinned).  With the bf16 recipe the hidden activation and the output
are rounded to bf16 (the GEMMs accumulate in higher precision, biases and GELU
in float); inputs and weights are taken as given.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from .bf16 import round_bf16


def gelu(t):
    t = np.asarray(t, dtype=np.float64)
    return 0.5 * t * (1.0 + erf(t / np.sqrt(2.0)))


def project(rows, W1, b1, W2, b2, recipe: str = "bf16"):
    """rows [m, d_in] -> [m, d_out] float64 (bf16-representable values with the bf16 recipe)."""
    rnd = round_bf16 if recipe == "bf16" else (lambda t: t)
    x = np.asarray(rows, dtype=np.float64)
    h = x @ np.asarray(W1, np.float64).T
    if b1 is not None:
        h = h + np.asarray(b1, np.float64)
    h = rnd(gelu(h))
    y = h @ np.asarray(W2, np.float64).T
    if b2 is not None:
        y = y + np.asarray(b2, np.float64)
    return rnd(y)


def assemble_projected(feats, idx_per_tile, text, tiles_per_sample: int, W1, b1, W2, b2, row0: int = 1,
                       recipe: str = "bf16"):
    """Decoder input rows: per sample, the projected kept rows of its tiles (tile
    order, patch order within a tile; patch i is row row0 + i of ``feats[g]``)
    followed by the sample's text rows.  Returns (x [rows, d_out], cu_seqlens)."""
    G = len(idx_per_tile)
    B = G // tiles_per_sample
    out, cu = [], [0]
    for b in range(B):
        for g in range(b * tiles_per_sample, (b + 1) * tiles_per_sample):
            idx = np.asarray(idx_per_tile[g], dtype=np.int64)
            if len(idx):
                out.append(project(np.asarray(feats[g])[row0 + idx], W1, b1, W2, b2, recipe))
        if text is not None and text.shape[1]:
            out.append(np.asarray(text[b], dtype=np.float64))
        cu.append(cu[-1] + sum(len(idx_per_tile[g]) for g in range(b * tiles_per_sample,
                                                                      (b + 1) * tiles_per_sample))
                  + (0 if text is None else text.shape[1]))
    d_out = np.asarray(W2).shape[0]
    x = np.concatenate(out, axis=0) if out else np.zeros((0, d_out))
    return x, np.asarray(cu, dtype=np.int64)
