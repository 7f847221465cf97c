"""Inputs of the sub-layer skip plan.

* Per-layer masks (``random_layer``): each (layer, sub-layer) slot is skipped
  for every visual row with probability p, drawn once per workload.
* Explicit masks (``mask``): the listed layers skip attention / FFN for every
  visual row.
* Adaptive plans (``adaptive``): the online skippability score S_sa of each
  visual token in each decision-window layer is drawn as
  clip(u_i + 0.1 * N(0,1), 0, 1) with u_i ~ U(0, u_max); u_max is chosen per
  workload so that roughly 41 % of the visual tokens enter skip mode with
  T_skip = 20, w1/w2 = 3 (the paper's operating point).  With random-init
  weights the paper's online score would be about 0 for every token, so the
  score is an input here.  The offline per-layer sub-layer contribution table
  (raw KL-like values for attention and FFN per layer) is built from the
  paper's replaced-sub-layer lists (Table 10): a layer listed under
  attention gets an attention value that grows with its position in the
  list and a large FFN value, and vice versa, so that the normalisation of
  Eq. 5 followed by the per-layer argmax reproduces the list.

Codes are bytes per (layer, visual row): bit 0 = skip attention,
bit 1 = skip FFN.
"""
from __future__ import annotations

import numpy as np

from .configs import Workload
from .vision import rng

# Table 10: replaced sub-layers, most skippable first, 0-indexed decoder layers.
REPLACED_LAYERS = {
    "llava15_7b": {
        "attn": (25, 27, 28, 30, 23, 26, 22, 24, 21, 0, 20, 3, 18, 4, 19, 17, 14, 15,
                 5, 16, 12, 1, 13, 7, 8, 9, 10),
        "ffn": (31, 29, 2, 11, 6),
    },
    "llava_next_7b": {
        "attn": (28, 29, 27, 30, 23, 24, 25, 22, 21, 26, 20, 19, 18, 17, 15, 16, 14, 12,
                 4, 13, 5, 0, 7, 6, 8),
        "ffn": (31, 1, 2, 3, 11, 9, 10),
    },
}


def synthetic_policy(L: int, n_ffn: int, seed: int = 0) -> dict:
    """A replaced-layer list for a decoder the paper does not list (e.g. 40 layers)."""
    r = rng(seed, 6000 + L)
    perm = [int(x) for x in r.permutation(L)]
    return {"attn": tuple(perm[n_ffn:]), "ffn": tuple(perm[:n_ffn])}


def policy_lists(name: str, L: int, seed: int = 0) -> dict:
    if name in REPLACED_LAYERS:
        return REPLACED_LAYERS[name]
    if name == "synthetic_40":
        return synthetic_policy(L, 7, seed)
    raise KeyError(name)


def slc_tables(lists: dict, L: int):
    """Raw (attention, FFN) contribution values per layer, float32 [L] each."""
    slc_attn = np.full(L, 1.0, dtype=np.float64)
    slc_ffn = np.full(L, 10.0, dtype=np.float64)
    for rank, layer in enumerate(lists["attn"]):
        slc_attn[layer] = 0.01 * (1 + rank)
    for rank, layer in enumerate(lists["ffn"]):
        slc_ffn[layer] = 0.1 * (1 + rank)
    return slc_attn.astype(np.float32), slc_ffn.astype(np.float32)


def layer_mask(w: Workload) -> np.ndarray:
    """[L, 2] bool: (layer, sub-layer) slots skipped for every visual row."""
    L = w.dec.L
    kind = w.skip.get("kind")
    m = np.zeros((L, 2), dtype=bool)
    if kind == "mask":
        for l in w.skip.get("attn_layers", ()):
            m[l, 0] = True
        for l in w.skip.get("ffn_layers", ()):
            m[l, 1] = True
    elif kind == "random_layer":
        p = float(w.skip.get("p", 0.0))
        m = rng(w.seed, 7000).random((L, 2)) < p
    else:
        raise ValueError(f"no per-layer mask for skip kind {kind!r}")
    return m


def layer_mask_codes(w: Workload, n_vis: int) -> np.ndarray:
    """[L, n_vis] uint8 codes of a per-layer mask (same code for every visual row)."""
    m = layer_mask(w)
    c = (m[:, 0].astype(np.uint8) | (m[:, 1].astype(np.uint8) << 1))
    return np.repeat(c[:, None], n_vis, axis=1)


def adaptive_scores(w: Workload, n_vis_max: int) -> np.ndarray:
    """S_sa [B, L//2, n_vis_max] float32 for the decision window."""
    W = w.dec.L // 2
    out = np.empty((w.B, W, n_vis_max), dtype=np.float32)
    u_max = float(w.skip.get("u_max", 0.7))
    for b in range(w.B):
        r = rng(w.seed, 8000 + b)
        u = r.uniform(0.0, u_max, size=n_vis_max)
        noise = 0.1 * r.standard_normal((W, n_vis_max))
        out[b] = np.clip(u[None, :] + noise, 0.0, 1.0).astype(np.float32)
    return out
