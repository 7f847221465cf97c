"""Decoder-side inputs: LLaMA-style layer weights, visual source rows, text rows.

Weight matrices use the nn.Linear layout ``[out_features, in_features]``
(row-major), values approximately N(0, 0.02) from the counter generator
(bf16 workloads) or exactly N(0, 0.02) from PCG64 (the fp32 tiny workload).
RMSNorm weights are 1.0.  Visual source rows are the vision tokens already in
the decoder width (the projector is not part of the path); text rows are
drawn the same way.  Both use std 0.02.
"""
from __future__ import annotations

import numpy as np
import torch

from .configs import DecoderCfg, Workload
from .counter_rng import normal_bf16
from .vision import rng

MATS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def _shape(dec: DecoderCfg, name: str):
    d, f = dec.d, dec.d_ff
    return {"wq": (d, d), "wk": (d, d), "wv": (d, d), "wo": (d, d),
            "wg": (f, d), "wu": (f, d), "wd": (d, f)}[name]


def _tensor(shape, dtype: str, seed: int, tensor_id: int, device) -> torch.Tensor:
    if dtype == "bf16":
        return normal_bf16(shape, seed, tensor_id, 0.02, device=device)
    x = rng(seed, 50000 + tensor_id).standard_normal(shape).astype(np.float32) * np.float32(0.02)
    return torch.from_numpy(x).to(device)


def layer_weights(dec: DecoderCfg, layer: int, seed: int = 0, device="cpu") -> dict:
    """Weights of one decoder layer as torch tensors on ``device``."""
    w = {"attn_norm": torch.ones(dec.d, dtype=torch.float32, device=device),
         "ffn_norm": torch.ones(dec.d, dtype=torch.float32, device=device)}
    for k, name in enumerate(MATS):
        w[name] = _tensor(_shape(dec, name), dec.dtype, seed, 16 * layer + k, device)
    return w


def all_weights(dec: DecoderCfg, seed: int = 0, device="cpu") -> list:
    return [layer_weights(dec, l, seed, device) for l in range(dec.L)]


def visual_src(w: Workload, device="cpu") -> torch.Tensor:
    """[G, n, d] visual rows in the decoder width (row i = patch i of the tile)."""
    return _tensor((w.score.G, w.score.n, w.dec.d), w.dec.dtype, w.seed, 4000, device)


def text_rows(w: Workload, device="cpu") -> torch.Tensor:
    """[B, n_text, d] text rows, appended after each sample's kept visual rows."""
    return _tensor((w.B, w.n_text, w.dec.d), w.dec.dtype, w.seed, 4001, device)
