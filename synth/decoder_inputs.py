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


def projector_weights(w: Workload, device="cpu") -> dict:
    """LLaVA's two-layer projector from the ViT width to the decoder width:
    w1 [d_model, d_v], w2 [d_model, d_model] approximately N(0, 0.02) in the
    workload dtype, biases b1, b2 fp32 N(0, 0.02)."""
    d_v, d = w.score.d_v, w.dec.d
    return {"w1": _tensor((d, d_v), w.dec.dtype, w.seed, 4600, device),
            "w2": _tensor((d, d), w.dec.dtype, w.seed, 4601, device),
            "b1": _tensor((d,), "f32", w.seed, 4602, device).float(),
            "b2": _tensor((d,), "f32", w.seed, 4603, device).float()}


def projector_inputs(w: Workload, device="cpu") -> torch.Tensor:
    """[G, n+1, d_v] ViT rows the projector reads (LLaVA takes the layer before the
    last; row 0 = [CLS]), approximately N(0, 1) in the workload dtype."""
    shape = (w.score.G, w.score.n + 1, w.score.d_v)
    if w.dec.dtype == "bf16":
        return normal_bf16(shape, w.seed, 4604, 1.0, device=device)
    x = rng(w.seed, 50000 + 4604).standard_normal(shape).astype(np.float32)
    return torch.from_numpy(x).to(device)
