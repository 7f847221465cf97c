"""Vision-side inputs of the scoring step: CLS attention rows and ViT taps.

Two sources:

* ``tiny_vit_taps``: a small random-weight ViT (pre-LayerNorm blocks, GELU MLP
  of width 4d, no biases, weights and patch embeddings N(0, 0.02)) run in
  float64 on CLS + 7x7 patch tokens.  It stands in for the frozen encoder of
  the tiny workload; its outputs are the CLS attention row of the last tapped
  layer (per head) and the hidden states after the tapped blocks.
* ``llava_taps``: CLIP-ViT-L/14-336-shaped synthetic taps for G tiles of 576
  patches.  CLS attention per (tile, head) is a softmax over n+1 logits drawn
  as 2*N(0,1), with +4 added on a seeded 5 % of the patches (the same salient
  patches for every head of a tile), which gives the peaked profile of CLIP's
  CLS attention.  Features are object-like blobs: each patch of the 24x24 grid
  belongs to the Voronoi region of the nearest of R seeded centres, and
  F[i] = c_region + 0.3 * N(0,1) with c ~ N(0,1)^d_v.  The last tapped layer
  uses 6 regions (coarse, global), earlier taps 12 (finer, object-centric),
  each with independent centres.  Values are rounded to bf16.

Every tensor draws from its own ``PCG64(SeedSequence([seed, tensor_id]))``.
"""
from __future__ import annotations

import math

import numpy as np
import torch
from scipy.special import erf

from .configs import ScoreCfg
from .counter_rng import f32_to_bf16_rne


def rng(seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor_id])))


def _layernorm(x: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def _gelu(x: np.ndarray) -> np.ndarray:
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def tiny_vit_taps(cfg: ScoreCfg, seed: int = 0, n_layers: int = 4):
    """Run the small random ViT; returns (cls_attn [G,H,n+1] f32, feats list of [G,n+1,d_v] f32).

    ``feats`` follows ``cfg.layers`` order (the last entry is the last tapped
    layer); ``cls_attn`` is row 0 of the softmax attention of that layer.
    """
    G, n, H, d = cfg.G, cfg.n, cfg.H, cfg.d_v
    dh = d // H
    T = n + 1
    cls_out = np.zeros((G, H, T), dtype=np.float32)
    feats = {l: np.zeros((G, T, d), dtype=np.float32) for l in cfg.layers}
    last = cfg.layers[-1]
    for g in range(G):
        x = rng(seed, 100 + g).standard_normal((T, d)) * 0.02
        for layer in range(1, n_layers + 1):
            r = rng(seed, 1000 + 16 * layer)
            wqkv = r.standard_normal((3 * d, d)) * 0.02
            wo = r.standard_normal((d, d)) * 0.02
            w1 = r.standard_normal((4 * d, d)) * 0.02
            w2 = r.standard_normal((d, 4 * d)) * 0.02
            y = _layernorm(x)
            qkv = y @ wqkv.T
            q = qkv[:, :d].reshape(T, H, dh).transpose(1, 0, 2)
            k = qkv[:, d:2 * d].reshape(T, H, dh).transpose(1, 0, 2)
            v = qkv[:, 2 * d:].reshape(T, H, dh).transpose(1, 0, 2)
            logits = q @ k.transpose(0, 2, 1) / math.sqrt(dh)
            logits -= logits.max(axis=-1, keepdims=True)
            p = np.exp(logits)
            p /= p.sum(axis=-1, keepdims=True)
            o = (p @ v).transpose(1, 0, 2).reshape(T, d)
            x = x + o @ wo.T
            x = x + _gelu(_layernorm(x) @ w1.T) @ w2.T
            if layer == last:
                cls_out[g] = p[:, 0, :].astype(np.float32)
            if layer in feats:
                feats[layer][g] = x.astype(np.float32)
    return cls_out, [feats[l] for l in cfg.layers]


def _voronoi_regions(n: int, n_regions: int, r: np.random.Generator) -> np.ndarray:
    side = int(round(math.sqrt(n)))
    if side * side == n:
        ys, xs = np.divmod(np.arange(n), side)
        pts = np.stack([ys, xs], axis=1).astype(np.float64)
        centres = r.uniform(0, side, size=(n_regions, 2))
    else:
        pts = np.stack([np.arange(n), np.zeros(n)], axis=1).astype(np.float64)
        centres = np.stack([r.uniform(0, n, size=n_regions), np.zeros(n_regions)], axis=1)
    d2 = ((pts[:, None, :] - centres[None, :, :]) ** 2).sum(-1)
    return d2.argmin(axis=1)


def _to_bf16(x: np.ndarray) -> torch.Tensor:
    return f32_to_bf16_rne(torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)))


def llava_taps(cfg: ScoreCfg, seed: int = 0, tie_stress: bool = False):
    """CLIP-shaped synthetic taps; returns (cls_attn f32 tensor [G,H,n+1], feats list of bf16 tensors [G,n+1,d_v])."""
    G, n, H, d = cfg.G, cfg.n, cfg.H, cfg.d_v
    T = n + 1
    n_sal = max(1, int(round(0.05 * n)))
    attn = np.empty((G, H, T), dtype=np.float32)
    for g in range(G):
        r = rng(seed, 2000 + g)
        logits = 2.0 * r.standard_normal((H, T))
        sal = r.choice(n, size=n_sal, replace=False)
        logits[:, 1 + sal] += 4.0
        logits -= logits.max(axis=-1, keepdims=True)
        p = np.exp(logits)
        p /= p.sum(axis=-1, keepdims=True)
        if tie_stress:
            p = np.round(p * 64.0) / 64.0
        attn[g] = p.astype(np.float32)
    feats = []
    for li, layer in enumerate(cfg.layers):
        n_regions = 6 if li == len(cfg.layers) - 1 else 12
        out = np.empty((G, T, d), dtype=np.float32)
        for g in range(G):
            r = rng(seed, 3000 + 64 * g + layer)
            region = _voronoi_regions(n, n_regions, r)
            centres = r.standard_normal((n_regions, d))
            f = centres[region] + 0.3 * r.standard_normal((n, d))
            out[g, 0] = r.standard_normal(d)
            out[g, 1:] = f
        feats.append(_to_bf16(out))
    return torch.from_numpy(attn), feats


def vision_inputs(cfg: ScoreCfg, seed: int = 0, tie_stress: bool = False):
    """Dispatch: fp32 taps from the tiny ViT, bf16 synthetic CLIP taps otherwise.

    Returns (cls_attn [G,H,n+1] fp32 torch tensor, list of feature tensors
    [G,n+1,d_v] in the workload's feature dtype).
    """
    if cfg.feat_dtype == "f32":
        a, f = tiny_vit_taps(cfg, seed)
        if tie_stress:
            a = (np.round(a * 64.0) / 64.0).astype(np.float32)
        return torch.from_numpy(a), [torch.from_numpy(x) for x in f]
    return llava_taps(cfg, seed, tie_stress)


def attention_maps(G: int, H: int, n: int, seed: int = 0, device="cpu") -> torch.Tensor:
    """Full self-attention maps [G, H, n, n] fp32 of an encoder without [CLS]:
    per (tile, head, query) a softmax over keys of 2 N(0,1) logits, plus +3 on a
    seeded 5 % of key patches per tile (patches most queries attend to, the
    peaked profile of ViT attention).  Logits from the counter generator (same
    bits on every device); the softmax is evaluated in float64 on the host
    when device is "cpu", else in float32 on the device (sweeps only)."""
    from .counter_rng import normal_f32
    z = normal_f32((G, H, n, n), seed, 4400, 2.0, device=device)
    r = rng(seed, 4401)
    boost = torch.zeros(G, 1, 1, n, dtype=torch.float32)
    for g in range(G):
        boost[g, 0, 0, r.choice(n, max(1, n // 20), replace=False)] = 3.0
    z = z + boost.to(device)
    if torch.device(device).type == "cpu":
        return torch.softmax(z.double(), dim=-1).float()
    return torch.softmax(z, dim=-1)


def cls_query_keys(G: int, H: int, dh: int, T: int, seed: int = 0, dtype: str = "bf16"):
    """CLS query [G, H, dh] and keys [G, T, H, dh] of a ViT layer (token 0 = [CLS]):
    N(0, 1) entries, and on a seeded 20 % of the patch tokens of each tile the keys
    of every head get b times that head's query added, b uniform in [0.5, 2]
    (salient patches of graded strength: the peaked [CLS] profile of CLIP with a
    spread of ranks among the patches a budget keeps).  Rounded once to bf16 (or
    kept fp32)."""
    r = rng(seed, 4500)
    q = r.standard_normal((G, H, dh))
    k = r.standard_normal((G, T, H, dh))
    for g in range(G if T > 1 else 0):
        sal = 1 + r.choice(T - 1, max(1, (T - 1) // 5), replace=False)
        b = r.uniform(0.5, 2.0, size=len(sal))
        k[g, sal] += b[:, None, None] * q[g][None]
    qt = torch.from_numpy(q.astype(np.float32))
    kt = torch.from_numpy(k.astype(np.float32))
    if dtype == "bf16":
        return f32_to_bf16_rne(qt), f32_to_bf16_rne(kt)
    return qt, kt
