"""Workload shapes for the synthetic LLaVA-shaped inputs.

Five workloads mirror the configurations the pruned-and-skipped prefill is
evaluated on: a tiny fp32 case that a plain CPU implementation finishes in
seconds, and four bf16 cases shaped like LLaVA-1.5-7B (576 visual tokens from
a CLIP ViT-L/14-336), LLaVA-NeXT-7B (AnyRes, 5 tiles of 576), LLaVA-1.5-13B at
batch 8, and a high-resolution stress sweep.  The vision side feeds the
scoring step (CLS attention of the last tapped ViT layer plus the hidden
states of the tapped layers); the decoder side is a LLaMA-style stack.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class ScoreCfg:
    G: int                  # tiles scored independently (batch x AnyRes tiles)
    n: int                  # patch tokens per tile (CLS excluded)
    H: int                  # ViT heads
    d_v: int                # ViT width
    layers: Tuple[int, ...]  # tapped ViT layers (1-indexed); the last one is F^L
    feat_dtype: str         # "f32" | "bf16"
    keep: int               # visual tokens kept per tile
    r_num: int = 7          # anchor ratio r = r_num / r_den (default 0.7)
    r_den: int = 10
    K: int = 4              # K-means clusters
    kmeans_iter: int = 10   # Lloyd iteration cap


@dataclass(frozen=True)
class DecoderCfg:
    L: int
    d: int
    H: int
    d_ff: int
    dtype: str              # "f32" | "bf16" (weights and activations)
    eps: float = 1e-5
    theta: float = 10000.0

    @property
    def dh(self) -> int:
        return self.d // self.H


@dataclass(frozen=True)
class Workload:
    name: str
    score: ScoreCfg
    dec: DecoderCfg
    B: int                  # samples
    tiles_per_sample: int   # AnyRes tiles per sample (G = B * tiles_per_sample)
    n_text: int             # text rows per sample, placed after the visual rows
    skip: dict = field(default_factory=dict)
    seed: int = 0
    quota_mode: int = 0     # 0 = literal Eq.2 rounding, 1 = exact budget

    def with_keep(self, keep: int) -> "Workload":
        return replace(self, score=replace(self.score, keep=keep))

    def with_layers(self, L: int) -> "Workload":
        return replace(self, dec=replace(self.dec, L=L))


_VIT_L = dict(n=576, H=16, d_v=1024, layers=(12, 24), feat_dtype="bf16")
_DEC_7B = DecoderCfg(L=32, d=4096, H=32, d_ff=11008, dtype="bf16")
_DEC_13B = DecoderCfg(L=40, d=5120, H=40, d_ff=13824, dtype="bf16")

WORKLOADS = {
    # 4-layer ViT (d=64, 2 heads, CLS + 7x7 patches), taps {2,4}, keep 16 of 49;
    # 2-layer decoder d=128, 4 heads, SwiGLU 344, 32 text rows; attention of
    # decoder layer 1 skipped for every visual row.
    "tiny": Workload(
        name="tiny",
        score=ScoreCfg(G=1, n=49, H=2, d_v=64, layers=(2, 4), feat_dtype="f32", keep=16),
        dec=DecoderCfg(L=2, d=128, H=4, d_ff=344, dtype="f32"),
        B=1, tiles_per_sample=1, n_text=32,
        skip={"kind": "mask", "attn_layers": (1,), "ffn_layers": ()},
    ),
    # LLaVA-1.5-7B shape, batch 1, keep 64/128/192 of 576 (128 by default);
    # every (layer, sub-layer) slot skipped for all visual rows with p = 0.25.
    "llava15_7b": Workload(
        name="llava15_7b",
        score=ScoreCfg(G=1, keep=128, **_VIT_L),
        dec=_DEC_7B, B=1, tiles_per_sample=1, n_text=64,
        skip={"kind": "random_layer", "p": 0.25},
    ),
    # LLaVA-NeXT-7B shape: AnyRes 5 x 576 tokens, keep 320 or 640 in total
    # (64 or 128 per tile); adaptive skip from the NeXT replaced-layer list.
    "llava_next_7b": Workload(
        name="llava_next_7b",
        score=ScoreCfg(G=5, keep=64, **_VIT_L),
        dec=_DEC_7B, B=1, tiles_per_sample=5, n_text=64,
        skip={"kind": "adaptive", "policy": "llava_next_7b", "T_skip": 20.0,
              "w1": 3.0, "w2": 1.0, "u_max": 0.21},
    ),
    # LLaVA-1.5-13B shape, batch 8, keep 128 of 576 per sample, per-sample
    # adaptive skip (synthetic 40-layer policy with 7 FFN layers; the threshold
    # is scaled with the 20-layer decision window, 20 * 20/16 = 25).
    "llava15_13b": Workload(
        name="llava15_13b",
        score=ScoreCfg(G=8, keep=128, **_VIT_L),
        dec=_DEC_13B, B=8, tiles_per_sample=1, n_text=128,
        skip={"kind": "adaptive", "policy": "synthetic_40", "T_skip": 25.0,
              "w1": 3.0, "w2": 1.0, "u_max": 0.185},
    ),
    # High-resolution stress: batch 4 x 2880 visual tokens (5 tiles of 576),
    # keep ratio 1.0/0.5/0.25/0.11 per tile (576/288/144/64), random per-layer
    # skip with fraction 0/0.25/0.5.
    "stress": Workload(
        name="stress",
        score=ScoreCfg(G=20, keep=576, **_VIT_L),
        dec=_DEC_7B, B=4, tiles_per_sample=5, n_text=64,
        skip={"kind": "random_layer", "p": 0.0},
    ),
}


def get_workload(name: str, keep: Optional[int] = None, L: Optional[int] = None,
                 skip_p: Optional[float] = None) -> Workload:
    w = WORKLOADS[name]
    if keep is not None:
        w = w.with_keep(keep)
    if L is not None:
        w = w.with_layers(L)
    if skip_p is not None:
        w = replace(w, skip={"kind": "random_layer", "p": float(skip_p)})
    return w
