"""One pass of the pruned-and-skipped prefill through the C ABI.

score (GPU) -> select + assembly (GPU) [-> projector on the kept rows (GPU)]
-> [one device-to-host copy of the
sample boundaries] -> skip plan (host, Algorithm 1 admission or a per-layer
mask) -> prefill (GPU); or, with the online policy, the prefill whose
controller scores and admits the visual rows on the device layer by layer
(spider_prefill_online).  This module only sequences library calls and packs
the per-sample skip codes into the [L, rows] layout of the prefill (visual
rows of a sample first, text rows never skip); buffers are allocated once.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from . import _lib


@dataclass
class SkipPolicy:
    kind: str                                  # "layer_mask" | "adaptive" | "online"
    layer_mask: Optional[np.ndarray] = None    # [L, 2] bool (attention, FFN)
    s_sa: Optional[np.ndarray] = None          # [B, L//2, n_vis_max] float32
    slc_sel: Optional[np.ndarray] = None       # [L] float64
    target: Optional[np.ndarray] = None        # [L] uint8
    w1: float = 3.0
    w2: float = 1.0
    T_skip: float = 20.0
    w_unembed: Optional[torch.Tensor] = None   # [V, d] (online)


class Pipeline:
    def __init__(self, *, G: int, n: int, K: int, keep: int, r_num: int, r_den: int,
                 kmeans_iter: int, tiles_per_sample: int, n_text: int, quota_mode: int,
                 dec: _lib.DecoderCfg, weights, device, projector: Optional[dict] = None):
        self.G, self.n, self.K = G, n, K
        self.n_anchor, self.n_cmp = _lib.budget(keep, r_num, r_den)
        self.n_anchor = min(self.n_anchor, n)
        self.cap = min(n, self.n_anchor + self.n_cmp + K)
        self.kmeans_iter = kmeans_iter
        self.tps, self.n_text, self.quota_mode = tiles_per_sample, n_text, quota_mode
        self.B = G // tiles_per_sample
        self.dec = dec
        self.weights = weights
        self.wtable = _lib.layer_weights(weights)
        self.device = device
        max_rows = self.B * (self.tps * self.cap + n_text)
        self.prefill_ws = torch.empty(_lib.prefill_workspace_size(dec, self.B, max_rows) + 256,
                                      dtype=torch.uint8, device=device)
        self.h = torch.empty(max_rows, dec.d, dtype=torch.float32, device=device)
        self.max_rows = max_rows
        self.online_ws = None
        # projector on the kept rows (weights dict w1, b1, w2, b2 on the device): the
        # assembly then places the text rows only and the projector writes the kept rows
        self.projector = projector
        self.proj_ws = None
        self.x_buf = None
        self.cu_host = torch.empty(self.B + 1, dtype=torch.int32, pin_memory=True)

    def codes(self, cu: np.ndarray, policy: SkipPolicy) -> np.ndarray:
        L = self.dec.L
        rows = int(cu[-1])
        out = np.zeros((L, rows), np.uint8)
        for b in range(self.B):
            n_vis = int(cu[b + 1] - cu[b]) - self.n_text
            if policy.kind == "layer_mask":
                m = policy.layer_mask
                col = (m[:, 0].astype(np.uint8) | (m[:, 1].astype(np.uint8) << 1))
                out[:, cu[b]:cu[b] + n_vis] = col[:, None]
            elif policy.kind == "adaptive":
                c, _ = _lib.plan_skips(policy.s_sa[b][:, :n_vis], policy.slc_sel, policy.target,
                                       policy.w1, policy.w2, policy.T_skip, L)
                out[:, cu[b]:cu[b] + n_vis] = c
            else:
                raise ValueError(policy.kind)
        return out

    def step(self, cls_attn, feats, src, text, policy: SkipPolicy):
        """``src``: visual rows already in the decoder width [G, n, d], or, with a
        projector, the ViT rows it reads [G, n+1, d_v] (row 0 = [CLS])."""
        sc = _lib.score(cls_attn, feats, self.n_anchor, self.K, self.kmeans_iter)
        if self.projector is not None:
            if self.x_buf is None:
                self.x_buf = torch.empty(self.max_rows, self.dec.d, dtype=text.dtype, device=self.device)
            sel = _lib.select(sc["cluster"], sc["s"], self.n_anchor, self.n_cmp, self.K,
                              self.quota_mode, self.cap, self.tps, text=text, text_only=True,
                              x_out=self.x_buf)
            if self.proj_ws is None:
                L = _lib.lib()
                w1, w2 = self.projector["w1"], self.projector["w2"]
                nb = L.spider_project_kept_workspace_size(self.G, self.cap, w1.shape[0], w2.shape[0],
                                                          _lib._dt(src))
                self.proj_ws = torch.empty(nb + 256, dtype=torch.uint8, device=self.device)
            _lib.project_kept(sel, src, self.projector, self.tps, self.n_text, workspace=self.proj_ws)
        else:
            sel = _lib.select(sc["cluster"], sc["s"], self.n_anchor, self.n_cmp, self.K,
                              self.quota_mode, self.cap, self.tps, src, text)
        self.cu_host.copy_(sel["cu_seqlens"], non_blocking=True)
        torch.cuda.current_stream(self.device).synchronize()
        cu = self.cu_host.numpy().copy()
        rows = int(cu[-1])
        if policy.kind == "online":
            V = int(policy.w_unembed.shape[0])
            if self.online_ws is None:
                nb = _lib.prefill_online_workspace_size(self.dec, self.B, self.max_rows, V)
                self.online_ws = torch.empty(nb + 256, dtype=torch.uint8, device=self.device)
            h, codes, admit, _ = _lib.prefill_online(
                self.dec, None, cu, sel["x"][:rows], self.n_text, policy.w_unembed, policy.slc_sel,
                policy.target, policy.w1, policy.w2, policy.T_skip, s_sa=False, out=self.h[:rows],
                workspace=self.online_ws, weight_table=self.wtable)
            return {"score": sc, "select": sel, "cu": cu, "codes": codes, "admit": admit, "h": h}
        codes = self.codes(cu, policy)
        h = _lib.prefill(self.dec, None, cu, sel["x"][:rows], codes, out=self.h[:rows],
                         workspace=self.prefill_ws, weight_table=self.wtable)
        return {"score": sc, "select": sel, "cu": cu, "codes": codes, "h": h}
