"""Decoder prefill driven by the online skip controller (Sec. 4.2.1, Eq. 4, Eq. 6, Algorithm 1).

Test infrastructure (the oracle), not part of the product path.

At every decision-window layer l (0-indexed, l < floor(L/2)) each visual
token of each sample that is not yet in skip mode gets its online
skippability from the hidden state entering layer l:

* E_ii: Shannon entropy of softmax(W_unembed h), divided by ln|V| (the logit
  lens, no final norm; with the bf16 recipe the lens reads bf16(h), the
  precision a bf16 GEMM consumes);
* F_itc: (1 + cos(h_i, q_t)) / 2 with q_t the mean hidden state of the
  sample's text rows entering layer l;
* S_sa = max(0, 1 - (E_ii + F_itc))                       (Eq. 4);

then S_skip += w1 * S_sa + w2 * SLC_sel(l) (float64) and, once S_skip reaches
T_skip, the token bypasses sub-layer m(l) from layer l (inclusive) to the
last layer (Eq. 6, Algorithm 1).  Layer l's forward runs after its
admissions.  Text rows never skip.

The ablations of the skip rule (Tab. 8), selected by ``variant`` bits (the
readings are the ones the paper's ablation text gives):

* NO_EII: the retention score is F_itc alone, S_sa = max(0, 1 - F_itc);
* NO_FITC: the retention score is E_ii alone, S_sa = max(0, 1 - E_ii);
* NO_ACCUM: no accumulation, S_skip(i, l) = S_fuse(i, l) (each layer's score
  is tested against T_skip on its own);
* WHOLE_LAYER (without SLC): S_fuse = w1 * S_sa (no SLC term) and an admitted
  token bypasses both sub-layers of every remaining layer.

Parity pins: with w1 = 0 the result equals Algorithm 1's plan with the same
SLC tables followed by the plain prefill; with all decoder weights zero the
hidden states never change, so the crossing layer follows by hand from the
closed-form E_ii and F_itc (for every variant).
"""
from __future__ import annotations

import numpy as np

from .asl_skip import SKIP_ATTN_BIT, SKIP_FFN_BIT, ATTN, entropy_norm, itc, skippability
from .bf16 import round_bf16
from .decoder import layer_forward

NO_EII, NO_FITC, NO_ACCUM, WHOLE_LAYER = 1, 2, 4, 8


def prefill_online(x, weights, cu_seqlens, n_text, W_unembed, slc_sel, m, w1, w2, T_skip, cfg,
                   recipe="bf16", dtype=np.float64, variant=0):
    """Returns (h [rows, d], codes [L, rows] uint8, admit [rows] int (-1 = never), S_sa [W, rows])."""
    get = weights if callable(weights) else (lambda l: weights[l])
    cu = np.asarray(cu_seqlens, np.int64)
    h = np.asarray(x, dtype=dtype).copy()
    rows = h.shape[0]
    L = cfg.L
    W = L // 2
    rnd = round_bf16 if recipe == "bf16" else (lambda t: t)
    slc_sel = np.asarray(slc_sel, np.float64)
    m = np.asarray(m)
    codes = np.zeros((L, rows), np.uint8)
    admit = np.full(rows, -1, np.int64)
    acc = np.zeros(rows, np.float64)
    S_tab = np.zeros((W, rows), np.float64)
    for l in range(L):
        if l < W:
            for b in range(len(cu) - 1):
                s0, s1 = int(cu[b]), int(cu[b + 1])
                n_vis = (s1 - s0) - n_text
                cand = [i for i in range(s0, s0 + n_vis) if admit[i] < 0]
                if not cand:
                    continue
                E = entropy_norm(np.asarray(rnd(h[cand]), np.float64), W_unembed)
                F = itc(h[cand], h[s0 + n_vis:s1])
                S = skippability(np.zeros_like(E) if variant & NO_EII else E,
                                 np.zeros_like(F) if variant & NO_FITC else F)
                slc_term = 0.0 if variant & WHOLE_LAYER else float(w2) * float(slc_sel[l])
                for t, i in enumerate(cand):
                    S_tab[l, i] = S[t]
                    fuse = float(w1) * float(S[t]) + slc_term
                    acc[i] = fuse if variant & NO_ACCUM else acc[i] + fuse
                    if acc[i] >= float(T_skip):
                        admit[i] = l
                        if variant & WHOLE_LAYER:
                            codes[l:, i] |= SKIP_ATTN_BIT | SKIP_FFN_BIT
                        else:
                            codes[l:, i] |= SKIP_ATTN_BIT if int(m[l]) == ATTN else SKIP_FFN_BIT
        h = layer_forward(h, get(l), cu, codes[l], cfg, recipe, dtype)
    return h, codes, admit, S_tab
