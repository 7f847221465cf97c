"""ASL-Skip (Sec. 4.2-4.3, Algorithm 1 stage 2): which visual rows bypass which sub-layer.

* ``entropy_norm``  - Sec. 4.2.1 (1): Shannon entropy of softmax(h W_unembed^T),
  normalised to [0, 1] by dividing by ln|V| (reading: the maximum entropy).
* ``itc``           - Sec. 4.2.1 (2): cosine of the visual hidden state with the
  mean text state, mapped to [0, 1] as (1 + cos) / 2 (reading).
* ``skippability``  - Eq. 4: S_sa = ReLU(1 - (E_ii + F_itc)).
* ``slc_normalize`` - Eq. 5, per module family, epsilon 1e-8 (reading).
* ``skip_targets``  - Sec. 4.2.2: m(l) = the module with the larger normalised
  score (ties go to attention, which the paper finds more redundant).
* ``plan``          - Eq. 6 and Algorithm 1: for layers l inside the decision
  window (0-indexed l < floor(L/2), i.e. 1-indexed l <= L/2) every visual
  token not yet in skip mode accumulates S_fuse = w1*S_sa + w2*SLC_norm(l);
  once the sum reaches T_skip (">=", as in Algorithm 1) the token enters
  skip mode with target m(l) frozen, and bypasses that sub-layer from layer
  l (inclusive) to the last layer.  Text rows never skip.
  Accumulation is in float64.

Parity pins: hand-worked tables with known crossing layers, the frozen-target
and window rules, and the Table 10 lists reproduced through Eq. 5.
"""
from __future__ import annotations

import numpy as np

ATTN, FFN = 0, 1
SKIP_ATTN_BIT, SKIP_FFN_BIT = 1, 2


def entropy_norm(h: np.ndarray, W_unembed: np.ndarray) -> np.ndarray:
    """E_ii per row of h [rows, d] against W_unembed [V, d]."""
    logits = np.asarray(h, np.float64) @ np.asarray(W_unembed, np.float64).T
    logits = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(logits)
    p /= p.sum(axis=1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore"):
        ent = -np.where(p > 0, p * np.log(p), 0.0).sum(axis=1)
    return ent / np.log(W_unembed.shape[0])


def itc(h_vis: np.ndarray, h_text: np.ndarray) -> np.ndarray:
    """F_itc per visual row: (1 + cos(h_i, mean of text rows)) / 2."""
    q = np.asarray(h_text, np.float64).mean(axis=0)
    hv = np.asarray(h_vis, np.float64)
    num = hv @ q
    den = np.linalg.norm(hv, axis=1) * np.linalg.norm(q)
    cos = np.where(den > 0, num / np.where(den > 0, den, 1.0), 0.0)
    return (1.0 + cos) / 2.0


def skippability(E_ii, F_itc) -> np.ndarray:
    """Eq. 4."""
    return np.maximum(0.0, 1.0 - (np.asarray(E_ii, np.float64) + np.asarray(F_itc, np.float64)))


def slc_normalize(slc_attn, slc_ffn, eps: float = 1e-8):
    """Eq. 5 for both module families; returns (norm_attn [L], norm_ffn [L]) float64."""
    out = []
    for v in (slc_attn, slc_ffn):
        v = np.asarray(v, np.float64)
        out.append(1.0 - (v - v.min()) / (v.max() - v.min() + eps))
    return out[0], out[1]


def skip_targets(norm_attn, norm_ffn):
    """Per-layer target m(l) (0 = attention, 1 = FFN) and its normalised score."""
    norm_attn = np.asarray(norm_attn, np.float64)
    norm_ffn = np.asarray(norm_ffn, np.float64)
    m = np.where(norm_ffn > norm_attn, FFN, ATTN).astype(np.uint8)
    sel = np.where(m == FFN, norm_ffn, norm_attn)
    return m, sel


def plan(S_sa: np.ndarray, slc_sel, m, w1: float, w2: float, T_skip: float, L: int):
    """Algorithm 1 admission rule for one sample.

    ``S_sa`` is [W, n_vis] (W >= floor(L/2) decision-window layers).
    Returns (codes [L, n_vis] uint8, admit_layer [n_vis] (-1 = never),
    target [n_vis] (-1 = none)).
    """
    S_sa = np.asarray(S_sa)
    n_vis = S_sa.shape[1]
    W = L // 2
    slc_sel = np.asarray(slc_sel, np.float64)
    m = np.asarray(m)
    acc = np.zeros(n_vis, np.float64)
    admit = np.full(n_vis, -1, np.int64)
    target = np.full(n_vis, -1, np.int64)
    for l in range(W):
        for i in range(n_vis):
            if admit[i] >= 0:
                continue
            acc[i] = acc[i] + (float(w1) * float(S_sa[l, i]) + float(w2) * float(slc_sel[l]))
            if acc[i] >= float(T_skip):
                admit[i] = l
                target[i] = int(m[l])
    codes = np.zeros((L, n_vis), np.uint8)
    for i in range(n_vis):
        if admit[i] >= 0:
            bit = SKIP_ATTN_BIT if target[i] == ATTN else SKIP_FFN_BIT
            codes[admit[i]:, i] |= bit
    return codes, admit, target


def pack_codes(per_sample_codes, n_vis, n_text, L: int) -> np.ndarray:
    """Per-sample [L, >= n_vis[b]] codes -> packed [L, rows]; text rows get 0."""
    cols = []
    for b, c in enumerate(per_sample_codes):
        cols.append(np.asarray(c, np.uint8)[:, :n_vis[b]])
        cols.append(np.zeros((L, n_text), np.uint8))
    return np.concatenate(cols, axis=1)
