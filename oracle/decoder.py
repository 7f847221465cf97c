"""LLaMA-style decoder prefill with per-row sub-layer bypass (Sec. 3.2, Alg. 1 stage 2).

The paper does not spell out the decoder (it is the LLaVA language model);
the reading used is the textbook LLaMA block:

    h <- h + Attn(RMSNorm(h))     unless the row bypasses attention here
    h <- h + FFN(RMSNorm(h))      unless the row bypasses the FFN here

with RMSNorm(x) = x / sqrt(mean(x^2) + eps) * w, rotary position embedding
(rotate-half pairing (i, i + dh/2), inverse frequency theta^(-2i/dh)) on
queries and keys, multi-head causal softmax attention with scale 1/sqrt(dh),
SwiGLU FFN W_down(silu(W_gate x) * W_up x), no biases.  Rows are packed
samples ([kept visual | text] each, cu_seqlens boundaries); positions restart
at 0 in every sample and attention never crosses samples.

VSkip-Attn (Sec. 3.2): a bypassing row is not a query (its hidden state gets
no attention update) but still serves as key and value; its K/V come from
its current hidden state.  VSkip-FFN: the row's FFN update is dropped.  The
oracle computes every sub-layer densely for all rows and then discards the
bypassed rows' updates, so a bypassed row keeps its input bit for bit.

Precision recipes: ``"f32"`` rounds nothing (all float64 here); ``"bf16"``
rounds to bfloat16 (via float32) the RMSNorm outputs, Q/K after RoPE and V,
the attention output, and silu(g)*u; the residual h, GEMM accumulations and
softmax are not rounded.  Codes: bit 0 = bypass attention, bit 1 = bypass FFN.

Parity pins: the dense forward (no bypass) against Hugging Face's
``LlamaModel`` run independently on the same weights; RoPE's relative-position
invariance; bypass semantics via rows that keep their input exactly and via
text rows that are unaffected by other rows' attention bypass.
"""
from __future__ import annotations

import math

import numpy as np

from .bf16 import round_bf16


def rmsnorm(h: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    return h / np.sqrt((h * h).mean(axis=-1, keepdims=True) + eps) * w


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """x [S, H, dh]; rotate-half RoPE at integer positions pos [S]."""
    dh = x.shape[-1]
    half = dh // 2
    inv = theta ** (-(2.0 * np.arange(half)) / dh)
    ang = pos.astype(np.float64)[:, None] * inv[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _positions(cu: np.ndarray) -> np.ndarray:
    pos = np.zeros(int(cu[-1]), np.int64)
    for b in range(len(cu) - 1):
        pos[cu[b]:cu[b + 1]] = np.arange(cu[b + 1] - cu[b])
    return pos


def attention(q, k, v, cu) -> np.ndarray:
    """Causal multi-head attention inside each sample; q/k/v [rows, H, dh]."""
    rows, H, dh = q.shape
    out = np.zeros_like(q)
    scale = 1.0 / math.sqrt(dh)
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        S = s1 - s0
        if S == 0:
            continue
        causal = np.tril(np.ones((S, S), dtype=bool))
        for hh in range(H):
            logits = (q[s0:s1, hh] @ k[s0:s1, hh].T) * scale
            logits = np.where(causal, logits, -np.inf)
            logits -= logits.max(axis=1, keepdims=True)
            p = np.exp(logits)
            p /= p.sum(axis=1, keepdims=True)
            out[s0:s1, hh] = p @ v[s0:s1, hh]
    return out


def layer_forward(h, w, cu, code_row, cfg, recipe="bf16", dtype=np.float64, kv=None):
    """One decoder layer over all packed rows; ``code_row`` [rows] uint8 bypass codes.
    ``kv`` (a list) receives this layer's keys after RoPE and values [rows, d], as
    attention used them (every row, bypassing or not)."""
    rnd = round_bf16 if recipe == "bf16" else (lambda t: t)
    L_d, H = cfg.d, cfg.H
    dh = L_d // H
    rows = h.shape[0]
    pos = _positions(cu)
    f = lambda a: np.asarray(a, dtype=dtype)
    skip_attn = (np.asarray(code_row) & 1).astype(bool)
    skip_ffn = (np.asarray(code_row) & 2).astype(bool)

    xn = f(rnd(rmsnorm(h, f(w["attn_norm"]), cfg.eps)))
    q = xn @ f(w["wq"]).T
    k = xn @ f(w["wk"]).T
    v = xn @ f(w["wv"]).T
    q = f(rnd(rope(q.reshape(rows, H, dh), pos, cfg.theta)))
    k = f(rnd(rope(k.reshape(rows, H, dh), pos, cfg.theta)))
    v = f(rnd(v.reshape(rows, H, dh)))
    if kv is not None:
        kv.append((k.reshape(rows, L_d).copy(), v.reshape(rows, L_d).copy()))
    o = f(rnd(attention(q, k, v, cu).reshape(rows, L_d)))
    upd = o @ f(w["wo"]).T
    h = np.where(skip_attn[:, None], h, h + upd)

    xn = f(rnd(rmsnorm(h, f(w["ffn_norm"]), cfg.eps)))
    g = xn @ f(w["wg"]).T
    u = xn @ f(w["wu"]).T
    act = f(rnd(silu(g) * u))
    upd = act @ f(w["wd"]).T
    h = np.where(skip_ffn[:, None], h, h + upd)
    return h


def prefill(x, weights, cu_seqlens, codes, cfg, recipe="bf16", dtype=np.float64,
            n_layers=None, kv=None):
    """Decoder prefill; returns the final residual stream h [rows, d] (before the final norm).

    ``weights`` is a list of per-layer dicts of arrays, or a callable
    ``layer -> dict`` (lets large weight sets be materialised one layer at a
    time).  ``codes`` is [L, rows] uint8.  ``kv`` (a list) receives every
    layer's (keys after RoPE, values), the KV cache a decode step reads.
    """
    get = weights if callable(weights) else (lambda l: weights[l])
    cu = np.asarray(cu_seqlens, np.int64)
    h = np.asarray(x, dtype=dtype).copy()
    L = cfg.L if n_layers is None else n_layers
    for l in range(L):
        h = layer_forward(h, get(l), cu, codes[l], cfg, recipe, dtype, kv)
    return h
