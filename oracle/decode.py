"""Autoregressive decoding over the pruned and skipped KV cache, and the LM head
(Algorithm 1 ends with the LM head on the prefill's last state; Sec. 5
measures decode latency over the cache the pruned prefill leaves).

Test infrastructure (the oracle), not part of the product path.

A decode step appends one token (its input row) to every sample.  Causal
attention makes the new token's state depend only on the rows before it, and
their keys and values are those the prefill computed, so the step is defined
as the skip-aware prefill over the extended sequence (prompt rows with their
bypass codes, generated rows never bypassing), read at the new rows.  The LM
head is W_unembed RMSNorm(h; final_norm); the next token is the arg max, ties
to the lowest id.  With the bf16 recipe the normalised row is rounded to bf16
(the GEMM operand).
"""
from __future__ import annotations

import numpy as np

from .bf16 import round_bf16
from .decoder import prefill, rmsnorm


def extend(x, cu_seqlens, codes, new_rows):
    """Packs every sample's prompt rows followed by its generated rows.

    ``new_rows[b]`` is [t, d] (the inputs of sample b's generated tokens, in
    order).  Returns (x_ext, cu_ext, codes_ext, rows of the generated tokens
    per sample in the packed layout)."""
    cu = np.asarray(cu_seqlens, np.int64)
    codes = np.asarray(codes, np.uint8)
    L = codes.shape[0]
    parts, cparts, cu_ext, where = [], [], [0], []
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        nb = np.asarray(new_rows[b], dtype=np.float64).reshape(-1, x.shape[1])
        parts += [np.asarray(x[s0:s1], np.float64), nb]
        cparts += [codes[:, s0:s1], np.zeros((L, len(nb)), np.uint8)]
        start = cu_ext[-1] + (s1 - s0)
        where.append(np.arange(start, start + len(nb)))
        cu_ext.append(start + len(nb))
    return (np.concatenate(parts, axis=0), np.asarray(cu_ext, np.int64),
            np.concatenate(cparts, axis=1), where)


def decode(x, weights, cu_seqlens, codes, new_rows, cfg, recipe="bf16", n_layers=None, kv=None):
    """States after the last layer of the generated rows: list per sample of [t, d]."""
    xe, cue, ce, where = extend(x, cu_seqlens, codes, new_rows)
    h = prefill(xe, weights, cue, ce, cfg, recipe=recipe, n_layers=n_layers, kv=kv)
    return [h[w] for w in where], (xe, cue, ce, where)


def lm_head(h, final_norm, W_unembed, eps, recipe="bf16"):
    """Logits [rows, V] of states h [rows, d]: W_unembed RMSNorm(h; final_norm)."""
    rnd = round_bf16 if recipe == "bf16" else (lambda t: t)
    xn = rnd(rmsnorm(np.asarray(h, np.float64), np.asarray(final_norm, np.float64), eps))
    return np.asarray(xn, np.float64) @ np.asarray(W_unembed, np.float64).T


def next_tokens(logits):
    """Greedy choice: arg max per row, ties to the lowest id."""
    return np.argmax(np.asarray(logits), axis=-1)
