"""Inputs of the online skip controller: decoder input rows and an unembedding.

With random-init weights the logit lens of a plain N(0, 0.02) hidden state is
close to uniform (normalised entropy about 1) for every token, so the online
skippability max(0, 1 - (E + F)) would be 0 everywhere.  These inputs give
the controller something to decide instead:

* per sample b a random unit direction u_b; text rows are
  0.5 sqrt(d) (0.7 u_b + 0.7 n) with n a random unit vector;
* visual row i is 0.5 sqrt(d) s_i (c_i u_b + sqrt(1 - c_i^2) n_i) with n_i a
  random unit vector orthogonal to u_b, a scale s_i log-uniform in [1/4, 4]
  (the lens temperature: larger rows give sharper, lower-entropy softmaxes)
  and an alignment c_i uniform in [-0.9, 0.5] (its similarity to the text);
* the unembedding matrix [V, d] is N(0, (3.2 / sqrt(d))^2), so a row with
  s = 1 has logits of standard deviation about 1.6.

Decoder weights stay as in ``decoder_inputs``.  Rows are drawn in fp64 from
PCG64 and rounded once to the workload's dtype (bf16 by round-to-nearest-even).
"""
from __future__ import annotations

import numpy as np
import torch

from .configs import DecoderCfg
from .counter_rng import f32_to_bf16_rne, normal_bf16, normal_f32
from .vision import rng


def _unit(v: np.ndarray) -> np.ndarray:
    return v / np.linalg.norm(v)


def decoder_rows(dec: DecoderCfg, cu_seqlens, n_text: int, seed: int = 0) -> torch.Tensor:
    """[rows, d] CPU tensor in the workload dtype: per sample visual rows then n_text text rows."""
    cu = np.asarray(cu_seqlens, np.int64)
    d = dec.d
    x = np.zeros((int(cu[-1]), d), np.float64)
    base = 0.5 * np.sqrt(d)
    for b in range(len(cu) - 1):
        g = rng(seed, 4300 + b)
        s0, s1 = int(cu[b]), int(cu[b + 1])
        n_vis = s1 - s0 - n_text
        u = _unit(g.standard_normal(d))
        for i in range(n_vis):
            s = np.exp(g.uniform(np.log(0.25), np.log(4.0)))
            c = g.uniform(-0.9, 0.5)
            n = g.standard_normal(d)
            n = _unit(n - (n @ u) * u)
            x[s0 + i] = base * s * (c * u + np.sqrt(1.0 - c * c) * n)
        for j in range(n_text):
            x[s0 + n_vis + j] = base * (0.7 * u + 0.7 * _unit(g.standard_normal(d)))
    t = torch.from_numpy(x.astype(np.float32))
    return f32_to_bf16_rne(t) if dec.dtype == "bf16" else t


def unembed_std(d: int) -> float:
    return 3.2 / float(np.sqrt(d))


def unembed(dec: DecoderCfg, V: int, seed: int = 0, device="cpu") -> torch.Tensor:
    """[V, d] unembedding matrix in the workload dtype (counter generator, any device)."""
    if dec.dtype == "bf16":
        return normal_bf16((V, dec.d), seed, 4200, unembed_std(dec.d), device=device)
    return normal_f32((V, dec.d), seed, 4200, unembed_std(dec.d), device=device)
