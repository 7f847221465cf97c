"""Pin of the oracle's bf16 precision recipe (where values are rounded to bfloat16).

The paper fixes no precision; the recipe is a reading: weights and inputs are
bf16, the residual stream is fp32, and a value is rounded to bf16 exactly
where a bf16 inference engine stores it as a GEMM operand or a kept
activation: the RMSNorm outputs, Q and K after RoPE, V, the attention output,
silu(g) * u, the LM head's normalised row and the logit lens's operand.  GEMM
accumulations, softmax and the residual additions stay in full precision.

The pin is an independent composition of the same block from library
primitives (torch.nn.functional in float64: rms_norm, linear, rotary
embedding as a complex rotation, scaled_dot_product_attention with a packed
causal mask, silu; bf16 through torch's own float32 -> bfloat16 cast) with
the casts placed at exactly those points.  It must agree with the oracle to
1e-12 relative, i.e. no bf16 rounding may differ.  The mutation tests then
plant single mistakes in the oracle (on the CPU): each rounding dropped in
turn, Q or K rounded before RoPE instead of after, V left unrounded, the lens
or LM-head operand unrounded.  Every mutant must miss the pin by far more than
the tolerance, so a misplaced rounding cannot pass.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decode as odecode
from oracle import decoder as odec
from oracle import online as oonline
from synth.configs import DecoderCfg
from synth.vision import rng

TOL = 1e-12
# the smallest miss a planted mistake must produce (a bf16 step is 2^-8 relative)
MISS = 1e-6

CFGS = {
    # the tiny decoder's shape (dh = 32) and one 512-wide slice with the 7B head size (dh = 128)
    "tiny_d128": DecoderCfg(L=2, d=128, H=4, d_ff=344, dtype="bf16"),
    "slice_d512": DecoderCfg(L=2, d=512, H=4, d_ff=1376, dtype="bf16"),
}


def _bf16(t: torch.Tensor) -> torch.Tensor:
    """Round to bfloat16 by torch's own cast (float64 -> float32 -> bfloat16), back to float64."""
    return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)


def _weights(cfg: DecoderCfg, seed: int):
    """bf16-valued weights (N(0, 0.02) rounded by torch), norm weights near 1."""
    out = []
    for l in range(cfg.L):
        r = rng(seed, 900 + l)
        d, f = cfg.d, cfg.d_ff
        w = {}
        for name, shape in (("wq", (d, d)), ("wk", (d, d)), ("wv", (d, d)), ("wo", (d, d)),
                            ("wg", (f, d)), ("wu", (f, d)), ("wd", (d, f))):
            w[name] = _bf16(torch.from_numpy(r.standard_normal(shape) * 0.02)).numpy()
        w["attn_norm"] = 1.0 + 0.1 * r.standard_normal(d)
        w["ffn_norm"] = 1.0 + 0.1 * r.standard_normal(d)
        out.append(w)
    return out


def _inputs(cfg: DecoderCfg, seed: int):
    """Two packed samples with per-row bypass codes (attention, FFN, both, none)."""
    r = rng(seed, 950)
    cu = np.array([0, 37, 90])
    x = _bf16(torch.from_numpy(r.standard_normal((90, cfg.d)) * 0.5)).numpy()
    codes = np.zeros((cfg.L, 90), np.uint8)
    codes[0, 3:12] = 1
    codes[1, 40:55] = 2
    codes[1, 5:8] = 3
    return x, cu, codes


def _rope_complex(x: torch.Tensor, pos: torch.Tensor, theta: float) -> torch.Tensor:
    """Rotary embedding of x [rows, H, dh] as a rotation of the complex numbers
    x[c] + i x[c + dh/2] by pos * theta^(-2c/dh)."""
    dh = x.shape[-1]
    half = dh // 2
    freq = 1.0 / torch.pow(torch.tensor(theta, dtype=torch.float64),
                           torch.arange(0, dh, 2, dtype=torch.float64) / dh)
    z = torch.complex(x[..., :half], x[..., half:])
    rot = torch.polar(torch.ones_like(freq)[None, :] * 1.0, pos[:, None].to(torch.float64) * freq[None, :])
    y = z * rot[:, None, :]
    return torch.cat([y.real, y.imag], dim=-1)


def _packed_causal_mask(cu) -> tuple:
    rows = int(cu[-1])
    seg = torch.zeros(rows, dtype=torch.int64)
    pos = torch.zeros(rows, dtype=torch.int64)
    for b in range(len(cu) - 1):
        seg[cu[b]:cu[b + 1]] = b
        pos[cu[b]:cu[b + 1]] = torch.arange(int(cu[b + 1] - cu[b]))
    idx = torch.arange(rows)
    mask = (seg[:, None] == seg[None, :]) & (idx[None, :] <= idx[:, None])
    return mask, pos


def _layer_independent(h, w, cu, code_row, cfg):
    """One block of the recipe from torch.nn.functional primitives (float64)."""
    d, H = cfg.d, cfg.H
    dh = d // H
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    h = t(h)
    rows = h.shape[0]
    mask, pos = _packed_causal_mask(cu)
    code = torch.from_numpy(np.asarray(code_row, np.uint8).astype(np.int64))

    xn = _bf16(F.rms_norm(h, (d,), weight=t(w["attn_norm"]), eps=cfg.eps))
    q = F.linear(xn, t(w["wq"])).view(rows, H, dh)
    k = F.linear(xn, t(w["wk"])).view(rows, H, dh)
    v = F.linear(xn, t(w["wv"])).view(rows, H, dh)
    q = _bf16(_rope_complex(q, pos, cfg.theta))
    k = _bf16(_rope_complex(k, pos, cfg.theta))
    v = _bf16(v)
    o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                       attn_mask=mask, scale=1.0 / math.sqrt(dh))
    o = _bf16(o.transpose(0, 1).reshape(rows, d))
    h = torch.where((code & 1).bool()[:, None], h, h + F.linear(o, t(w["wo"])))

    xn = _bf16(F.rms_norm(h, (d,), weight=t(w["ffn_norm"]), eps=cfg.eps))
    act = _bf16(F.silu(F.linear(xn, t(w["wg"]))) * F.linear(xn, t(w["wu"])))
    h = torch.where((code & 2).bool()[:, None], h, h + F.linear(act, t(w["wd"])))
    return h.numpy()


def _rel(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b))) / np.max(np.abs(np.asarray(b))))


def _oracle_two_layers(cfg, W, x, cu, codes):
    return odec.prefill(x, W, cu, codes, cfg, recipe="bf16")


def _independent_two_layers(cfg, W, x, cu, codes):
    h = np.asarray(x, np.float64)
    for l in range(cfg.L):
        h = _layer_independent(h, W[l], cu, codes[l], cfg)
    return h


@pytest.fixture(scope="module", params=list(CFGS))
def case(request):
    cfg = CFGS[request.param]
    W = _weights(cfg, 3)
    x, cu, codes = _inputs(cfg, 3)
    ref = _independent_two_layers(cfg, W, x, cu, codes)
    return cfg, W, x, cu, codes, ref


def test_decoder_recipe_matches_independent_composition(case):
    cfg, W, x, cu, codes, ref = case
    got = _oracle_two_layers(cfg, W, x, cu, codes)
    assert _rel(got, ref) <= TOL
    # the recipe is not vacuous here: without any rounding the result moves far
    plain = odec.prefill(x, W, cu, codes, cfg, recipe="f32")
    assert _rel(plain, ref) > 100 * MISS


class _DropNth:
    """round_bf16 stand-in that leaves the n-th call of every layer unrounded."""

    def __init__(self, real, n, per_layer):
        self.real, self.n, self.per_layer, self.calls = real, n, per_layer, 0

    def __call__(self, v):
        i = self.calls % self.per_layer
        self.calls += 1
        return np.asarray(v, np.float64) if i == self.n else self.real(v)


# the oracle's rounding points in one layer, in call order
POINTS = ("attn_norm_out", "q_after_rope", "k_after_rope", "v", "attn_out", "ffn_norm_out", "silu_g_u")


@pytest.mark.parametrize("point", range(len(POINTS)), ids=POINTS)
def test_each_dropped_rounding_misses_the_pin(case, point, monkeypatch):
    cfg, W, x, cu, codes, ref = case
    real = odec.round_bf16
    counter = _DropNth(real, point, len(POINTS))
    monkeypatch.setattr(odec, "round_bf16", counter)
    got = _oracle_two_layers(cfg, W, x, cu, codes)
    assert counter.calls == len(POINTS) * cfg.L   # every point was reached
    assert _rel(got, ref) > MISS


@pytest.mark.parametrize("which", ["q", "k"])
def test_rounding_before_rope_misses_the_pin(case, which, monkeypatch):
    """Q (or K) rounded before the rotation instead of after it."""
    cfg, W, x, cu, codes, ref = case
    real_round, real_rope = odec.round_bf16, odec.rope
    n = POINTS.index(f"{which}_after_rope")
    monkeypatch.setattr(odec, "round_bf16", _DropNth(real_round, n, len(POINTS)))
    calls = {"i": 0}

    def rope_rounding_input(t, pos, theta):
        i = calls["i"]
        calls["i"] += 1
        target = 0 if which == "q" else 1
        return real_rope(real_round(t) if i % 2 == target else t, pos, theta)

    monkeypatch.setattr(odec, "rope", rope_rounding_input)
    got = _oracle_two_layers(cfg, W, x, cu, codes)
    assert _rel(got, ref) > MISS


# ------------------------------------------------------------------ LM head
def _lm_case():
    r = rng(5, 960)
    d, V = 512, 640
    h = r.standard_normal((6, d)) * 0.7
    fn = 1.0 + 0.1 * r.standard_normal(d)
    Wu = _bf16(torch.from_numpy(r.standard_normal((V, d)) * 0.05)).numpy()
    return h, fn, Wu


def _lm_independent(h, fn, Wu, eps=1e-5):
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    xn = _bf16(F.rms_norm(t(h), (h.shape[1],), weight=t(fn), eps=eps))
    return F.linear(xn, t(Wu)).numpy()


def test_lm_head_recipe_matches_independent_composition(monkeypatch):
    h, fn, Wu = _lm_case()
    ref = _lm_independent(h, fn, Wu)
    assert _rel(odecode.lm_head(h, fn, Wu, 1e-5, recipe="bf16"), ref) <= TOL
    monkeypatch.setattr(odecode, "round_bf16", lambda v: np.asarray(v, np.float64))
    assert _rel(odecode.lm_head(h, fn, Wu, 1e-5, recipe="bf16"), ref) > MISS


# ------------------------------------------------------------------ logit lens operand
def _lens_case():
    r = rng(6, 970)
    d, V, n_text = 128, 384, 8
    cfg = DecoderCfg(L=2, d=d, H=4, d_ff=344, dtype="bf16")
    x = r.standard_normal((40, d)) * 0.8
    Wu = _bf16(torch.from_numpy(r.standard_normal((V, d)) * (3.0 / math.sqrt(d)))).numpy()
    return cfg, x, np.array([0, 40]), n_text, Wu


def _s_sa_independent(x, cu, n_text, Wu):
    """S_sa at the first window layer: E_ii from the lens on bf16(h), F_itc from the fp32 h."""
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    h = t(x)
    n_vis = int(cu[1]) - n_text
    vis, text = h[:n_vis], h[n_vis:int(cu[1])]
    logp = F.log_softmax(F.linear(_bf16(vis), t(Wu)), dim=-1)
    E = -(logp.exp() * logp).sum(-1) / math.log(Wu.shape[0])
    Fi = (1.0 + F.cosine_similarity(vis, text.mean(0, keepdim=True), dim=-1, eps=0.0)) / 2.0
    return torch.clamp(1.0 - (E + Fi), min=0.0).numpy()


def test_lens_operand_recipe_matches_independent_composition(monkeypatch):
    cfg, x, cu, n_text, Wu = _lens_case()
    W = _weights(cfg, 4)
    ref = _s_sa_independent(x, cu, n_text, Wu)
    n_vis = int(cu[1]) - n_text
    sel = np.zeros(cfg.L)
    tgt = np.zeros(cfg.L, np.uint8)
    # a threshold nobody reaches: S_sa is recorded for every visual row at layer 0
    _, _, _, S = oonline.prefill_online(x, W, cu, n_text, Wu, sel, tgt, 1.0, 0.0, 1e9, cfg, recipe="bf16")
    assert np.max(np.abs(S[0, :n_vis] - ref)) <= TOL
    assert np.max(ref) > 0.05          # rows with a positive skippability exist
    monkeypatch.setattr(oonline, "round_bf16", lambda v: np.asarray(v, np.float64))
    _, _, _, S2 = oonline.prefill_online(x, W, cu, n_text, Wu, sel, tgt, 1.0, 0.0, 1e9, cfg, recipe="bf16")
    assert np.max(np.abs(S2[0, :n_vis] - ref)) > MISS
