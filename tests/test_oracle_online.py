"""Pins of the online-controller prefill oracle (Sec. 4.2.1, Eq. 4, Eq. 6, Algorithm 1)."""
import math

import numpy as np
import pytest

from oracle import asl_skip as ak
from oracle import decoder as odec
from oracle.online import prefill_online
from synth import get_workload


def _tiny(L=6):
    w = get_workload("tiny", L=L)
    return w.dec


def _weights(dec, r, scale=0.1):
    out = []
    for _ in range(dec.L):
        out.append({"attn_norm": np.ones(dec.d), "ffn_norm": np.ones(dec.d),
                    "wq": r.standard_normal((dec.d, dec.d)) * scale, "wk": r.standard_normal((dec.d, dec.d)) * scale,
                    "wv": r.standard_normal((dec.d, dec.d)) * scale, "wo": r.standard_normal((dec.d, dec.d)) * scale,
                    "wg": r.standard_normal((dec.d_ff, dec.d)) * scale, "wu": r.standard_normal((dec.d_ff, dec.d)) * scale,
                    "wd": r.standard_normal((dec.d, dec.d_ff)) * scale})
    return out


def test_no_online_term_equals_plan_then_prefill():
    """w1 = 0: admission depends on the SLC tables only, i.e. Algorithm 1's plan
    with any S_sa, followed by the plain prefill."""
    dec = _tiny(8)
    r = np.random.default_rng(3)
    W = _weights(dec, r)
    cu = np.array([0, 30, 70])
    n_text = 10
    x = r.standard_normal((70, dec.d))
    WU = r.standard_normal((16, dec.d))
    sel = r.uniform(0.2, 1.0, dec.L)
    m = (r.random(dec.L) < 0.5).astype(np.uint8)
    h, codes, admit, _ = prefill_online(x, W, cu, n_text, WU, sel, m, 0.0, 1.0, 1.5, dec, recipe="f32")
    per_sample = []
    n_vis = [20, 30]
    for b in range(2):
        c, adm, _ = ak.plan(np.zeros((dec.L // 2, n_vis[b])), sel, m, 0.0, 1.0, 1.5, dec.L)
        per_sample.append(c)
    ref_codes = ak.pack_codes(per_sample, n_vis, n_text, dec.L)
    assert np.array_equal(codes, ref_codes)
    assert (codes != 0).any()
    assert np.array_equal(h, odec.prefill(x, W, cu, ref_codes, dec, recipe="f32"))


def _entropy_closed_form(z, V):
    """Normalised entropy of softmax([z, 0, ..., 0]) over V outcomes."""
    p0 = math.exp(z) / (math.exp(z) + V - 1)
    p = 1.0 / (math.exp(z) + V - 1)
    H = -p0 * math.log(p0) - (V - 1) * p * math.log(p)
    return H / math.log(V)


def test_constant_states_cross_where_the_closed_form_says():
    """Zero decoder weights keep every hidden state fixed, so S_sa is the same
    at every window layer and the crossing layer is the first l with
    (l + 1) * (w1 * S_sa + w2 * sel) >= T_skip."""
    dec = _tiny(12)
    zero = [{"attn_norm": np.ones(dec.d), "ffn_norm": np.ones(dec.d),
             "wq": np.zeros((dec.d, dec.d)), "wk": np.zeros((dec.d, dec.d)), "wv": np.zeros((dec.d, dec.d)),
             "wo": np.zeros((dec.d, dec.d)), "wg": np.zeros((dec.d_ff, dec.d)), "wu": np.zeros((dec.d_ff, dec.d)),
             "wd": np.zeros((dec.d, dec.d_ff))} for _ in range(dec.L)]
    V, c = 4, 1.0
    WU = np.zeros((V, dec.d))
    WU[0, 0] = c
    alphas = [0.0, 1.0, 2.5, 6.0, 12.0]
    n_vis, n_text = len(alphas), 3
    x = np.zeros((n_vis + n_text, dec.d))
    for i, a in enumerate(alphas):
        x[i, 0] = a            # along the lens' only nonzero direction
    x[n_vis:, 1] = 1.0         # text rows orthogonal to every visual row: cos = 0, F_itc = 1/2
    cu = np.array([0, n_vis + n_text])
    sel = np.full(dec.L, 0.25)
    m = np.array([l % 2 for l in range(dec.L)], np.uint8)
    w1, w2, T = 2.0, 1.0, 2.4
    h, codes, admit, S = prefill_online(x, zero, cu, n_text, WU, sel, m, w1, w2, T, dec, recipe="f32")
    assert np.array_equal(h, x)
    W = dec.L // 2
    for i, a in enumerate(alphas):
        s = max(0.0, 1.0 - (_entropy_closed_form(c * a, V) + 0.5))
        step = w1 * s + w2 * 0.25
        cross = math.ceil(T / step - 1e-12) - 1
        expect = cross if cross < W else -1
        assert admit[i] == expect, (i, a, s, admit[i], expect)
        if expect >= 0:
            bit = ak.SKIP_ATTN_BIT if m[expect] == ak.ATTN else ak.SKIP_FFN_BIT
            assert np.all(codes[:expect, i] == 0) and np.all(codes[expect:, i] == bit)
        assert np.allclose(S[:min(W, expect + 1 if expect >= 0 else W), i], s)
    assert np.all(codes[:, n_vis:] == 0)
    # the least peaked rows never cross inside the window
    assert admit[0] == -1 and admit[n_vis - 1] >= 0


@pytest.mark.parametrize("variant", [1, 2, 4, 8, 4 | 8, 1 | 4])
def test_skip_rule_ablations_cross_where_the_closed_form_says(variant):
    """The skip-rule ablations of Tab. 8 on constant states (zero decoder weights):
    without E_ii or F_itc the retention score is the other term alone; without
    accumulation a row is admitted at the first window layer whose own S_fuse
    reaches T_skip (here: layer 0 or never); without SLC S_fuse = w1 S_sa and an
    admitted row bypasses both sub-layers."""
    from oracle.online import NO_EII, NO_FITC, NO_ACCUM, WHOLE_LAYER
    dec = _tiny(12)
    zero = [{"attn_norm": np.ones(dec.d), "ffn_norm": np.ones(dec.d),
             "wq": np.zeros((dec.d, dec.d)), "wk": np.zeros((dec.d, dec.d)), "wv": np.zeros((dec.d, dec.d)),
             "wo": np.zeros((dec.d, dec.d)), "wg": np.zeros((dec.d_ff, dec.d)), "wu": np.zeros((dec.d_ff, dec.d)),
             "wd": np.zeros((dec.d, dec.d_ff))} for _ in range(dec.L)]
    V, c = 4, 1.0
    WU = np.zeros((V, dec.d))
    WU[0, 0] = c
    alphas = [0.0, 1.0, 2.5, 6.0, 12.0]
    n_vis, n_text = len(alphas), 3
    x = np.zeros((n_vis + n_text, dec.d))
    for i, a in enumerate(alphas):
        x[i, 0] = a
    x[n_vis:, 1] = 1.0         # cos = 0: F_itc = 1/2 for every visual row
    cu = np.array([0, n_vis + n_text])
    sel = np.full(dec.L, 0.25)
    m = np.array([l % 2 for l in range(dec.L)], np.uint8)
    w1, w2 = 2.0, 1.0
    T = (0.8 if variant & WHOLE_LAYER else 1.0) if variant & NO_ACCUM else 2.4
    h, codes, admit, S = prefill_online(x, zero, cu, n_text, WU, sel, m, w1, w2, T, dec, recipe="f32",
                                        variant=variant)
    assert np.array_equal(h, x)
    W = dec.L // 2
    for i, a in enumerate(alphas):
        E = 0.0 if variant & NO_EII else _entropy_closed_form(c * a, V)
        F = 0.0 if variant & NO_FITC else 0.5
        s = max(0.0, 1.0 - (E + F))
        step = w1 * s + (0.0 if variant & WHOLE_LAYER else w2 * 0.25)
        if variant & NO_ACCUM:
            expect = 0 if step >= T else -1
        elif step > 0:
            cross = math.ceil(T / step - 1e-12) - 1
            expect = cross if cross < W else -1
        else:
            expect = -1
        assert admit[i] == expect, (i, a, s, admit[i], expect)
        if expect >= 0:
            if variant & WHOLE_LAYER:
                bit = ak.SKIP_ATTN_BIT | ak.SKIP_FFN_BIT
            else:
                bit = ak.SKIP_ATTN_BIT if m[expect] == ak.ATTN else ak.SKIP_FFN_BIT
            assert np.all(codes[:expect, i] == 0) and np.all(codes[expect:, i] == bit)
        else:
            assert np.all(codes[:, i] == 0)
        assert np.allclose(S[:min(W, expect + 1 if expect >= 0 else W), i], s)
    assert np.all(codes[:, n_vis:] == 0)
    assert (admit >= 0).any() and (admit < 0).any() or variant & NO_EII


def test_ablation_bits_zero_is_the_paper_rule():
    dec = _tiny(8)
    r = np.random.default_rng(5)
    W = _weights(dec, r)
    cu = np.array([0, 30, 70])
    x = r.standard_normal((70, dec.d))
    WU = r.standard_normal((16, dec.d))
    sel = r.uniform(0.2, 1.0, dec.L)
    m = (r.random(dec.L) < 0.5).astype(np.uint8)
    a = prefill_online(x, W, cu, 10, WU, sel, m, 3.0, 1.0, 2.0, dec, recipe="f32")
    b = prefill_online(x, W, cu, 10, WU, sel, m, 3.0, 1.0, 2.0, dec, recipe="f32", variant=0)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
