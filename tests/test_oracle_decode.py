"""Pins of the oracle's decode step and LM head (Algorithm 1's LM head; decoding
over the KV cache the pruned and skipped prefill leaves)."""
import dataclasses

import numpy as np
import pytest

from oracle import decode as od
from oracle import decoder as odec
from synth import get_workload
from synth.decoder_inputs import layer_weights


def _tiny(L=2):
    dec = dataclasses.replace(get_workload("tiny").dec, L=L)
    W = [{k: v.numpy().astype(np.float64) for k, v in layer_weights(dec, l, 0).items()} for l in range(L)]
    return dec, W


def test_kv_cache_closed_form_with_identity_projections():
    dec = dataclasses.replace(get_workload("tiny").dec, L=1)
    d, H = dec.d, dec.H
    dh, half = d // H, d // H // 2
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, d))
    w = {"attn_norm": np.ones(d), "ffn_norm": np.ones(d), "wq": np.eye(d), "wk": np.eye(d), "wv": np.eye(d),
         "wo": np.zeros((d, d)), "wg": np.zeros((dec.d_ff, d)), "wu": np.zeros((dec.d_ff, d)),
         "wd": np.zeros((d, dec.d_ff))}
    kv = []
    odec.prefill(x, [w], [0, 5], np.zeros((1, 5), np.uint8), dec, recipe="f32", kv=kv)
    K, V = kv[0]
    xn = x / np.sqrt((x * x).mean(axis=1, keepdims=True) + dec.eps)
    assert np.allclose(V, xn, rtol=0, atol=1e-14)
    # keys: each head's pair (i, i + half) rotated as a complex number by p * theta^(-2i/dh)
    for p in range(5):
        for h in range(H):
            seg = xn[p, h * dh:(h + 1) * dh]
            z = (seg[:half] + 1j * seg[half:]) * np.exp(1j * p * dec.theta ** (-2.0 * np.arange(half) / dh))
            assert np.allclose(K[p, h * dh:h * dh + half], z.real, atol=1e-13)
            assert np.allclose(K[p, h * dh + half:(h + 1) * dh], z.imag, atol=1e-13)


def test_a_generated_token_does_not_depend_on_later_ones():
    dec, W = _tiny()
    rng = np.random.default_rng(1)
    x = rng.standard_normal((12, dec.d)) * 0.5
    codes = np.zeros((dec.L, 12), np.uint8)
    codes[:, 2:5] = 1
    t1, t2 = rng.standard_normal((1, dec.d)), rng.standard_normal((1, dec.d))
    h1, _ = od.decode(x, W, [0, 12], codes, [t1], dec, recipe="f32")
    h12, _ = od.decode(x, W, [0, 12], codes, [np.vstack([t1, t2])], dec, recipe="f32")
    assert np.allclose(h1[0][0], h12[0][0], rtol=0, atol=1e-12)


def test_samples_decode_independently_and_prompt_cache_is_unchanged():
    dec, W = _tiny()
    rng = np.random.default_rng(2)
    x = rng.standard_normal((20, dec.d)) * 0.5
    codes = (rng.random((dec.L, 20)) < 0.3).astype(np.uint8) * 3
    codes[:, 6:9] = 0
    codes[:, 17:20] = 0
    cu = [0, 9, 20]
    new = [rng.standard_normal((2, dec.d)), rng.standard_normal((3, dec.d))]
    kv_both = []
    hb, (_, cue, _, where) = od.decode(x, W, cu, codes, new, dec, recipe="f32", kv=kv_both)
    for b in range(2):
        s0, s1 = cu[b], cu[b + 1]
        ha, _ = od.decode(x[s0:s1], W, [0, s1 - s0], codes[:, s0:s1], [new[b]], dec, recipe="f32")
        assert np.allclose(hb[b], ha[0], rtol=0, atol=1e-12)
    kv_prompt = []
    odec.prefill(x, W, cu, codes, dec, recipe="f32", kv=kv_prompt)
    rows = np.r_[0:9, 11:22]     # prompt rows inside the extended packing
    for (ke, ve), (kp, vp) in zip(kv_both, kv_prompt):
        assert np.allclose(ke[rows], kp, rtol=0, atol=1e-12) and np.allclose(ve[rows], vp, rtol=0, atol=1e-12)
    assert list(cue) == [0, 11, 25]


def test_prompt_rows_keep_their_bypass_and_generated_rows_never_bypass():
    dec, W = _tiny()
    rng = np.random.default_rng(3)
    x = rng.standard_normal((8, dec.d)) * 0.5
    codes = np.zeros((dec.L, 8), np.uint8)
    codes[:, 3] = 3
    xe, cue, ce, where = od.extend(x, [0, 8], codes, [rng.standard_normal((2, dec.d))])
    assert np.all(ce[:, 8:] == 0) and np.all(ce[:, 3] == 3)
    h = odec.prefill(xe, W, cue, ce, dec, recipe="f32")
    assert np.array_equal(h[3], xe[3])


def test_lm_head_identity_unembedding_picks_the_largest_component():
    d = 16
    rng = np.random.default_rng(4)
    h = rng.standard_normal((3, d))
    logits = od.lm_head(h, np.ones(d), np.eye(d), 1e-5, recipe="f32")
    scale = 1.0 / np.sqrt((h * h).mean(axis=1, keepdims=True) + 1e-5)
    assert np.allclose(logits, h * scale, rtol=0, atol=1e-14)
    assert list(od.next_tokens(logits)) == list(np.argmax(h, axis=1))
    tie = np.zeros((1, d))
    tie[0, 5] = tie[0, 2] = 1.0
    assert od.next_tokens(od.lm_head(tie, np.ones(d), np.eye(d), 1e-5, recipe="f32"))[0] == 2
