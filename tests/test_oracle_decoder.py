"""Pins of the decoder oracle: dense forward vs Hugging Face LLaMA, RoPE, bypass semantics."""
import numpy as np
import pytest
import torch

from oracle import decoder as dec
from oracle.bf16 import round_bf16
from synth import get_workload
from synth.decoder_inputs import all_weights
from synth.vision import rng


def _tiny():
    w = get_workload("tiny")
    W = [{k: v.numpy().astype(np.float64) for k, v in lw.items()} for lw in all_weights(w.dec, 0)]
    return w, W


def _hf_dense(cfg, W, x):
    from transformers import LlamaConfig, LlamaModel
    hc = LlamaConfig(hidden_size=cfg.d, intermediate_size=cfg.d_ff, num_hidden_layers=cfg.L,
                     num_attention_heads=cfg.H, num_key_value_heads=cfg.H, rms_norm_eps=cfg.eps,
                     vocab_size=8, max_position_embeddings=4096, attention_bias=False,
                     mlp_bias=False, rope_parameters={"rope_type": "default", "rope_theta": cfg.theta})
    hc._attn_implementation = "eager"
    m = LlamaModel(hc).to(torch.float64).eval()
    with torch.no_grad():
        for l, lw in enumerate(W):
            L = m.layers[l]
            L.self_attn.q_proj.weight.copy_(torch.from_numpy(lw["wq"]))
            L.self_attn.k_proj.weight.copy_(torch.from_numpy(lw["wk"]))
            L.self_attn.v_proj.weight.copy_(torch.from_numpy(lw["wv"]))
            L.self_attn.o_proj.weight.copy_(torch.from_numpy(lw["wo"]))
            L.mlp.gate_proj.weight.copy_(torch.from_numpy(lw["wg"]))
            L.mlp.up_proj.weight.copy_(torch.from_numpy(lw["wu"]))
            L.mlp.down_proj.weight.copy_(torch.from_numpy(lw["wd"]))
            L.input_layernorm.weight.copy_(torch.from_numpy(lw["attn_norm"]))
            L.post_attention_layernorm.weight.copy_(torch.from_numpy(lw["ffn_norm"]))
        m.norm = torch.nn.Identity()
        return m(inputs_embeds=torch.from_numpy(x)[None]).last_hidden_state[0].numpy()


def test_dense_forward_matches_huggingface_llama():
    w, W = _tiny()
    x = rng(0, 11).standard_normal((48, w.dec.d)) * 0.5
    ours = dec.prefill(x, W, [0, 48], np.zeros((w.dec.L, 48), np.uint8), w.dec, recipe="f32")
    ref = _hf_dense(w.dec, W, x)
    # Hugging Face builds its rotary tables in float32 even for float64 models,
    # which bounds the agreement at about 1e-8 relative; any structural slip
    # (a sign, a pairing, a missing term) shows up at 1e-2 or more
    assert np.max(np.abs(ours - ref)) / np.max(np.abs(ref)) < 1e-6


def test_packed_samples_equal_separate_runs():
    w, W = _tiny()
    x = rng(1, 11).standard_normal((70, w.dec.d)) * 0.5
    cu = [0, 30, 70]
    ours = dec.prefill(x, W, cu, np.zeros((w.dec.L, 70), np.uint8), w.dec, recipe="f32")
    for b in range(2):
        ref = _hf_dense(w.dec, W, x[cu[b]:cu[b + 1]])
        assert np.max(np.abs(ours[cu[b]:cu[b + 1]] - ref)) < 1e-6


def test_rope_relative_position_and_norm():
    r = rng(2, 12)
    q = r.standard_normal((1, 3, 64))
    k = r.standard_normal((1, 3, 64))
    for (p, pk, c) in [(5, 2, 7), (100, 0, 33), (3, 3, 1000)]:
        a = (dec.rope(q, np.array([p]), 1e4) * dec.rope(k, np.array([pk]), 1e4)).sum(-1)
        b = (dec.rope(q, np.array([p + c]), 1e4) * dec.rope(k, np.array([pk + c]), 1e4)).sum(-1)
        assert np.allclose(a, b, atol=1e-9)
    assert np.allclose(np.linalg.norm(dec.rope(q, np.array([17]), 1e4), axis=-1),
                       np.linalg.norm(q, axis=-1))
    assert np.array_equal(dec.rope(q, np.array([0]), 1e4), q)


def test_fully_bypassed_rows_keep_their_input_exactly():
    w, W = _tiny()
    x = rng(3, 11).standard_normal((40, w.dec.d)) * 0.5
    codes = np.zeros((w.dec.L, 40), np.uint8)
    codes[:, 3:9] = 3
    for recipe in ("f32", "bf16"):
        h = dec.prefill(x, W, [0, 40], codes, w.dec, recipe=recipe)
        assert np.array_equal(h[3:9], x[3:9])


def test_attention_bypass_still_feeds_keys_and_values():
    w, W = _tiny()
    x = rng(4, 11).standard_normal((40, w.dec.d)) * 0.5
    cfg1 = w.with_layers(1).dec
    dense = dec.prefill(x, W, [0, 40], np.zeros((1, 40), np.uint8), cfg1, recipe="f32")
    codes = np.zeros((1, 40), np.uint8)
    codes[0, :24] = 1          # visual rows bypass attention in this layer
    skip = dec.prefill(x, W, [0, 40], codes, cfg1, recipe="f32")
    # text rows (queries) see the same keys/values and equal the dense result
    assert np.array_equal(skip[24:], dense[24:])
    # dropping the visual rows from the sequence instead would change the text rows
    dropped = dec.prefill(x[24:], W, [0, 16], np.zeros((1, 16), np.uint8), cfg1, recipe="f32")
    assert np.max(np.abs(dropped - dense[24:])) > 1e-3


def test_ffn_bypass_only_changes_the_bypassing_row():
    w, W = _tiny()
    x = rng(5, 11).standard_normal((20, w.dec.d)) * 0.5
    cfg1 = w.with_layers(1).dec
    dense = dec.prefill(x, W, [0, 20], np.zeros((1, 20), np.uint8), cfg1, recipe="f32")
    codes = np.zeros((1, 20), np.uint8)
    codes[0, 7] = 2
    skip = dec.prefill(x, W, [0, 20], codes, cfg1, recipe="f32")
    mask = np.arange(20) != 7
    assert np.array_equal(skip[mask], dense[mask])
    assert np.max(np.abs(skip[7] - dense[7])) > 1e-4


def test_bf16_recipe_close_to_f32():
    w, W = _tiny()
    Wb = [{k: (round_bf16(v) if k.startswith("w") else v) for k, v in lw.items()} for lw in W]
    x = round_bf16(rng(6, 11).standard_normal((48, w.dec.d)) * 0.5)
    a = dec.prefill(x, Wb, [0, 48], np.zeros((2, 48), np.uint8), w.dec, recipe="bf16")
    b = dec.prefill(x, Wb, [0, 48], np.zeros((2, 48), np.uint8), w.dec, recipe="f32")
    rel = np.max(np.abs(a - b)) / np.max(np.abs(b))
    assert 0 < rel < 2e-2


def test_round_bf16_matches_torch():
    r = rng(7, 13)
    v = np.concatenate([r.standard_normal(100000) * 10.0 ** r.integers(-20, 20, 100000),
                        np.array([0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1 + 2 ** -8)])])
    v32 = v.astype(np.float32)
    ref = torch.from_numpy(v32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(round_bf16(v32), ref)
    # ties to even
    assert round_bf16(np.float32(1 + 2 ** -8)) == 1.0
    assert round_bf16(np.float32(1 + 3 * 2 ** -8)) == 1 + 2 ** -6
    with pytest.raises(ValueError):
        round_bf16(np.array([np.inf]))
