"""The seeded input generators: determinism, distributions and shapes."""
import numpy as np
import torch

from synth import get_workload, normal_bf16, normal_f32
from synth.counter_rng import f32_to_bf16_rne, _CHUNK
from synth.vision import vision_inputs
from synth.skip_inputs import adaptive_scores, layer_mask


def test_counter_rng_deterministic_and_distinct():
    a = normal_f32((1000,), 0, 5)
    b = normal_f32((1000,), 0, 5)
    c = normal_f32((1000,), 0, 6)
    d = normal_f32((1000,), 1, 5)
    assert torch.equal(a, b)
    assert not torch.equal(a, c) and not torch.equal(a, d)


def test_counter_rng_moments():
    x = normal_f32((2_000_000,), 3, 1, std=0.02).double()
    assert abs(x.mean().item()) < 1e-4
    assert abs(x.std().item() - 0.02) < 2e-4
    assert x.abs().max().item() < 0.02 * 3.47


def test_counter_rng_chunking_invariant():
    n = _CHUNK + 1000
    full = normal_f32((n,), 0, 9)
    tail = normal_f32((n,), 0, 9)[_CHUNK:]
    assert torch.equal(full[_CHUNK:], tail)


def test_bf16_rne_matches_torch_conversion():
    x = normal_f32((100000,), 0, 2, std=3.0)
    assert torch.equal(f32_to_bf16_rne(x), x.to(torch.bfloat16))
    y = normal_bf16((100000,), 0, 2, std=3.0)
    assert torch.equal(y, x.to(torch.bfloat16))


def test_vision_inputs_shapes_and_profile():
    w = get_workload("llava15_7b")
    attn, feats = vision_inputs(w.score, 0)
    assert attn.shape == (1, 16, 577) and attn.dtype == torch.float32
    assert len(feats) == 2 and feats[0].shape == (1, 577, 1024) and feats[0].dtype == torch.bfloat16
    assert torch.allclose(attn.double().sum(-1), torch.ones(1, 16, dtype=torch.float64), atol=1e-5)
    # peaked: the salient 5 % of patches hold most of the mass
    top = attn[0].mean(0)[1:].sort(descending=True).values
    assert top[:29].sum() > 0.5
    w2 = get_workload("tiny")
    a2, f2 = vision_inputs(w2.score, 0)
    assert a2.shape == (1, 2, 50) and f2[0].shape == (1, 50, 64)
    a3, _ = vision_inputs(w2.score, 0)
    assert torch.equal(a2, a3)


def test_skip_inputs():
    w = get_workload("llava15_7b")
    m = layer_mask(w)
    assert m.shape == (32, 2) and 0.1 < m.mean() < 0.4
    w3 = get_workload("llava_next_7b")
    s = adaptive_scores(w3, 100)
    assert s.shape == (1, 16, 100) and s.min() >= 0 and s.max() <= 1
    assert np.array_equal(s, adaptive_scores(w3, 100))
