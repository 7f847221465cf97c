"""Pins of the oracle's projector on kept rows (LLaVA's two-layer GELU MLP,
applied after pruning in the ViT feature space)."""
import math

import numpy as np
import pytest

from oracle import msv_prune as mp
from oracle import projector as pj


@pytest.mark.parametrize("t,expect", [
    (0.0, 0.0),
    (1.0, 0.8413447460685429),      # Phi(1)
    (-1.0, -0.15865525393145707),   # -(1 - Phi(1))
    (2.0, 2 * 0.9772498680518208),  # 2 Phi(2)
    (10.0, 10.0),
    (-10.0, 0.0),
])
def test_gelu_is_t_times_the_normal_cdf(t, expect):
    assert abs(pj.gelu(t) - expect) < 1e-15 + 1e-15 * abs(expect)


def test_identity_weights_give_gelu_of_the_input_plus_bias():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 4))
    b2 = rng.standard_normal(4)
    y = pj.project(x, np.eye(4), None, np.eye(4), b2, recipe="f32")
    assert np.allclose(y, pj.gelu(x) + b2, rtol=0, atol=1e-15)


def test_brute_force_on_tiny_shapes():
    rng = np.random.default_rng(1)
    m, d_in, d_h, d_out = 3, 4, 5, 2
    x = rng.standard_normal((m, d_in))
    W1, b1 = rng.standard_normal((d_h, d_in)), rng.standard_normal(d_h)
    W2, b2 = rng.standard_normal((d_out, d_h)), rng.standard_normal(d_out)
    y = pj.project(x, W1, b1, W2, b2, recipe="f32")
    for r in range(m):
        h = []
        for k in range(d_h):
            t = sum(W1[k, c] * x[r, c] for c in range(d_in)) + b1[k]
            h.append(t * 0.5 * (1.0 + math.erf(t / math.sqrt(2.0))))
        for o in range(d_out):
            v = sum(W2[o, k] * h[k] for k in range(d_h)) + b2[o]
            assert abs(y[r, o] - v) < 1e-12


def test_bf16_recipe_rounds_hidden_and_output():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((4, 8))
    W1, W2 = rng.standard_normal((16, 8)) * 0.3, rng.standard_normal((8, 16)) * 0.3
    y = pj.project(x, W1, None, W2, None, recipe="bf16")
    assert np.array_equal(y, pj.round_bf16(y))
    y32 = pj.project(x, W1, None, W2, None, recipe="f32")
    assert np.max(np.abs(y - y32)) < 0.05 * np.max(np.abs(y32))


def test_projecting_kept_rows_equals_keeping_projected_rows():
    rng = np.random.default_rng(3)
    G, n, d_in, d_out, n_text = 3, 20, 8, 6, 4
    feats = rng.standard_normal((G, n + 1, d_in))
    W1, b1 = rng.standard_normal((12, d_in)), rng.standard_normal(12)
    W2, b2 = rng.standard_normal((d_out, 12)), rng.standard_normal(d_out)
    idx = [sorted(rng.choice(n, 7, replace=False)) for _ in range(G)]
    text = rng.standard_normal((G, n_text, d_out))
    x, cu = pj.assemble_projected(feats, idx, text, 1, W1, b1, W2, b2, recipe="f32")
    allp = np.stack([pj.project(feats[g][1:], W1, b1, W2, b2, recipe="f32") for g in range(G)])
    ref, rcu = mp.assemble(allp, idx, text, 1)
    assert np.array_equal(cu, rcu)
    assert np.allclose(x, ref, rtol=0, atol=1e-12)


def test_two_tiles_per_sample_keep_tile_order():
    rng = np.random.default_rng(4)
    feats = rng.standard_normal((4, 9, 3))
    W1, W2 = np.eye(3), np.eye(3)
    idx = [[0, 2], [1], [], [4, 5, 6]]
    text = np.zeros((2, 2, 3))
    x, cu = pj.assemble_projected(feats, idx, text, 2, W1, None, W2, None, recipe="f32")
    assert list(cu) == [0, 5, 10]
    assert np.allclose(x[0], pj.gelu(feats[0][1])) and np.allclose(x[2], pj.gelu(feats[1][2]))
    assert np.allclose(x[5], pj.gelu(feats[3][5])) and np.allclose(x[8:10], 0.0)
