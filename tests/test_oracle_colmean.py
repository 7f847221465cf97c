"""Pins of the oracle's anchor scores for encoders without [CLS] (Sec. 4.1.1:
the mean attention each patch receives) and of the ratio budget (the
Qwen3-VL setting: a retention ratio R_v of an input-dependent token count).
"""
import itertools

import numpy as np
import pytest

from oracle import msv_prune as mp


def _softmax_maps(rng, H, n, scale=2.0):
    z = rng.standard_normal((H, n, n)) * scale
    z -= z.max(axis=2, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=2, keepdims=True)


def test_uniform_attention_gives_uniform_scores():
    H, n = 3, 7
    a = mp.anchor_scores_colmean(np.full((H, n, n), 1.0 / n))
    assert np.allclose(a, 1.0 / n, rtol=0, atol=1e-15)


def test_identity_attention_gives_uniform_scores():
    H, n = 2, 5
    a = mp.anchor_scores_colmean(np.stack([np.eye(n)] * H))
    assert np.allclose(a, 1.0 / n, rtol=0, atol=1e-15)


@pytest.mark.parametrize("c", [0, 3, 8])
def test_all_queries_on_one_patch_gives_indicator(c):
    H, n = 4, 9
    A = np.zeros((H, n, n))
    A[:, :, c] = 1.0
    a = mp.anchor_scores_colmean(A)
    expect = np.zeros(n)
    expect[c] = 1.0
    assert np.array_equal(a, expect)


def test_heads_with_different_targets_average():
    # head 0 sends every query to patch 1, head 1 to patch 4: each gets 1/2
    n = 6
    A = np.zeros((2, n, n))
    A[0, :, 1] = 1.0
    A[1, :, 4] = 1.0
    a = mp.anchor_scores_colmean(A)
    assert a[1] == 0.5 and a[4] == 0.5 and a.sum() == 1.0


def test_row_stochastic_maps_give_scores_summing_to_one():
    rng = np.random.default_rng(0)
    a = mp.anchor_scores_colmean(_softmax_maps(rng, 16, 64))
    assert abs(a.sum() - 1.0) < 1e-12


def test_brute_force_on_a_tiny_tile():
    rng = np.random.default_rng(1)
    H, n = 3, 5
    A = rng.random((H, n, n))
    a = mp.anchor_scores_colmean(A)
    for j in range(n):
        tot = 0.0
        for h, i in itertools.product(range(H), range(n)):
            tot += A[h, i, j]
        assert abs(a[j] - tot / (H * n)) < 1e-15


def test_invariant_to_head_and_query_order_and_equivariant_to_key_order():
    rng = np.random.default_rng(2)
    A = _softmax_maps(rng, 4, 12)
    a = mp.anchor_scores_colmean(A)
    ph, pq, pk = rng.permutation(4), rng.permutation(12), rng.permutation(12)
    assert np.allclose(mp.anchor_scores_colmean(A[ph]), a, rtol=0, atol=1e-15)
    assert np.allclose(mp.anchor_scores_colmean(A[:, pq]), a, rtol=0, atol=1e-15)
    assert np.allclose(mp.anchor_scores_colmean(A[:, :, pk]), a[pk], rtol=0, atol=1e-15)


def test_prune_tile_takes_given_anchor_scores():
    rng = np.random.default_rng(3)
    n, d = 40, 16
    feats = [np.vstack([np.zeros((1, d)), rng.standard_normal((n, d))]) for _ in range(2)]
    a = rng.random(n)
    out = mp.prune_tile(None, feats, keep=12, a=a)
    assert out["anchors"] == mp.anchor_set(a, 8)       # floor(12 * 0.7) = 8
    assert np.array_equal(out["a"], a)


@pytest.mark.parametrize("n,num,den,expect", [
    (576, 1, 2, (288, 201, 87)),     # R_v = 0.5 of a CLIP-L tile
    (1000, 2, 5, (400, 280, 120)),   # R_v = 0.4
    (7, 1, 2, (3, 2, 1)),            # floor, not round
    (1369, 1, 2, (684, 478, 206)),
    (50, 1, 1, (50, 35, 15)),        # keep everything
    (50, 0, 3, (0, 0, 0)),
])
def test_ratio_budget_by_hand(n, num, den, expect):
    assert mp.budget_ratio(n, num, den) == expect


def test_ratio_budget_rejects_bad_arguments():
    for args in [(-1, 1, 2), (10, 3, 2), (10, 1, 0), (10, -1, 2)]:
        with pytest.raises(ValueError):
            mp.budget_ratio(*args)
