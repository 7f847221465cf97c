"""Pins of the oracle's [CLS] attention rebuilt from the query and the keys
(the row Sec. 4.1.1 averages, for ViTs that never store attention maps)."""
import numpy as np
import pytest

from oracle import msv_prune as mp


def test_identical_keys_give_uniform_rows():
    rng = np.random.default_rng(0)
    H, dh, T = 3, 8, 11
    k = np.broadcast_to(rng.standard_normal((1, H, dh)), (T, H, dh))
    A = mp.cls_attention(rng.standard_normal((H, dh)), k, 0.125)
    assert np.allclose(A, 1.0 / T, rtol=0, atol=1e-15)


def test_one_aligned_key_with_a_large_scale_takes_all_the_weight():
    H, dh, T = 2, 4, 6
    q = np.zeros((H, dh))
    q[:, 0] = 1.0
    k = np.zeros((T, H, dh))
    k[3, 0, 0] = 1.0      # head 0: token 3 aligned with q
    k[5, 1, 0] = 1.0      # head 1: token 5
    A = mp.cls_attention(q, k, 1e3)
    assert A[0, 3] == 1.0 and A[1, 5] == 1.0
    assert A[0].sum() == 1.0 and np.count_nonzero(A[0] > 1e-300) == 1


def test_two_tokens_closed_form():
    # logits s*q.k0 and s*q.k1: weight of token 1 = sigmoid(s*q.(k1 - k0))
    q = np.array([[1.0, 2.0]])
    k = np.array([[[0.5, 0.0]], [[1.0, 1.0]]])
    s = 0.5
    A = mp.cls_attention(q, k, s)
    expect = 1.0 / (1.0 + np.exp(-s * (3.0 - 0.5)))
    assert abs(A[0, 1] - expect) < 1e-15 and abs(A[0, 0] - (1 - expect)) < 1e-15


def test_rows_sum_to_one_and_shift_invariance():
    rng = np.random.default_rng(1)
    H, dh, T = 4, 16, 50
    q = rng.standard_normal((H, dh))
    k = rng.standard_normal((T, H, dh))
    A = mp.cls_attention(q, k, 0.25)
    assert np.allclose(A.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    # adding one vector per head to every key shifts that head's logits by a constant
    shift = rng.standard_normal((1, H, dh))
    assert np.allclose(mp.cls_attention(q, k + shift, 0.25), A, rtol=0, atol=1e-14)


def test_brute_force_and_head_mean():
    rng = np.random.default_rng(2)
    H, dh, T = 2, 3, 5
    q = rng.standard_normal((H, dh))
    k = rng.standard_normal((T, H, dh))
    A = mp.cls_attention(q, k, 0.7)
    for h in range(H):
        z = [0.7 * sum(q[h, c] * k[j, h, c] for c in range(dh)) for j in range(T)]
        e = [np.exp(v - max(z)) for v in z]
        for j in range(T):
            assert abs(A[h, j] - e[j] / sum(e)) < 1e-15
    a = mp.anchor_scores(A.astype(np.float32), col0=1)
    assert a.shape == (T - 1,)
