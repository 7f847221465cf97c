"""Pins of the MSV-Prune oracle (Sec. 4.1) against closed forms, brute force and libraries."""
import json
import math
import os

import numpy as np
import pytest

from oracle import msv_prune as mp
from synth import get_workload
from synth.vision import vision_inputs, rng

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- anchor scores
def test_anchor_scores_single_head_is_identity():
    row = rng(1, 1).random((1, 30)).astype(np.float32)
    a = mp.anchor_scores(row, col0=1)
    assert a.dtype == np.float32
    assert np.array_equal(a, row[0, 1:])


def test_anchor_scores_exact_mean_of_dyadic_values():
    # values are multiples of 1/8: the float32 sum and the division by 4 are exact
    A = np.array([[0, 1, 2, 3], [0, 3, 2, 1], [0, 0, 0, 8], [0, 4, 4, 4]], np.float32) / 8
    assert np.array_equal(mp.anchor_scores(A, col0=1), np.array([8, 8, 16], np.float32) / 32)


def test_anchor_scores_sequential_float32_order():
    # (1 + 2^-24) + 2^-24 rounds twice in sequential float32; a float64 sum would not
    A = np.array([[0, 1.0], [0, 2.0 ** -24], [0, 2.0 ** -24]], np.float32)
    a = mp.anchor_scores(A, col0=1)
    expect = np.float32(np.float32(np.float32(1.0) + np.float32(2 ** -24)) + np.float32(2 ** -24)) / np.float32(3)
    assert a[0] == expect


# ---------------------------------------------------------------- budget
@pytest.mark.parametrize("keep,exp", [(16, (11, 5)), (64, (44, 20)), (128, (89, 39)),
                                      (192, (134, 58)), (576, (403, 173)), (1440, (1008, 432)),
                                      (0, (0, 0))])
def test_budget_integer_rule(keep, exp):
    assert mp.budget(keep, 7, 10) == exp


def test_budget_float_pitfall():
    # floor(1440 * 0.7) in binary floating point is 1007; the rational rule gives 1008
    assert math.floor(1440 * 0.7) == 1007
    assert mp.budget(1440)[0] == 1008


# ---------------------------------------------------------------- anchor top-k
def test_anchor_set_matches_threshold_set_on_distinct_values():
    for seed in range(20):
        a = rng(seed, 2).permutation(200).astype(np.float32) / 7.0
        for k in (0, 1, 17, 140, 200):
            assert mp.anchor_set(a, k) == mp.threshold_set(a, k)


def test_anchor_set_ties_go_to_lower_index():
    a = np.array([0.5, 0.9, 0.5, 0.9, 0.1, 0.5], np.float32)
    assert mp.anchor_set(a, 3) == [0, 1, 3]
    assert mp.anchor_set(a, 4) == [0, 1, 2, 3]
    assert mp.anchor_set(np.array([0.0, -0.0, 0.0], np.float32), 2) == [0, 1]


def test_anchor_set_brute_force_rank_on_quantised_values():
    for seed in range(10):
        a = (np.round(rng(seed, 3).random(300) * 16) / 16).astype(np.float32)
        k = 101
        got = set(mp.anchor_set(a, k))
        # independent definition: i is an anchor iff fewer than k tokens beat it
        for i in range(len(a)):
            better = np.sum((a > a[i]) | ((a == a[i]) & (np.arange(len(a)) < i)))
            assert (better < k) == (i in got)


def test_anchor_nan_rejected():
    with pytest.raises(ValueError):
        mp.anchor_set(np.array([0.1, np.nan], np.float32), 1)


# ---------------------------------------------------------------- k-means
def _blobs(seed, m=300, d=32, K=4, spread=0.05):
    r = rng(seed, 4)
    centres = r.standard_normal((K, d)) * 3
    lab = r.integers(0, K, size=m)
    return (centres[lab] + spread * r.standard_normal((m, d))).astype(np.float32), lab


def test_kmeans_matches_sklearn_lloyd_with_same_init():
    # scikit-learn relocates clusters that become empty while this reading
    # keeps their centroid, so only runs without an empty cluster are compared
    from sklearn.cluster import KMeans
    compared = 0
    for seed in range(12):
        X, _ = _blobs(seed, K=6)   # 6 blobs into 4 clusters: centroids move
        K = 4
        init = X[[(k * len(X)) // K for k in range(K)]].astype(np.float64)
        ours, _, passes, margin = mp.kmeans(X, K, 50)
        if np.bincount(ours, minlength=K).min() == 0:
            continue
        sk = KMeans(n_clusters=K, init=init, n_init=1, max_iter=50, tol=0.0,
                    algorithm="lloyd").fit(X.astype(np.float64))
        assert np.array_equal(ours, sk.labels_)
        assert margin.min() > 1e-3
        compared += 1
    assert compared >= 8


def test_kmeans_fixed_point_properties():
    X, _ = _blobs(7, m=200, d=16, K=5, spread=0.5)
    assign, c, passes, _ = mp.kmeans(X, 4, 100)
    assert passes < 100  # converged
    Xd = X.astype(np.float64)
    for k in range(4):
        members = Xd[assign == k]
        if len(members):
            assert np.allclose(c[k], members.mean(axis=0), atol=1e-5)
    d2 = ((Xd[:, None, :] - c[None].astype(np.float64)) ** 2).sum(-1)
    assert np.array_equal(assign, d2.argmin(axis=1))


def test_kmeans_recovers_separated_blobs():
    X, lab = _blobs(3, m=400, d=64, K=4, spread=0.01)
    assign, _, _, _ = mp.kmeans(X, 4, 10)
    # same partition up to relabelling
    for k in range(4):
        assert len(set(lab[assign == k])) <= 1
    assert len(set(zip(assign, lab))) == len(set(lab))


def test_kmeans_init_rows_and_tie_to_lower_cluster():
    X = np.array([[0.0], [1.0], [1.0], [3.0]], np.float32)
    # K=4 over m=4 rows: init rows 0,1,2,3; rows 1 and 2 are identical, so row 2
    # ties between clusters 1 and 2 and goes to 1; cluster 2 is then empty and keeps (1.0)
    assign, c, _, _ = mp.kmeans(X, 4, 10)
    assert list(assign) == [0, 1, 1, 3]
    assert c[2, 0] == 1.0


def test_kmeans_single_pass_cap():
    X, _ = _blobs(9, K=6)
    a1, _, p1, _ = mp.kmeans(X, 4, 1)
    assert p1 == 1
    init = X[[(k * len(X)) // 4 for k in range(4)]]
    d2 = ((X[:, None, :].astype(np.float64) - init[None]) ** 2).sum(-1)
    assert np.array_equal(a1, d2.argmin(1))


# ---------------------------------------------------------------- quotas (Eq. 2)
def test_quotas_hand_cases():
    # 5*19/38 = 2.5 -> 2 (half to even), 1.32 -> 1, 0.79 -> 1, 0.39 -> max(1, 0) = 1
    assert mp.quotas([19, 10, 6, 3], 5) == [2, 1, 1, 1]
    # overshoot: 0.5 -> 0 -> max(1, .) = 1 in every cluster, total 4 > 2
    assert mp.quotas([10, 10, 10, 10], 2) == [1, 1, 1, 1]
    # empty clusters get nothing; 1.5 -> 2 (half to even)
    assert mp.quotas([5, 0, 5, 0], 3) == [2, 0, 2, 0]
    # budget above the token count: 4.5 -> 4 and 1.5 -> 2, each clipped to its cluster size
    assert mp.quotas([3, 1], 6) == [3, 1]
    assert mp.quotas([3, 1], 3) == [2, 1]      # 2.25 -> 2, 0.75 -> 1
    # keep-all: every token of every cluster
    assert mp.quotas([7, 11, 2, 30], 50) == [7, 11, 2, 30]
    assert mp.quotas([4, 4], 0) == [0, 0]


def test_quotas_exact_mode_sums_to_budget():
    assert mp.quotas([19, 10, 6, 3], 5, "exact") == [3, 1, 1, 0]
    for seed in range(50):
        sizes = list(rng(seed, 5).integers(0, 60, size=4))
        D = sum(sizes)
        for n_cmp in (0, 1, 7, D // 2, D):
            q = mp.quotas(sizes, n_cmp, "exact")
            assert sum(q) == (min(n_cmp, D) if D else 0)
            assert all(0 <= a <= s for a, s in zip(q, sizes))


# ---------------------------------------------------------------- Eq. 3 scores
def test_eq3_hand_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "eq3_worked_example.json")))
    attn = np.array(g["cls_attn"], np.float32)
    feats = [np.array(g["feat_mid"], np.float64), np.array(g["feat_last"], np.float64)]
    out = mp.prune_tile(attn, feats, g["keep"], g["r_num"], g["r_den"], K=g["K"], max_iter=10)
    for i, expr in g["expected_s"].items():
        assert out["s"][int(i)] == pytest.approx(eval(expr, {"sqrt": math.sqrt}), abs=1e-12)
    assert out["idx"] == g["expected_idx"]
    assert out["anchors"] == [0]
    assert np.isinf(out["s"][0])


def test_eq3_orthonormal_rows_closed_form():
    n, d, L = 12, 40, 3
    eye = np.eye(d)
    feats = [np.vstack([np.zeros(d), eye[perm[:n]]]) for perm in
             (rng(s, 6).permutation(d) for s in range(L))]
    cluster = np.array([-1, -1, 0, 0, 0, 1, 1, 1, 1, 2, 3, 3])
    s, mvec = mp.complementary_scores([f[1:] for f in feats], [0, 1], cluster)
    assert np.allclose(mvec, [1, 1] + [0] * 10)
    for k in range(4):
        C = cluster == k
        assert np.allclose(s[C], L / C.sum())


def test_eq3_collinear_cluster_closed_form():
    d = 8
    base = rng(0, 7).standard_normal(d)
    other = np.zeros(d)
    other[0] = 1.0
    base[0] = 0.0                      # base orthogonal to the anchor direction
    scales = np.array([1.0, 2.5, 0.1, 7.0])
    F = np.vstack([other, scales[:, None] * base])      # token 0 = anchor
    cluster = np.array([-1, 0, 0, 0, 0])
    s, mvec = mp.complementary_scores([F, F], [0], cluster)
    assert np.allclose(s[1:], 2.0)      # two layers, every cosine 1, anchor term 0
    F2 = np.vstack([base, scales[:, None] * base])      # anchor collinear too
    s2, _ = mp.complementary_scores([F2, F2], [0], cluster)
    assert np.allclose(s2[1:], 4.0)     # 2 + m_i + m_j = 2 + 1 + 1


def test_eq3_zero_rows_and_no_anchors():
    F = np.array([[0.0, 0.0], [1.0, 0.0], [0.0, 1.0]])
    s, mvec = mp.complementary_scores([F], [], np.array([0, 0, 0]))
    assert np.allclose(mvec, 0)
    # zero row: all its cosines 0; rows 1,2: self 1, each other 0
    assert np.allclose(s, [0.0, 1 / 3, 1 / 3])


def test_eq3_scale_and_permutation_invariance():
    r = rng(2, 8)
    n, d = 40, 16
    F = [r.standard_normal((n, d)) for _ in range(2)]
    cluster = r.integers(0, 3, size=n)
    cluster[:5] = -1
    anchors = list(range(5))
    s, _ = mp.complementary_scores(F, anchors, cluster)
    scale = r.uniform(0.1, 10, size=(n, 1))
    s2, _ = mp.complementary_scores([f * scale for f in F], anchors, cluster)
    assert np.allclose(s, s2)
    perm = r.permutation(n)
    inv = np.argsort(perm)
    s3, _ = mp.complementary_scores([f[perm] for f in F], list(inv[anchors]), cluster[perm])
    assert np.allclose(s3, s[perm])


def test_eq3_factored_identity():
    # mean_j S_ij == sum_l u_i . mean_j u_j + m_i + mean_j m_j (the form the GPU path uses)
    r = rng(5, 9)
    n, d = 60, 24
    F = [r.standard_normal((n, d)) for _ in range(3)]
    cluster = r.integers(0, 4, size=n)
    cluster[:9] = -1
    s, mvec = mp.complementary_scores(F, list(range(9)), cluster)
    U = [f / np.linalg.norm(f, axis=1, keepdims=True) for f in F]
    for k in range(4):
        C = cluster == k
        fac = sum(u[C] @ u[C].mean(axis=0) for u in U) + mvec[C] + mvec[C].mean()
        assert np.allclose(s[C], fac, atol=1e-12)


# ---------------------------------------------------------------- selection
def test_select_brute_force_rank_with_ties():
    for seed in range(20):
        r = rng(seed, 10)
        n, K = 200, 4
        cluster = r.integers(0, K, size=n)
        cluster[r.choice(n, 30, replace=False)] = -1
        s = (np.round(r.random(n) * 8) / 8).astype(np.float32)
        s[cluster < 0] = np.inf
        n_cmp = int(r.integers(0, 60))
        idx, N = mp.select(cluster, s, n_cmp, K)
        got = set(idx)
        assert idx == sorted(got)
        for i in range(n):
            if cluster[i] < 0:
                assert i in got
                continue
            C = np.nonzero(cluster == cluster[i])[0]
            better = sum(1 for j in C if (s[j], j) < (s[i], i))
            assert (better < N[cluster[i]]) == (i in got)


def test_prune_tile_keep_all_is_identity():
    w = get_workload("tiny", keep=49)
    attn, feats = vision_inputs(w.score, 0)
    out = mp.prune_tile(attn[0].numpy(), [f[0].numpy() for f in feats], 49)
    assert out["idx"] == list(range(49))


def test_prune_tile_tiny_invariants():
    w = get_workload("tiny")
    attn, feats = vision_inputs(w.score, 0)
    out = mp.prune_tile(attn[0].numpy(), [f[0].numpy() for f in feats], 16)
    assert out["k_anc"] == 11 and out["n_cmp"] == 5
    assert set(out["anchors"]) <= set(out["idx"])
    assert len(out["idx"]) == 11 + sum(out["quotas"])
    assert out["idx"] == sorted(out["idx"])
    assert (out["cluster"] == -1).sum() == 11
    assert out["margin"].min() > 1e-4


def test_assemble_layout():
    src = np.arange(2 * 5 * 3).reshape(2, 5, 3).astype(np.float64)
    text = -np.ones((1, 2, 3))
    x, cu = mp.assemble(src, [[0, 4], [1, 2, 3]], text, tiles_per_sample=2)
    assert list(cu) == [0, 7]
    assert np.array_equal(x[:2], src[0, [0, 4]])
    assert np.array_equal(x[2:5], src[1, [1, 2, 3]])
    assert np.array_equal(x[5:], text[0])
