"""GPU [CLS] attention rebuilt from the CLS query and keys (spider_cls_attention)
against the oracle, and scoring from it (Sec. 4.1.1 for encoders that never
store attention maps).

Bars: every attention row within 1e-5 of the float64 oracle relative to the
row's largest weight; deterministic.  Scoring: the anchor scores (head means)
follow from fp32 rows on the GPU and float64 rows in the oracle, so the test
first requires every oracle anchor's score, less its GPU error, to stay above
every other patch's score plus its error; then anchors, clusters, s and m
follow the bars of the stored-attention path.
"""
import numpy as np
import pytest
import torch

from oracle import msv_prune as mp
from synth import get_workload
from synth.vision import cls_query_keys, vision_inputs
from gpu_common import need_gpu, log

CASES = {
    # name: (G, H, dh, T, dtype)
    "clip_l_bf16_3_tiles": (3, 16, 64, 577, "bf16"),
    "clip_l_f32": (1, 16, 64, 577, "f32"),
    "ragged_tokens_dh128": (2, 4, 128, 301, "bf16"),
    "one_token": (1, 2, 8, 1, "f32"),
    "dh256_4097_tokens": (1, 1, 256, 4097, "bf16"),
}


def _oracle(q, k, scale):
    return np.stack([mp.cls_attention(q[g].double().numpy(), k[g].double().numpy(), scale)
                     for g in range(q.shape[0])])


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_cls_attention_parity(case):
    L = need_gpu()
    G, H, dh, T, dt = CASES[case]
    log(f"[cls_attention] case={case} G={G} H={H} dh={dh} T={T} {dt}")
    q, k = cls_query_keys(G, H, dh, T, seed=1, dtype=dt)
    scale = float(dh) ** -0.5
    A = L.cls_attention(q.cuda(), k.cuda(), scale)
    A2 = L.cls_attention(q.cuda(), k.cuda(), scale)
    torch.cuda.synchronize()
    assert torch.equal(A, A2)
    ref = _oracle(q, k, scale)
    err = float(np.max(np.abs(A.cpu().numpy() - ref) / ref.max(axis=2, keepdims=True)))
    log(f"  max rel err {err:.2e}")
    assert err <= 1e-5


@pytest.mark.gpu
def test_scoring_from_rebuilt_cls_attention():
    L = need_gpu()
    w = get_workload("llava_next_7b", keep=128)
    sc = w.score
    G, n = sc.G, sc.n
    _, feats = vision_inputs(sc, w.seed)
    q, k = cls_query_keys(G, 16, 64, n + 1, seed=2)
    scale = 0.125
    A = L.cls_attention(q.cuda(), k.cuda(), scale)
    n_anchor, _ = mp.budget(128)
    out = L.score(A, [f.cuda() for f in feats], n_anchor, sc.K, sc.kmeans_iter)
    torch.cuda.synchronize()
    a_g = out["a"].cpu().numpy().astype(np.float64)
    cl = out["cluster"].cpu().numpy()
    s = out["s"].cpu().numpy()
    ref = _oracle(q, k, scale).astype(np.float32)
    for g in range(G):
        o = mp.prune_tile(ref[g], [f[g].float().numpy() for f in feats], 128, K=sc.K, max_iter=sc.kmeans_iter)
        a_o = o["a"].astype(np.float64)
        e = np.abs(a_g[g] - a_o)
        top = np.zeros(n, bool)
        top[o["anchors"]] = True
        assert np.min(a_o[top] - e[top]) > np.max(a_o[~top] + e[~top]), \
            "scores too close at the anchor boundary for an exact check"
        assert set(np.nonzero(cl[g] < 0)[0]) == set(o["anchors"]), f"tile {g}: anchors differ"
        if len(o["margin"]):
            assert o["margin"].min() > 1e-4, "input too close to a K-means tie for an exact check"
        assert np.array_equal(cl[g], o["cluster"]), f"tile {g}: clusters differ"
        na = o["cluster"] >= 0
        err = np.abs(s[g][na] - o["s"][na]) / np.maximum(1.0, np.abs(o["s"][na]))
        assert err.size == 0 or err.max() <= 1e-5, f"tile {g}: s error {err.max()}"
