"""GPU anchor scores of encoders without [CLS] (spider_anchor_colmean: the mean
attention each patch receives, Sec. 4.1.1) and scoring from given anchor
scores (spider_score with cls_attn = NULL), against the oracle.

Bars: anchor scores within 1e-5 relative of the float64 oracle (fp32
accumulation of H n terms per patch); bitwise deterministic and independent
of the tensor strides.  Scoring from the GPU's scores: the anchor set is
decided on fp32 scores on the GPU and on float64 scores in the oracle, so the
test first requires every oracle anchor's score, less its GPU score error, to
stay above every other patch's score plus its error (then the sets must be
identical), after which clusters, scores s and m, and the selection follow the
bars of the CLS path.
"""
import numpy as np
import pytest
import torch

from oracle import msv_prune as mp
from synth import get_workload
from synth.vision import attention_maps, vision_inputs
from gpu_common import need_gpu, log

CASES = {
    # name: (G, H, n)
    "clip_l_shape_3_tiles": (3, 16, 576),
    "ragged_100": (2, 3, 100),
    "smallest_4": (1, 1, 4),
    "1024_patches": (1, 16, 1024),
    "n_not_multiple_of_64_or_256": (2, 5, 300),
}


def _ref(A):
    return np.stack([mp.anchor_scores_colmean(A[g].double().numpy()) for g in range(A.shape[0])])


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_colmean_parity(case):
    L = need_gpu()
    G, H, n = CASES[case]
    log(f"[colmean] case={case} G={G} H={H} n={n}")
    A = attention_maps(G, H, n, seed=1)
    a = L.anchor_colmean(A.cuda())
    torch.cuda.synchronize()
    a = a.cpu().numpy().astype(np.float64)
    ref = _ref(A)
    err = float(np.max(np.abs(a - ref) / np.abs(ref).max(axis=1, keepdims=True)))
    log(f"  max rel err {err:.2e}")
    assert err <= 1e-5


@pytest.mark.gpu
def test_colmean_strides_and_determinism():
    L = need_gpu()
    G, H, n = 2, 4, 200
    A = attention_maps(G, H, n, seed=2)
    padded = torch.zeros(G + 1, H, n + 8, n + 4)
    padded[1:, :, 3:3 + n, :n] = A
    view = padded.cuda()[1:, :, 3:3 + n, :n]
    a1 = L.anchor_colmean(A.cuda())
    a2 = L.anchor_colmean(view)
    a3 = L.anchor_colmean(A.cuda())
    torch.cuda.synchronize()
    assert torch.equal(a1, a2) and torch.equal(a1, a3)


@pytest.mark.gpu
@pytest.mark.parametrize("keep", [128, 288])   # 288 = floor(576 * R_v) at R_v = 1/2
def test_scoring_from_column_means(keep):
    L = need_gpu()
    w = get_workload("llava_next_7b", keep=keep)
    sc = w.score
    G, n = sc.G, sc.n
    log(f"[colmean] scoring G={G} n={n} keep={keep}")
    _, feats = vision_inputs(sc, w.seed)
    A = attention_maps(G, 16, n, seed=3)
    n_anchor, _ = mp.budget(keep)
    a_g = L.anchor_colmean(A.cuda())
    out = L.score(None, [f.cuda() for f in feats], n_anchor, sc.K, sc.kmeans_iter, a=a_g)
    torch.cuda.synchronize()
    a_o = _ref(A)
    cl = out["cluster"].cpu().numpy()
    s = out["s"].cpu().numpy()
    m = out["m"].cpu().numpy()
    assert torch.equal(out["a"], a_g)
    a_gpu = a_g.cpu().numpy().astype(np.float64)
    ores = []
    for g in range(G):
        o = mp.prune_tile(None, [f[g].float().numpy() for f in feats], keep, a=a_o[g], K=sc.K,
                          max_iter=sc.kmeans_iter)
        ores.append(o)
        # every oracle anchor stays above every other patch by more than both score errors
        e = np.abs(a_gpu[g] - a_o[g])
        top = np.zeros(n, bool)
        top[o["anchors"]] = True
        assert np.min(a_o[g][top] - e[top]) > np.max(a_o[g][~top] + e[~top]), \
            "scores too close at the anchor boundary for an exact check"
        assert set(np.nonzero(cl[g] < 0)[0]) == set(o["anchors"]), f"tile {g}: anchors differ"
        if len(o["margin"]):
            assert o["margin"].min() > 1e-4, "input too close to a K-means tie for an exact check"
        assert np.array_equal(cl[g], o["cluster"]), f"tile {g}: clusters differ"
        na = o["cluster"] >= 0
        err = np.abs(s[g][na] - o["s"][na]) / np.maximum(1.0, np.abs(o["s"][na]))
        assert err.size == 0 or err.max() <= 1e-5, f"tile {g}: s error {err.max()}"
        merr = np.abs(m[g] - o["mvec"]) / np.maximum(1.0, np.abs(o["mvec"]))
        assert merr.max() <= 1e-5, f"tile {g}: m error {merr.max()}"
    # selection from the GPU scores equals the oracle's selection
    _, n_cmp = mp.budget(keep)
    sel = L.select(out["cluster"], out["s"], n_anchor, n_cmp, sc.K)
    torch.cuda.synchronize()
    idx = sel["idx"].cpu().numpy()
    cnt = sel["count"].cpu().numpy()
    for g, o in enumerate(ores):
        assert list(idx[g][:cnt[g]]) == list(o["idx"]), f"tile {g}: selection differs"
