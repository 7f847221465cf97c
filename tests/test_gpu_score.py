"""GPU scoring (spider_score) against the oracle on the same seeded inputs.

Bars: head-mean scores and the anchor set bit-exact; K-means assignments
identical (the oracle also reports how far every decision is from a tie, and
the inputs are required to keep that margin well above float32 rounding, so
equality is the expected outcome rather than luck); scores s and anchor
max-similarities m within 1e-5 relative of the float64 oracle.
"""
import numpy as np
import pytest
import torch

from synth import get_workload
from synth.vision import vision_inputs
from gpu_common import need_gpu, oracle_tiles, log

CASES = {
    # name: (workload, keep, tie_stress, K, r_num, r_den)
    "tiny": ("tiny", 16, False, 4, 7, 10),
    "tiny_keep_all": ("tiny", 49, False, 4, 7, 10),
    "tiny_no_anchor": ("tiny", 16, False, 4, 0, 10),
    "tiny_K1": ("tiny", 16, False, 1, 7, 10),
    "llava15_k64": ("llava15_7b", 64, False, 4, 7, 10),
    "llava15_k128": ("llava15_7b", 128, False, 4, 7, 10),
    "llava15_k192": ("llava15_7b", 192, False, 4, 7, 10),
    "llava15_ties": ("llava15_7b", 128, True, 4, 7, 10),
    "llava15_K8": ("llava15_7b", 128, False, 8, 7, 10),
    "next_5tiles": ("llava_next_7b", 128, False, 4, 7, 10),
    "all_anchors": ("llava15_7b", 576, False, 4, 10, 10),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_score_parity(case):
    L = need_gpu()
    wl, keep, ties, K, rn, rd = CASES[case]
    w = get_workload(wl, keep=keep)
    log(f"[score] case={case} G={w.score.G} n={w.score.n} keep={keep} K={K}")
    attn, feats = vision_inputs(w.score, w.seed, tie_stress=ties)
    n_anchor = (keep * rn) // rd
    out = L.score(attn.cuda(), [f.cuda() for f in feats], n_anchor, K, w.score.kmeans_iter)
    torch.cuda.synchronize()
    a = out["a"].cpu().numpy()
    cl = out["cluster"].cpu().numpy()
    s = out["s"].cpu().numpy()
    m = out["m"].cpu().numpy()
    ref = oracle_tiles(attn, feats, keep, rn, rd, K, w.score.kmeans_iter)
    for g, o in enumerate(ref):
        assert np.array_equal(a[g], o["a"]), f"tile {g}: anchor scores differ"
        assert set(np.nonzero(cl[g] < 0)[0]) == set(o["anchors"]), f"tile {g}: anchors differ"
        if len(o["margin"]):
            assert o["margin"].min() > 1e-4, "input too close to a K-means tie for an exact check"
        assert np.array_equal(cl[g], o["cluster"]), f"tile {g}: clusters differ"
        na = o["cluster"] >= 0
        assert np.all(np.isinf(s[g][~na]))
        err = np.abs(s[g][na] - o["s"][na]) / np.maximum(1.0, np.abs(o["s"][na]))
        assert err.size == 0 or err.max() <= 1e-5, f"tile {g}: s error {err.max()}"
        merr = np.abs(m[g] - o["mvec"]) / np.maximum(1.0, np.abs(o["mvec"]))
        assert merr.max() <= 1e-5, f"tile {g}: m error {merr.max()}"


@pytest.mark.gpu
def test_score_deterministic():
    L = need_gpu()
    w = get_workload("llava_next_7b", keep=128)
    attn, feats = vision_inputs(w.score, 1)
    fa = [f.cuda() for f in feats]
    r1 = L.score(attn.cuda(), fa, 89)
    r2 = L.score(attn.cuda(), fa, 89)
    torch.cuda.synchronize()
    for k in ("a", "cluster", "s", "m"):
        assert torch.equal(r1[k], r2[k]), k


@pytest.mark.gpu
def test_score_large_tile_batch_matches_per_tile():
    """64 tiles in one call give the same bits as the same tiles scored separately."""
    L = need_gpu()
    w = get_workload("llava15_7b", keep=128)
    from dataclasses import replace
    w64 = replace(w, score=replace(w.score, G=64))
    attn, feats = vision_inputs(w64.score, 3)
    log("[score] G=64 batch")
    allr = L.score(attn.cuda(), [f.cuda() for f in feats], 89)
    for g in (0, 17, 63):
        one = L.score(attn[g:g + 1].contiguous().cuda(), [f[g:g + 1].contiguous().cuda() for f in feats], 89)
        for k in ("a", "cluster", "s", "m"):
            assert torch.equal(allr[k][g:g + 1], one[k]), (g, k)


@pytest.mark.gpu
def test_score_zero_norm_rows():
    """Feature rows that are exactly zero (cosine with a zero row is 0): some only in the
    middle layer, some only in the last, some in both, one of them an anchor's row; the
    anchor set, clusters and selection inputs must still match the oracle."""
    L = need_gpu()
    w = get_workload("llava15_7b", keep=128)
    attn, feats = vision_inputs(w.score, 11)
    fm, fl = feats[0].clone(), feats[-1].clone()
    a_host = attn[0, :, 1:].sum(0)
    top = int(torch.argmax(a_host))            # the strongest anchor (patch index)
    for i in (3, 40, 41, 200, 575):            # zero in the last layer only
        fl[0, 1 + i] = 0
    for i in (7, 41, 300):                     # zero in the middle layer (41: in both)
        fm[0, 1 + i] = 0
    fl[0, 1 + top] = 0                         # an anchor with a zero last-layer row
    feats = [fm, fl]
    n_anchor = (128 * 7) // 10
    log(f"[score] zero-norm rows, anchor {top} zeroed")
    out = L.score(attn.cuda(), [f.cuda() for f in feats], n_anchor, 4, w.score.kmeans_iter)
    torch.cuda.synchronize()
    cl = out["cluster"].cpu().numpy()[0]
    s = out["s"].cpu().numpy()[0]
    m = out["m"].cpu().numpy()[0]
    o = oracle_tiles(attn, feats, 128, 7, 10, 4, w.score.kmeans_iter)[0]
    assert np.array_equal(out["a"].cpu().numpy()[0], o["a"])
    assert top in set(o["anchors"]) and cl[top] < 0
    assert o["margin"].min() > 1e-4, "input too close to a K-means tie for an exact check"
    assert np.array_equal(cl, o["cluster"])
    na = o["cluster"] >= 0
    err = np.abs(s[na] - o["s"][na]) / np.maximum(1.0, np.abs(o["s"][na]))
    assert err.max() <= 1e-5, err.max()
    merr = np.abs(m - o["mvec"]) / np.maximum(1.0, np.abs(o["mvec"]))
    assert merr.max() <= 1e-5, merr.max()
    # a row that is zero in the last layer has no similarity to any anchor
    for i in (3, 40, 41, 200, 575):
        assert m[i] == 0.0 and o["mvec"][i] == 0.0


@pytest.mark.gpu
@pytest.mark.parametrize("variant", ["last_layer_only", "three_tapped_layers"])
def test_score_tapped_layer_variants(variant):
    """Eq. 3 over other sets of tapped layers (the layer ablations of Tab. 7): the last
    layer alone, and three layers (the middle one, a second middle-layer stand-in, the
    last).  Clustering always runs on the last entry; the oracle sums the same layers."""
    L = need_gpu()
    w = get_workload("llava15_7b", keep=128)
    attn, feats = vision_inputs(w.score, 21)
    fm, fl = feats[0], feats[-1]
    layers = [fl] if variant == "last_layer_only" else [fm, fm.roll(1, dims=-1).contiguous(), fl]
    n_anchor = (128 * 7) // 10
    log(f"[score] {variant}: {len(layers)} tapped layer(s)")
    out = L.score(attn.cuda(), [f.cuda() for f in layers], n_anchor, 4, w.score.kmeans_iter)
    torch.cuda.synchronize()
    o = oracle_tiles(attn, layers, 128, 7, 10, 4, w.score.kmeans_iter)[0]
    cl = out["cluster"].cpu().numpy()[0]
    s = out["s"].cpu().numpy()[0]
    m = out["m"].cpu().numpy()[0]
    assert np.array_equal(out["a"].cpu().numpy()[0], o["a"])
    assert set(np.nonzero(cl < 0)[0]) == set(o["anchors"])
    assert o["margin"].min() > 1e-4, "input too close to a K-means tie for an exact check"
    assert np.array_equal(cl, o["cluster"])
    na = o["cluster"] >= 0
    err = np.abs(s[na] - o["s"][na]) / np.maximum(1.0, np.abs(o["s"][na]))
    assert err.max() <= 1e-5, f"s error {err.max()}"
    assert np.max(np.abs(m - o["mvec"]) / np.maximum(1.0, np.abs(o["mvec"]))) <= 1e-5


WIDE = {
    # name: (patches n, width d_v, heads, tapped layers, keep, K, fp32 features): the
    # feature-width paths of the scoring kernels not taken by the CLIP-L and tiny
    # workloads -- bf16 at d_v <= 512 (ViT-S-like 384), fp32 past 512 (the CLIP-L
    # tile with its bf16 features widened exactly), past 1024 (SigLIP-like 27 x 27 x
    # 1152, a Qwen-ViT-like 1280 with three taps) -- and the largest tile the entry
    # point takes (4096 patches, d_v 2048: the anchor top-k sorts 4096 keys)
    "vit_s_576x384_bf16": (576, 384, 6, (6, 12), 144, 4, False),
    "clip_l_576x1024_fp32": (576, 1024, 16, (12, 24), 128, 4, True),
    "siglip_729x1152": (729, 1152, 16, (13, 26), 182, 4, False),
    "qwen_1024x1280_three_taps": (1024, 1280, 16, (8, 16, 32), 256, 4, False),
    "max_4096x2048": (4096, 2048, 16, (12, 24), 1024, 4, False),
    # the score pass per cluster-mean layout: the block kernel while layers x K x d_v
    # fits its LDS (8192 floats), the per-wave kernel past that, for each width class
    # and dtype
    "qwen_1024x1280_fp32": (1024, 1280, 16, (8, 16), 256, 4, True),
    "qwen_1024x1280_fp32_K3": (1024, 1280, 16, (8, 16), 256, 3, True),
    "siglip_729x1152_K3": (729, 1152, 16, (13, 26), 182, 3, False),
    "vit_s_576x384_K8_three_taps": (576, 384, 6, (4, 8, 12), 144, 8, False),
    "vit_s_576x384_fp32_K8_three_taps": (576, 384, 6, (4, 8, 12), 144, 8, True),
    "clip_l_576x1024_fp32_K8": (576, 1024, 16, (12, 24), 128, 8, True),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(WIDE))
def test_score_feature_width_paths(case):
    """Same bars as test_score_parity on one tile of each shape (seeded CLIP-style taps)."""
    import dataclasses
    L = need_gpu()
    n, dv, H, layers, keep, K, f32 = WIDE[case]
    cfg = dataclasses.replace(get_workload("llava15_7b", keep=keep).score, G=1, n=n, d_v=dv, H=H,
                              layers=layers, keep=keep, K=K)
    log(f"[score width] case={case} n={n} d_v={dv} taps={layers} keep={keep} K={K} fp32={f32}")
    attn, feats = vision_inputs(cfg, 7)
    if f32:
        feats = [f.float() for f in feats]
    n_anchor = (keep * 7) // 10
    out = L.score(attn.cuda(), [f.cuda() for f in feats], n_anchor, K, cfg.kmeans_iter)
    torch.cuda.synchronize()
    a, cl = out["a"].cpu().numpy()[0], out["cluster"].cpu().numpy()[0]
    s, m = out["s"].cpu().numpy()[0], out["m"].cpu().numpy()[0]
    o = oracle_tiles(attn, feats, keep, 7, 10, K, cfg.kmeans_iter)[0]
    assert np.array_equal(a, o["a"])
    assert set(np.nonzero(cl < 0)[0]) == set(o["anchors"])
    assert o["margin"].min() > 1e-4, "input too close to a K-means tie for an exact check"
    assert np.array_equal(cl, o["cluster"])
    na = o["cluster"] >= 0
    assert np.all(np.isinf(s[~na]))
    err = np.abs(s[na] - o["s"][na]) / np.maximum(1.0, np.abs(o["s"][na]))
    assert err.max() <= 1e-5, f"s error {err.max()}"
    merr = np.abs(m - o["mvec"]) / np.maximum(1.0, np.abs(o["mvec"]))
    assert merr.max() <= 1e-5, f"m error {merr.max()}"


NT_BATCH = {
    # name: (patches n, width d_v, fp32 features, tiles G): one call over more than
    # 256 MB of features, which the scoring pass reads with non-temporal loads
    "bf16_384": (576, 384, False, 312),
    "bf16_1024": (576, 1024, False, 120),
    "bf16_1152": (729, 1152, False, 88),
    "fp32_384": (576, 384, True, 160),
    "fp32_1024": (576, 1024, True, 64),
    "fp32_1280": (1024, 1280, True, 32),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(NT_BATCH))
def test_score_nontemporal_batch_matches_small_batch(case):
    """A batch past 256 MB of features (non-temporal loads in the scoring pass) gives
    the bits of the same tiles scored 8 at a time (cached loads): the batch repeats
    8 seeded tiles, so every tile is compared."""
    import dataclasses
    L = need_gpu()
    n, dv, f32, G = NT_BATCH[case]
    cfg = dataclasses.replace(get_workload("llava15_7b", keep=128).score, G=8, n=n, d_v=dv,
                              layers=(12, 24), keep=n // 4, K=4)
    attn, feats = vision_inputs(cfg, 11)
    if f32:
        feats = [f.float() for f in feats]
    esize = 4 if f32 else 2
    assert G * n * dv * esize * len(feats) > (256 << 20) and G % 8 == 0
    log(f"[score nt] case={case} G={G} n={n} d_v={dv} fp32={f32}")
    n_anchor = (cfg.keep * 7) // 10
    attn_d, feats_d = attn.cuda(), [f.cuda() for f in feats]
    small = L.score(attn_d, feats_d, n_anchor)
    big = L.score(attn_d.repeat(G // 8, 1, 1), [f.repeat(G // 8, 1, 1) for f in feats_d], n_anchor)
    torch.cuda.synchronize()
    for k in ("a", "cluster", "s", "m"):
        ref = small[k].repeat(G // 8, 1)
        assert torch.equal(big[k], ref), k
