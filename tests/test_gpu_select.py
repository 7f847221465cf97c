"""GPU selection/assembly (spider_select) against the oracle, given identical fp32 scores.

Indices and counts must be bit-exact; assembled rows are byte copies.
"""
import numpy as np
import pytest
import torch

from oracle import msv_prune as mp
from synth import get_workload
from synth.decoder_inputs import text_rows, visual_src
from synth.vision import rng
from gpu_common import need_gpu, log


def _inputs(G, n, K, n_anchor, seed, quantise):
    r = rng(seed, 900)
    cl = r.integers(0, K, size=(G, n)).astype(np.int32)
    s = r.standard_normal((G, n)).astype(np.float32)
    if quantise:
        s = (np.round(s * 8) / 8).astype(np.float32)
    for g in range(G):
        anc = r.choice(n, size=n_anchor, replace=False)
        cl[g, anc] = -1
        s[g, anc] = np.inf
    if K > 2:
        cl[0][cl[0] == 2] = 1      # an empty cluster in tile 0
    return cl, s


SEL_CASES = [
    # G, n, K, keep, quantise, mode
    (1, 49, 4, 16, False, 0),
    (1, 576, 4, 64, True, 0),
    (1, 576, 4, 128, True, 0),
    (1, 576, 4, 192, False, 0),
    (5, 576, 4, 128, True, 1),
    (3, 576, 1, 128, True, 0),
    (2, 576, 8, 144, True, 0),
    (2, 576, 4, 576, False, 0),
    (2, 576, 4, 10, True, 1),
    (1, 4096, 4, 700, True, 0),
    (1, 7, 4, 3, False, 0),
]


@pytest.mark.gpu
@pytest.mark.parametrize("G,n,K,keep,quant,mode", SEL_CASES)
def test_select_parity(G, n, K, keep, quant, mode):
    L = need_gpu()
    n_anchor, n_cmp = mp.budget(keep)
    n_anchor = min(n_anchor, n)
    log(f"[select] G={G} n={n} K={K} keep={keep} mode={mode}")
    cl, s = _inputs(G, n, K, n_anchor, keep + n, quant)
    out = L.select(torch.from_numpy(cl).cuda(), torch.from_numpy(s).cuda(), n_anchor, n_cmp, K, mode)
    torch.cuda.synchronize()
    idx = out["idx"].cpu().numpy()
    cnt = out["count"].cpu().numpy()
    for g in range(G):
        ref, _ = mp.select(cl[g], s[g], n_cmp, K, "literal" if mode == 0 else "exact")
        assert cnt[g] == len(ref)
        assert idx[g, :cnt[g]].tolist() == ref
        assert np.all(idx[g, cnt[g]:] == -1)


@pytest.mark.gpu
def test_select_zero_budget_keeps_only_anchors():
    L = need_gpu()
    cl, s = _inputs(2, 576, 4, 50, 7, True)
    out = L.select(torch.from_numpy(cl).cuda(), torch.from_numpy(s).cuda(), 50, 0, 4, 0)
    idx = out["idx"].cpu().numpy()
    for g in range(2):
        assert idx[g, :50].tolist() == sorted(np.nonzero(cl[g] < 0)[0].tolist())


@pytest.mark.gpu
@pytest.mark.parametrize("wl,keep", [("tiny", 16), ("llava_next_7b", 64), ("llava15_13b", 128)])
def test_assemble_parity(wl, keep):
    L = need_gpu()
    w = get_workload(wl, keep=keep)
    G, n, K = w.score.G, w.score.n, w.score.K
    n_anchor, n_cmp = mp.budget(keep)
    log(f"[assemble] {wl} keep={keep}")
    cl, s = _inputs(G, n, K, n_anchor, 11, True)
    src = visual_src(w)
    text = text_rows(w)
    out = L.select(torch.from_numpy(cl).cuda(), torch.from_numpy(s).cuda(), n_anchor, n_cmp, K, 0,
                   tiles_per_sample=w.tiles_per_sample, src=src.cuda(), text=text.cuda())
    torch.cuda.synchronize()
    idx = [mp.select(cl[g], s[g], n_cmp, K)[0] for g in range(G)]
    x_ref, cu_ref = mp.assemble(src.float().numpy(), idx, text.float().numpy(), w.tiles_per_sample)
    cu = out["cu_seqlens"].cpu().numpy()
    assert cu.tolist() == cu_ref.tolist()
    x = out["x"][:cu[-1]].float().cpu().numpy()
    assert np.array_equal(x, x_ref)
