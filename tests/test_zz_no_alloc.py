"""spider_score_noalloc (static device scratch, no allocation) against spider_score.

Two calls of the no-allocation entry point in a row, the second on a smaller
input (fewer tiles, a smaller budget, another seed) so it runs over the first
call's stale scratch; each must give spider_score's outputs bit for bit (the
same kernels on the same inputs: anchor scores, clusters, s and m).
"""
import numpy as np
import pytest
import torch

from synth import get_workload
from synth.vision import vision_inputs
from gpu_common import need_gpu, log

CALLS = [
    # (workload, keep, seed): LLaVA-NeXT's five tiles, then one LLaVA-1.5 tile
    ("llava_next_7b", 128, 0),
    ("llava15_7b", 64, 1),
]


@pytest.mark.gpu
def test_score_noalloc_matches_score_on_two_calls():
    L = need_gpu()
    inputs, refs = [], []
    for wl, keep, seed in CALLS:
        w = get_workload(wl, keep=keep)
        attn, feats = vision_inputs(w.score, seed)
        attn, feats = attn.cuda(), [f.cuda() for f in feats]
        n_anchor = (keep * w.score.r_num) // w.score.r_den
        inputs.append((attn, feats, n_anchor, w.score.K, w.score.kmeans_iter))
        refs.append(L.score(attn, feats, n_anchor, w.score.K, w.score.kmeans_iter))
    torch.cuda.synchronize()
    # the two no-allocation calls back to back on the same stream
    got = [L.score(a, f, na, K, it, noalloc=True) for a, f, na, K, it in inputs]
    torch.cuda.synchronize()
    for (wl, keep, seed), (_, _, na, _, _), r, g in zip(CALLS, inputs, refs, got):
        log(f"[noalloc] {wl} keep={keep} seed={seed} G={r['a'].shape[0]}")
        for k in ("a", "cluster", "s", "m"):
            assert torch.equal(r[k], g[k]), (wl, k)
        # every tile has its n_anchor anchors: the outputs are this call's, not stale buffers
        assert np.all((g["cluster"] < 0).sum(1).cpu().numpy() == na)
