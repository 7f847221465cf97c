"""GPU projector on the kept rows (spider_project_kept, after spider_select's
text-only assembly) against the oracle's projector (pruning in the ViT feature
space before the projector).

Bars: kept rows land in the packed rows the assembly gives them, text rows and
boundaries as spider_select writes them (bit-exact), padding slots write
nothing; projected values within 1e-5 (fp32) / 1e-2 (bf16: the output is
rounded to bf16, 2^-8 of a value, plus rounding flips of the bf16 hidden rows)
of the float64 oracle, relative to the largest output of the sample.
"""
import numpy as np
import pytest
import torch

from oracle import msv_prune as mp
from oracle import projector as pj
from synth import get_workload
from synth.decoder_inputs import projector_inputs, projector_weights, text_rows
from synth.vision import vision_inputs
from gpu_common import need_gpu, oracle_tiles, log

CASES = {
    # name: (workload, keep, quota_mode)
    "tiny_fp32": ("tiny", 16, 0),
    "llava15_7b_keep128": ("llava15_7b", 128, 0),
    "llava15_7b_keep64_exact_budget": ("llava15_7b", 64, 1),
    "llava_next_5_tiles_keep128": ("llava_next_7b", 128, 0),
    "llava15_13b_batch8": ("llava15_13b", 128, 0),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_projected_assembly(case):
    L = need_gpu()
    wl, keep, qm = CASES[case]
    w = get_workload(wl, keep=keep)
    sc = w.score
    bf16 = w.dec.dtype == "bf16"
    log(f"[projector] case={case} G={sc.G} keep={keep} d_v={sc.d_v} d={w.dec.d}")
    attn, feats = vision_inputs(sc, w.seed)
    pin = projector_inputs(w)
    proj = projector_weights(w)
    text = text_rows(w)
    n_anchor, n_cmp = mp.budget(keep, sc.r_num, sc.r_den)
    n_anchor = min(n_anchor, sc.n)
    cap = min(sc.n, n_anchor + n_cmp + sc.K)
    sco = L.score(attn.cuda(), [f.cuda() for f in feats], n_anchor, sc.K, sc.kmeans_iter)
    B = sc.G // w.tiles_per_sample
    x = torch.full((B * (w.tiles_per_sample * cap + w.n_text), w.dec.d), float("nan"),
                   dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
    sel = L.select(sco["cluster"], sco["s"], n_anchor, n_cmp, sc.K, qm, cap, w.tiles_per_sample,
                   text=text.cuda(), text_only=True, x_out=x)
    L.project_kept(sel, pin.cuda(), {k: v.cuda() for k, v in proj.items()}, w.tiles_per_sample, w.n_text)
    torch.cuda.synchronize()
    cu = sel["cu_seqlens"].cpu().numpy()
    rows = int(cu[-1])
    xg = x[:rows].float().cpu().numpy()
    assert np.all(np.isnan(x[rows:].float().cpu().numpy()))

    ref_tiles = oracle_tiles(attn, feats, keep, sc.r_num, sc.r_den, sc.K, sc.kmeans_iter,
                             "literal" if qm == 0 else "exact")
    idx = [t["idx"] for t in ref_tiles]
    P = {k: v.float().numpy() for k, v in proj.items()}
    xo, cuo = pj.assemble_projected(pin.float().numpy(), idx, text.float().numpy(), w.tiles_per_sample,
                                    P["w1"], P["b1"], P["w2"], P["b2"], recipe="bf16" if bf16 else "f32")
    assert np.array_equal(cu, cuo)
    tol = 1e-2 if bf16 else 1e-5
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        n_vis = s1 - s0 - w.n_text
        assert np.array_equal(xg[s1 - w.n_text:s1], xo[s1 - w.n_text:s1]), f"sample {b}: text rows"
        v, vo = xg[s0:s0 + n_vis], xo[s0:s0 + n_vis]
        assert np.all(np.isfinite(v)), f"sample {b}: kept rows not written"
        err = float(np.max(np.abs(v - vo)) / np.max(np.abs(vo)))
        log(f"  sample {b}: {n_vis} projected rows, max rel err {err:.2e}")
        assert err <= tol, f"sample {b}: {err}"
