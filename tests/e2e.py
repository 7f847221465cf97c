"""End-to-end pass (score -> select/assemble -> skip plan -> prefill) vs the oracle.

Used by the GPU test suite and by the smoke entry point.
"""
import numpy as np
import torch

from oracle import asl_skip as ak
from oracle import decoder as odec
from oracle import msv_prune as mp
from synth import get_workload
from synth.decoder_inputs import all_weights, text_rows, visual_src
from synth.skip_inputs import layer_mask
from synth.vision import vision_inputs


def run_tiny_end_to_end(device="cuda:0", keep=16):
    from paper_2609_34977_amd import _lib
    from paper_2609_34977_amd.pipeline import Pipeline, SkipPolicy

    w = get_workload("tiny", keep=keep)
    sc, dec = w.score, w.dec
    attn, feats = vision_inputs(sc, w.seed)
    src, text = visual_src(w), text_rows(w)
    W = all_weights(dec, w.seed)
    mask = layer_mask(w)

    # ---- GPU
    dev = torch.device(device)
    Wd = [{k: v.to(dev) for k, v in lw.items()} for lw in W]
    cfg = _lib.decoder_cfg(dec.L, dec.d, dec.H, dec.d_ff, _lib.F32, dec.eps, dec.theta)
    pipe = Pipeline(G=sc.G, n=sc.n, K=sc.K, keep=keep, r_num=sc.r_num, r_den=sc.r_den,
                    kmeans_iter=sc.kmeans_iter, tiles_per_sample=w.tiles_per_sample,
                    n_text=w.n_text, quota_mode=w.quota_mode, dec=cfg, weights=Wd, device=dev)
    out = pipe.step(attn.to(dev), [f.to(dev) for f in feats], src.to(dev), text.to(dev),
                    SkipPolicy(kind="layer_mask", layer_mask=mask))
    torch.cuda.synchronize(dev)
    h_gpu = out["h"].cpu().numpy()
    idx_gpu = out["select"]["idx"].cpu().numpy()
    cnt_gpu = out["select"]["count"].cpu().numpy()

    # ---- oracle
    tiles = [mp.prune_tile(attn[g].numpy(), [f[g].numpy() for f in feats], keep, sc.r_num,
                           sc.r_den, sc.K, sc.kmeans_iter) for g in range(sc.G)]
    x, cu = mp.assemble(src.numpy().astype(np.float64), [t["idx"] for t in tiles],
                        text.numpy().astype(np.float64), w.tiles_per_sample)
    col = (mask[:, 0].astype(np.uint8) | (mask[:, 1].astype(np.uint8) << 1))
    per_sample = [np.repeat(col[:, None], int(cu[b + 1] - cu[b]) - w.n_text, axis=1)
                  for b in range(w.B)]
    codes = ak.pack_codes(per_sample, [int(cu[b + 1] - cu[b]) - w.n_text for b in range(w.B)],
                          w.n_text, dec.L)
    Wo = [{k: v.numpy().astype(np.float64) for k, v in lw.items()} for lw in W]
    h_ref = odec.prefill(x, Wo, cu, codes, dec, recipe="f32")

    res = {"idx_equal": all(idx_gpu[g, :cnt_gpu[g]].tolist() == tiles[g]["idx"] for g in range(sc.G)),
           "cu_equal": list(out["cu"]) == list(cu),
           "codes_equal": bool(np.array_equal(out["codes"], codes)),
           "rel_err": float(np.max(np.abs(h_gpu - h_ref)) / np.max(np.abs(h_ref))),
           "rows": int(cu[-1])}
    return res


def run_end_to_end(name: str, device="cuda:0", keep=None, n_layers=None, skip_p=None, spread=False):
    """Whole hot path on a named workload (GPU pipeline vs oracle pipeline).

    Inputs are the workload's seeded synthetic tensors (weights and rows are
    generated on the device; the generator gives the same bits on the host).
    The oracle takes its own skip plan from the paper's rule (a per-layer mask,
    or Algorithm 1's admission on the same S_sa and SLC tables) and runs the
    decoder in float64 with the workload's rounding recipe, one layer's
    weights at a time.  With ``spread`` the oracle also runs in float32 and the
    result reports how far that evaluation lands from the float64 one (the
    rounding-order sensitivity of the recipe at this depth).
    """
    from paper_2609_34977_amd import _lib
    from paper_2609_34977_amd.pipeline import Pipeline, SkipPolicy
    from synth.decoder_inputs import layer_weights
    from synth.skip_inputs import adaptive_scores, policy_lists, slc_tables

    w = get_workload(name, keep=keep, L=n_layers, skip_p=skip_p)
    sc, dec = w.score, w.dec
    dev = torch.device(device)
    attn, feats = vision_inputs(sc, w.seed)
    src, text = visual_src(w, dev), text_rows(w, dev)
    Wd = [layer_weights(dec, l, w.seed, dev) for l in range(dec.L)]
    cap = min(sc.n, sc.keep + sc.K)
    adaptive = w.skip["kind"] not in ("random_layer", "mask")
    if adaptive:
        sa, sf = slc_tables(policy_lists(w.skip["policy"], dec.L, w.seed), dec.L)
        sel, tgt = _lib.slc_policy(sa, sf)
        s_sa = adaptive_scores(w, w.tiles_per_sample * cap)
        pol = SkipPolicy(kind="adaptive", s_sa=s_sa, slc_sel=sel, target=tgt, w1=w.skip["w1"],
                         w2=w.skip["w2"], T_skip=w.skip["T_skip"])
    else:
        mask = layer_mask(w)
        pol = SkipPolicy(kind="layer_mask", layer_mask=mask)
    bf16 = dec.dtype == "bf16"
    cfg = _lib.decoder_cfg(dec.L, dec.d, dec.H, dec.d_ff, _lib.BF16 if bf16 else _lib.F32, dec.eps, dec.theta)
    pipe = Pipeline(G=sc.G, n=sc.n, K=sc.K, keep=sc.keep, r_num=sc.r_num, r_den=sc.r_den,
                    kmeans_iter=sc.kmeans_iter, tiles_per_sample=w.tiles_per_sample,
                    n_text=w.n_text, quota_mode=w.quota_mode, dec=cfg, weights=Wd, device=dev)
    out = pipe.step(attn.to(dev), [f.to(dev) for f in feats], src, text, pol)
    torch.cuda.synchronize(dev)
    h_gpu = out["h"].cpu().numpy()
    idx_gpu = out["select"]["idx"].cpu().numpy()
    cnt_gpu = out["select"]["count"].cpu().numpy()

    # ---- oracle
    mode = "exact" if w.quota_mode == 1 else "literal"
    A = attn.numpy()
    F = [f.float().numpy() for f in feats]
    tiles = [mp.prune_tile(A[g], [f[g] for f in F], sc.keep, sc.r_num, sc.r_den, sc.K,
                           sc.kmeans_iter, mode) for g in range(sc.G)]
    x, cu = mp.assemble(src.float().cpu().numpy().astype(np.float64), [t["idx"] for t in tiles],
                        text.float().cpu().numpy().astype(np.float64), w.tiles_per_sample)
    n_vis = [int(cu[b + 1] - cu[b]) - w.n_text for b in range(w.B)]
    per_sample = []
    if adaptive:
        na, nf = ak.slc_normalize(sa, sf)
        m, sel_o = ak.skip_targets(na, nf)
        for b in range(w.B):
            c, _, _ = ak.plan(s_sa[b][:, :n_vis[b]], sel_o, m, w.skip["w1"], w.skip["w2"],
                              w.skip["T_skip"], dec.L)
            per_sample.append(c)
    else:
        col = (mask[:, 0].astype(np.uint8) | (mask[:, 1].astype(np.uint8) << 1))
        per_sample = [np.repeat(col[:, None], n_vis[b], axis=1) for b in range(w.B)]
    codes = ak.pack_codes(per_sample, n_vis, w.n_text, dec.L)

    def layer(l):
        return {k: v.float().cpu().numpy().astype(np.float64) for k, v in Wd[l].items()}

    h_ref = odec.prefill(x, layer, cu, codes, dec, recipe="bf16" if bf16 else "f32")

    def per_sample(h):
        return [float(np.max(np.abs(h[cu[b]:cu[b + 1]] - h_ref[cu[b]:cu[b + 1]])) /
                      max(np.max(np.abs(h_ref[cu[b]:cu[b + 1]])), 1e-30)) for b in range(w.B)]

    errs = per_sample(h_gpu)
    spread_errs = None
    if spread:
        h32 = odec.prefill(x.astype(np.float32), lambda l: {k: v.astype(np.float32) for k, v in layer(l).items()},
                           cu, codes, dec, recipe="bf16" if bf16 else "f32", dtype=np.float32)
        spread_errs = per_sample(h32.astype(np.float64))
    return {"idx_equal": all(idx_gpu[g, :cnt_gpu[g]].tolist() == list(tiles[g]["idx"]) for g in range(sc.G)),
            "cu_equal": list(out["cu"]) == list(cu),
            "codes_equal": bool(np.array_equal(out["codes"], codes)),
            "rel_err": errs, "oracle_f32_spread": spread_errs, "rows": int(cu[-1]),
            "skipped_fraction": float((codes != 0).mean())}
