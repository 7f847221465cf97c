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


def gpu_pipeline(name: str, device="cuda:0", keep=None, n_layers=None, skip_p=None):
    """The GPU pipeline (score -> select/assemble -> host plan -> prefill) on a named
    workload's seeded inputs.  Returns the workload, the inputs (CPU copies of the
    vision taps), the device weights, the pipeline object and its step output."""
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
    plan = {}
    if w.skip["kind"] not in ("random_layer", "mask"):
        sa, sf = slc_tables(policy_lists(w.skip["policy"], dec.L, w.seed), dec.L)
        sel, tgt = _lib.slc_policy(sa, sf)
        s_sa = adaptive_scores(w, w.tiles_per_sample * cap)
        pol = SkipPolicy(kind="adaptive", s_sa=s_sa, slc_sel=sel, target=tgt, w1=w.skip["w1"],
                         w2=w.skip["w2"], T_skip=w.skip["T_skip"])
        plan = {"slc_attn": sa, "slc_ffn": sf, "s_sa": s_sa}
    else:
        plan = {"mask": layer_mask(w)}
        pol = SkipPolicy(kind="layer_mask", layer_mask=plan["mask"])
    bf16 = dec.dtype == "bf16"
    cfg = _lib.decoder_cfg(dec.L, dec.d, dec.H, dec.d_ff, _lib.BF16 if bf16 else _lib.F32, dec.eps, dec.theta)
    pipe = Pipeline(G=sc.G, n=sc.n, K=sc.K, keep=sc.keep, r_num=sc.r_num, r_den=sc.r_den,
                    kmeans_iter=sc.kmeans_iter, tiles_per_sample=w.tiles_per_sample,
                    n_text=w.n_text, quota_mode=w.quota_mode, dec=cfg, weights=Wd, device=dev)
    out = pipe.step(attn.to(dev), [f.to(dev) for f in feats], src, text, pol)
    torch.cuda.synchronize(dev)
    return {"w": w, "attn": attn, "feats": feats, "src": src, "text": text, "Wd": Wd, "pipe": pipe,
            "out": out, "plan": plan}


def oracle_plan(g):
    """The oracle's side of selection and skip planning on the same inputs as
    gpu_pipeline's result ``g``: kept tiles, packed input x (float64), cu_seqlens
    and the [L, rows] codes from the paper's rules."""
    w = g["w"]
    sc, dec = w.score, w.dec
    mode = "exact" if w.quota_mode == 1 else "literal"
    A = g["attn"].numpy()
    F = [f.float().numpy() for f in g["feats"]]
    tiles = [mp.prune_tile(A[i], [f[i] for f in F], sc.keep, sc.r_num, sc.r_den, sc.K,
                           sc.kmeans_iter, mode) for i in range(sc.G)]
    x, cu = mp.assemble(g["src"].float().cpu().numpy().astype(np.float64), [t["idx"] for t in tiles],
                        g["text"].float().cpu().numpy().astype(np.float64), w.tiles_per_sample)
    n_vis = [int(cu[b + 1] - cu[b]) - w.n_text for b in range(w.B)]
    per_sample = []
    if "mask" in g["plan"]:
        mask = g["plan"]["mask"]
        col = (mask[:, 0].astype(np.uint8) | (mask[:, 1].astype(np.uint8) << 1))
        per_sample = [np.repeat(col[:, None], n_vis[b], axis=1) for b in range(w.B)]
    else:
        na, nf = ak.slc_normalize(g["plan"]["slc_attn"], g["plan"]["slc_ffn"])
        m, sel_o = ak.skip_targets(na, nf)
        for b in range(w.B):
            c, _, _ = ak.plan(g["plan"]["s_sa"][b][:, :n_vis[b]], sel_o, m, w.skip["w1"], w.skip["w2"],
                              w.skip["T_skip"], dec.L)
            per_sample.append(c)
    codes = ak.pack_codes(per_sample, n_vis, w.n_text, dec.L)
    return {"tiles": tiles, "x": x, "cu": cu, "codes": codes}


def selection_equal(g, o) -> dict:
    out = g["out"]
    idx_gpu = out["select"]["idx"].cpu().numpy()
    cnt_gpu = out["select"]["count"].cpu().numpy()
    return {"idx_equal": all(idx_gpu[i, :cnt_gpu[i]].tolist() == list(t["idx"]) for i, t in enumerate(o["tiles"])),
            "cu_equal": list(out["cu"]) == list(o["cu"]),
            "codes_equal": bool(np.array_equal(out["codes"], o["codes"]))}


def oracle_layer_weights(g, l):
    """Layer l's synthetic weights (the seeded generator's bf16 values) as float64 host arrays."""
    return {k: v.float().cpu().numpy().astype(np.float64) for k, v in g["Wd"][l].items()}


def sample_errors(h, ref, cu):
    """max|h - ref| / max|ref| per sample."""
    return [float(np.max(np.abs(h[cu[b]:cu[b + 1]] - ref[cu[b]:cu[b + 1]])) /
                  max(np.max(np.abs(ref[cu[b]:cu[b + 1]])), 1e-30)) for b in range(len(cu) - 1)]


def run_end_to_end(name: str, device="cuda:0", keep=None, n_layers=None, skip_p=None):
    """Whole hot path on a named workload (GPU pipeline vs oracle pipeline).

    Inputs are the workload's seeded synthetic tensors (weights and rows are
    generated on the device; the generator gives the same bits on the host).
    The oracle takes its own skip plan from the paper's rule (a per-layer mask,
    or Algorithm 1's admission on the same S_sa and SLC tables) and runs the
    decoder in float64 with the workload's rounding recipe, one layer's
    weights at a time.
    """
    g = gpu_pipeline(name, device, keep, n_layers, skip_p)
    o = oracle_plan(g)
    w = g["w"]
    dec = w.dec
    bf16 = dec.dtype == "bf16"
    h_gpu = g["out"]["h"].cpu().numpy()
    h_ref = odec.prefill(o["x"], lambda l: oracle_layer_weights(g, l), o["cu"], o["codes"], dec,
                         recipe="bf16" if bf16 else "f32")
    res = selection_equal(g, o)
    res.update({"rel_err": sample_errors(h_gpu, h_ref, o["cu"]), "rows": int(o["cu"][-1]),
                "skipped_fraction": float((o["codes"] != 0).mean())})
    return res
