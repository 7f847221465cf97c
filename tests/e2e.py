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
