"""Benchmark of the pruned-and-skipped multimodal prefill on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload stress] [--keep 288] [--skip-p 0.25]

With no workload flags the step is the largest single-GPU configuration
that both prunes and skips: the high-resolution stress shape (batch 4 x 2880
visual tokens in 5 AnyRes tiles of 576, keep 288 per tile, LLaVA-1.5-7B-shaped
decoder, each of the 2 x 32 sub-layer slots bypassed by every visual row with
probability 0.25); the same JSON line then carries the LLaVA-1.5-7B keep-128
batch-1 step as an extra field (`llava15_7b_keep128`).

One step = the whole hot path over one batch of synthetic LLaVA-shaped input
already resident in HBM: multi-layer scoring of the vision tokens
(spider_score), quota/selection/assembly of [kept visual | text]
(spider_select), one device-to-host copy of the sample boundaries, the skip
plan on the host, and the skip-aware decoder prefill (spider_prefill).

Prints one JSON line.  `value` is decoder rows (kept visual + text tokens)
prefilled per second; `roofline` reports the dominant kernel class against
its roofline (kernel times from HIP events recorded around every launch on
the launch stream, over the timed steps); `cpu_baseline` times the CPU oracle
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
FP32_PEAK_TFLOPS = 157.3
METRIC = "pruned+skipped prefill tokens/s and ms/sample; % MFMA peak, % HBM peak"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default=None,
                   help="workload name (default: the stress shape at keep 288, skip 0.25)")
    p.add_argument("--keep", type=int, default=None)
    p.add_argument("--layers", type=int, default=None)
    p.add_argument("--skip-p", type=float, default=None)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-layers", type=int, default=4)
    p.add_argument("--no-secondary", action="store_true",
                   help="do not add the LLaVA-1.5-7B keep-128 step to the default line")
    p.add_argument("--copy-probe-mib", type=int, default=0,
                   help="run one plain device copy of this size after warm-up (counter calibration)")
    p.add_argument("--score-sweep", action="store_true",
                   help="instead of the step: time scoring over 20/64/256/512 tiles (one JSON line each)")
    p.add_argument("--select-sweep", action="store_true",
                   help="instead of the step: time quota/selection (spider_select) and the gather of the kept "
                        "rows over 20/64/256/512 tiles at keep 128 and keep-all (one JSON line each)")
    p.add_argument("--curve", action="store_true",
                   help="instead of the headline step: the stress shape over keep {576, 288, 144, 64} per "
                        "tile x skip {0, 0.25, 0.5} (one JSON line per point, weights shared)")
    p.add_argument("--colmean-sweep", action="store_true",
                   help="instead of the step: time the anchor scores of encoders without [CLS] "
                        "(column means of 16-head attention maps) over 1/8/64 tiles of 576 and 1024 patches")
    p.add_argument("--online", action="store_true",
                   help="decoder mask from the online skip controller on the device (logit lens over a "
                        "32000-token unembedding, w1=3, w2=1, T_skip=20) instead of the workload's mask")
    p.add_argument("--vocab", type=int, default=32000)
    p.add_argument("--decode", type=int, default=0,
                   help="after the step, also time this many greedy decode steps (LM head included) over the "
                        "KV cache of the pruned and skipped prefill; reported in the `decode` field")
    p.add_argument("--vendor-gemm", action="store_true",
                   help="context, not the benchmark step: the library's per-launch decoder GEMM times in a "
                        "prefill without skipping beside torch.nn.functional.linear (hipBLASLt) on the same "
                        "shapes, one JSON line per workload")
    p.add_argument("--projector", action="store_true",
                   help="prune before the projector: the step also runs LLaVA's two-layer GELU projector "
                        "(ViT width -> decoder width) on the kept rows only")
    return p.parse_args()


def online_policy(w, dev, V):
    """Online controller policy: the paper's operating point (w1/w2 = 3, T_skip = 20) with the
    workload's replaced-layer list (or a drawn one), and an unembedding of V rows."""
    from synth.online_inputs import unembed
    from synth.skip_inputs import REPLACED_LAYERS, policy_lists, slc_tables, synthetic_policy
    from paper_2609_34977_amd import _lib
    from paper_2609_34977_amd.pipeline import SkipPolicy

    L = w.dec.L
    name = w.skip.get("policy", w.name)
    lists = policy_lists(name, L, w.seed) if name in REPLACED_LAYERS else synthetic_policy(L, 7, w.seed)
    sa, sf = slc_tables(lists, L)
    sel, tgt = _lib.slc_policy(sa, sf)
    return SkipPolicy(kind="online", slc_sel=sel, target=tgt, w1=3.0, w2=1.0, T_skip=20.0,
                      w_unembed=unembed(w.dec, V, w.seed, dev))


def build_inputs(w, dev, weights=None):
    from synth.decoder_inputs import layer_weights, text_rows, visual_src
    from synth.skip_inputs import (adaptive_scores, layer_mask, policy_lists, slc_tables)
    from synth.vision import vision_inputs
    from paper_2609_34977_amd import _lib
    from paper_2609_34977_amd.pipeline import SkipPolicy

    attn, feats = vision_inputs(w.score, w.seed)
    attn, feats = attn.to(dev), [f.to(dev) for f in feats]
    src, text = visual_src(w, dev), text_rows(w, dev)
    W = weights if weights is not None else [layer_weights(w.dec, l, w.seed, dev) for l in range(w.dec.L)]
    if w.skip["kind"] in ("random_layer", "mask"):
        pol = SkipPolicy(kind="layer_mask", layer_mask=layer_mask(w))
    else:
        L = w.dec.L
        sa, sf = slc_tables(policy_lists(w.skip["policy"], L, w.seed), L)
        sel, tgt = _lib.slc_policy(sa, sf)
        cap = min(w.score.n, w.score.keep + w.score.K)
        pol = SkipPolicy(kind="adaptive", s_sa=adaptive_scores(w, w.tiles_per_sample * cap),
                         slc_sel=sel, target=tgt, w1=w.skip["w1"], w2=w.skip["w2"],
                         T_skip=w.skip["T_skip"])
    return attn, feats, src, text, W, pol


def algorithmic(w, cu, codes, admit=None, V=0):
    """Per kernel class: (bytes, flops) summed over one step, from the per-layer row counts.
    With the online controller (admit given) the logit-lens GEMM of every window layer reads
    the unembedding [V, d] and the candidate rows once and writes fp32 logits."""
    d, f, L, dh = w.dec.d, w.dec.d_ff, w.dec.L, w.dec.dh
    rows = int(cu[-1])
    out = {k: [0.0, 0.0] for k in ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down", "attention",
                                   "gemm_lens")}
    if admit is not None:
        vis = np.concatenate([np.arange(cu[b], cu[b + 1] - w.n_text) for b in range(len(cu) - 1)])
        for l in range(L // 2):
            nc = int(np.sum((admit[vis] < 0) | (admit[vis] >= l)))
            if nc:
                out["gemm_lens"][0] += V * d * 2 + nc * d * 2 + nc * V * 4
                out["gemm_lens"][1] += 2.0 * V * d * nc
    pos = np.concatenate([np.arange(cu[b + 1] - cu[b]) for b in range(len(cu) - 1)])
    for l in range(L):
        A = codes[l] & 1 == 0
        F = codes[l] & 2 == 0
        nA, nF = int(A.sum()), int(F.sum())
        if nA:
            out["gemm_qkv"][0] += 3 * d * d * 2 + rows * d * 2 + (nA + 2 * rows) * d * 2
            out["gemm_qkv"][1] += 2.0 * d * d * (nA + 2 * rows)
            out["gemm_o"][0] += d * d * 2 + nA * d * 2 + nA * d * 4
            out["gemm_o"][1] += 2.0 * d * d * nA
            out["attention"][0] += nA * d * 2 * 2 + 2 * rows * d * 2
            out["attention"][1] += 4.0 * d * float((pos[A] + 1).sum())
        if nF:
            out["gemm_gateup"][0] += 2 * f * d * 2 + nF * d * 2 + nF * f * 2
            out["gemm_gateup"][1] += 2.0 * 2 * f * d * nF
            out["gemm_down"][0] += d * f * 2 + nF * f * 2 + nF * d * 4
            out["gemm_down"][1] += 2.0 * d * f * nF
    return out


def cpu_baseline(w, n_layers: int, W_dev=None):
    """Oracle (as it is) on a bounded sample: scoring+selection of every tile and
    n_layers of the decoder with the oracle's own skip plan for the workload (the
    per-layer mask, or Algorithm 1's admission on the same S_sa and SLC tables),
    decoder time scaled to all layers.  Decoder weights are the benchmark's own
    (copied to host memory) when given."""
    import threadpoolctl
    from oracle import asl_skip as ak
    from oracle import decoder as odec
    from oracle import msv_prune as mp
    from synth.decoder_inputs import layer_weights, text_rows, visual_src
    from synth.vision import vision_inputs
    from synth.skip_inputs import adaptive_scores, layer_mask, policy_lists, slc_tables

    cores = len(os.sched_getaffinity(0))
    attn, feats = vision_inputs(w.score, w.seed)
    A = attn.numpy()
    Fs = [f.float().numpy() for f in feats]
    src, text = visual_src(w).float().numpy(), text_rows(w).float().numpy()
    if W_dev is not None:
        Wl = [{k: v.float().cpu().numpy() for k, v in W_dev[l].items()} for l in range(n_layers)]
    else:
        Wl = [{k: v.float().numpy() for k, v in layer_weights(w.dec, l, w.seed).items()}
              for l in range(n_layers)]
    mode = "exact" if w.quota_mode == 1 else "literal"
    with threadpoolctl.threadpool_limits(cores):
        torch.set_num_threads(cores)
        t0 = time.perf_counter()
        tiles = [mp.prune_tile(A[g], [f[g] for f in Fs], w.score.keep, w.score.r_num,
                               w.score.r_den, w.score.K, w.score.kmeans_iter, mode)
                 for g in range(w.score.G)]
        x, cu = mp.assemble(src, [t["idx"] for t in tiles], text, w.tiles_per_sample)
        n_vis = [int(cu[b + 1] - cu[b]) - w.n_text for b in range(w.B)]
        if w.skip["kind"] in ("random_layer", "mask"):
            m = layer_mask(w)
            col = (m[:, 0].astype(np.uint8) | (m[:, 1].astype(np.uint8) << 1))
            per_sample = [np.repeat(col[:, None], n_vis[b], axis=1) for b in range(w.B)]
        else:
            L = w.dec.L
            cap = min(w.score.n, w.score.keep + w.score.K)
            sa, sf = slc_tables(policy_lists(w.skip["policy"], L, w.seed), L)
            na, nf = ak.slc_normalize(sa, sf)
            tgt, sel = ak.skip_targets(na, nf)
            s_sa = adaptive_scores(w, w.tiles_per_sample * cap)
            per_sample = [ak.plan(s_sa[b][:, :n_vis[b]], sel, tgt, w.skip["w1"], w.skip["w2"],
                                  w.skip["T_skip"], L)[0] for b in range(w.B)]
        codes = ak.pack_codes(per_sample, n_vis, w.n_text, w.dec.L)
        t1 = time.perf_counter()
        odec.prefill(x.astype(np.float32), Wl, cu, codes, w.dec, recipe="bf16",
                     dtype=np.float32, n_layers=n_layers)
        t2 = time.perf_counter()
    t_step = (t1 - t0) + (t2 - t1) * w.dec.L / n_layers
    rows = int(cu[-1])
    return {"value": rows / t_step, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "ms_per_step_extrapolated": t_step * 1e3,
            "extrapolated": n_layers < w.dec.L,
            "sample": (f"oracle scoring+selection+skip plan of all {w.score.G} tile(s) "
                       f"({(t1 - t0):.2f} s) plus decoder layers 0..{n_layers - 1} of {w.dec.L} "
                       f"({(t2 - t1):.2f} s, float32 with the bf16 rounding recipe, the oracle's own "
                       f"skip codes), decoder time extrapolated by {w.dec.L}/{n_layers}; {rows} rows")}


def kmeans_passes(attn, feats, n_anchor, K, max_iter):
    """Lloyd passes per tile that read the features in a call allowed max_iter of them:
    pass 1, then every pass up to and including the first that changes no assignment
    (the launches after it return at once).  Found from the assignments after
    1, 2, ... passes, each its own call."""
    from paper_2609_34977_amd import _lib

    prev, passes = None, None
    for k in range(1, max_iter + 1):
        cl = _lib.score(attn, feats, n_anchor, K, k)["cluster"]
        if prev is None:
            passes = torch.full((cl.shape[0],), max_iter, dtype=torch.int64, device=cl.device)
        else:
            settled = (cl == prev).all(dim=1) & (passes == max_iter)
            passes[settled] = k
        prev = cl
    return passes.cpu()


def score_sweep(w, dev, args):
    """Scoring (spider_score) over many tiles: time per call, and the compulsory
    HBM bytes (CLS attention + every tapped layer's features, read once, plus
    the outputs) over that time.  Tiles are the workload's synthetic tiles
    repeated up to G (20 distinct tiles are generated).

    Per kernel class also the effective bytes its design reads from HBM (each
    input row once per pass that reads it; L2 re-reads of the anchors and
    centroids not counted) and the rate they imply:
      score_prep     CLS rows + every tapped layer's rows, a_i and 1/|F| out
      anchor_topk    a in, anchor and non-anchor lists out
      anchor_maxsim  the last layer's rows, m out
      kmeans         the last layer's non-anchor rows once per working pass
      score_final    every tapped layer's non-anchor rows twice (cluster sums,
                     scores), cluster ids and scores out"""
    import dataclasses
    from synth.vision import vision_inputs
    from paper_2609_34977_amd import _lib

    sc = w.score
    base = dataclasses.replace(sc, G=20)
    attn0, feats0 = vision_inputs(base, w.seed)
    attn0, feats0 = attn0.to(dev), [f.to(dev) for f in feats0]
    n_anchor, _ = _lib.budget(sc.keep, sc.r_num, sc.r_den)
    na = min(n_anchor, sc.n)
    passes0 = kmeans_passes(attn0, feats0, na, sc.K, sc.kmeans_iter)
    for G in (20, 64, 256, 512):
        reps = (G + 19) // 20
        attn = attn0.repeat(reps, 1, 1)[:G].contiguous()
        feats = [f.repeat(reps, 1, 1)[:G].contiguous() for f in feats0]
        passes = int(passes0.repeat(reps)[:G].sum())
        for _ in range(2):
            _lib.score(attn, feats, na, sc.K, sc.kmeans_iter)
        torch.cuda.synchronize()
        _lib.profile_mask(None)
        _lib.profile_enable(True)
        iters = 5
        t0 = time.perf_counter()
        for _ in range(iters):
            _lib.score(attn, feats, na, sc.K, sc.kmeans_iter)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        prof = _lib.profile_read()
        _lib.profile_enable(False)
        ms = (t1 - t0) * 1e3 / iters
        H, n, dv = attn.shape[1], sc.n, feats[0].shape[2]
        es, nl, m = feats[0].element_size(), len(feats), n - na
        byts = G * (H * (n + 1) * 4 + nl * n * dv * es + 16 * n)
        row = dv * es
        eff = {"score_prep": G * (H * n * 4 + nl * n * row + (1 + nl) * n * 4),
               "anchor_topk": G * 3 * n * 4,
               "anchor_maxsim": G * (n * row + n * 4),
               "kmeans": passes * m * row,
               "score_final": G * (2 * nl * m * row + 8 * n)}
        kms = {k: round(v[1] / iters, 4) for k, v in prof.items() if v[0]}
        kgb = {k: round(eff[k] / (kms[k] * 1e-3) / 1e9, 1) for k in eff if kms.get(k)}
        ach = byts / (ms * 1e-3) / 1e9
        print(json.dumps({"mode": "score_sweep", "tiles": G, "ms_per_call": ms,
                          "compulsory_bytes": byts, "achieved_GBs": ach, "frac_of_hbm_peak": ach / HBM_PEAK_GBS,
                          "kernel_ms_per_call": kms, "kmeans_working_passes": passes,
                          "kernel_effective_bytes": eff, "kernel_effective_GBs": kgb}), flush=True)
        del attn, feats
        torch.cuda.empty_cache()


def select_sweep(w, dev, args):
    """Quota/selection (select_kernel) and the gather of the kept rows into the packed
    decoder input (assemble_kernel) over G tiles, from the workload's own score
    outputs repeated up to G.  Algorithmic bytes: selection reads cluster ids and
    scores and writes the kept indices and counts (12 n + 4 cap per tile); the
    gather reads and writes every kept row once (2 x rows x d_model x 2 bytes)
    plus the text rows."""
    import dataclasses
    from synth.decoder_inputs import text_rows, visual_src
    from synth.vision import vision_inputs
    from paper_2609_34977_amd import _lib

    sc = w.score
    for keep in (128, sc.n):
        base = dataclasses.replace(sc, G=20, keep=keep)
        attn0, feats0 = vision_inputs(base, w.seed)
        n_anchor, n_cmp = _lib.budget(keep, sc.r_num, sc.r_den)
        n_anchor = min(n_anchor, sc.n)
        r0 = _lib.score(attn0.to(dev), [f.to(dev) for f in feats0], n_anchor, sc.K, sc.kmeans_iter)
        wl = dataclasses.replace(w, score=dataclasses.replace(sc, G=20))
        src0 = visual_src(wl, dev)
        for G in (20, 64, 256, 512):  # multiples of the 4 tiles per sample
            reps = (G + 19) // 20
            cl = r0["cluster"].repeat(reps, 1)[:G].contiguous()
            sv = r0["s"].repeat(reps, 1)[:G].contiguous()
            src = src0.repeat(reps, 1, 1)[:G].contiguous()
            tps = 4  # four tiles per sample (AnyRes-like): at most 255 samples per call
            text = text_rows(dataclasses.replace(w, B=G // tps), dev)
            cap = min(sc.n, n_anchor + n_cmp + sc.K)
            for _ in range(2):
                _lib.select(cl, sv, n_anchor, n_cmp, sc.K, w.quota_mode, cap, tps, src, text)
            torch.cuda.synchronize()
            _lib.profile_mask(["select", "assemble"])
            _lib.profile_enable(True)
            iters = 5
            for _ in range(iters):
                out = _lib.select(cl, sv, n_anchor, n_cmp, sc.K, w.quota_mode, cap, tps, src, text)
            torch.cuda.synchronize()
            prof = _lib.profile_read()
            _lib.profile_enable(False)
            _lib.profile_mask(None)
            kept = int(out["count"].sum())
            d = src.shape[-1]
            sel_bytes = G * (12 * sc.n + 4 * cap)
            gat_bytes = 2 * (kept + (G // tps) * w.n_text) * d * src.element_size()
            t_sel = prof["select"][1] / iters
            t_gat = prof["assemble"][1] / iters
            print(json.dumps({"mode": "select_sweep", "tiles": G, "keep_per_tile": keep, "kept_rows": kept,
                              "select_ms": t_sel, "select_bytes": sel_bytes,
                              "select_frac_of_hbm_peak": sel_bytes / (t_sel * 1e-3) / 1e9 / HBM_PEAK_GBS,
                              "gather_ms": t_gat, "gather_bytes": gat_bytes,
                              "gather_frac_of_hbm_peak": gat_bytes / (t_gat * 1e-3) / 1e9 / HBM_PEAK_GBS}),
                  flush=True)
            del cl, sv, src, text, out
            torch.cuda.empty_cache()


def curve(args, dev):
    """The stress shape (batch 4 x 5 tiles of 576) over keep per tile {576, 288, 144, 64}
    x skip fraction {0, 0.25, 0.5}: one JSON line per point with the step time and the
    dominant kernel class against its roofline (weights generated once)."""
    from synth import get_workload
    W = None
    for keep in (576, 288, 144, 64):
        for p in (0.0, 0.25, 0.5):
            w = get_workload("stress", keep=keep, L=args.layers, skip_p=p)
            res, W = run_step(w, args, dev, weights=W, cpu=False)
            r = {"mode": "curve", "keep_per_tile": keep, "skip_p": p, "ms_per_step": res["ms_per_step"],
                 "tokens_per_s": res["value"], "decoder_rows": res["config"]["decoder_rows"],
                 "skipped_sublayer_slots": res["config"]["skipped_sublayer_slots"],
                 "prefill_tflop_per_step": res["prefill_tflop_per_step"], "roofline": res["roofline"],
                 "kernel_ms_per_step": res["kernel_ms_per_step"]}
            print(json.dumps(r), flush=True)


def decode_latency(w, pipe, out, dev, args):
    """Greedy decoding after the step's prefill: spider_prefill_kv fills the KV cache of
    the pruned and skipped prompt, then args.decode steps of spider_decode_step (one token
    per sample, LM head over a vocabulary of args.vocab rows, arg max fed back through a
    synthetic embedding table).  Reports time per decode step (HIP events around the loop)."""
    from paper_2609_34977_amd import _lib
    from synth.online_inputs import unembed
    from synth.counter_rng import normal_bf16

    cfg = pipe.dec
    cu, codes = out["cu"], out["codes"]
    rows, B = int(cu[-1]), len(cu) - 1
    x = out["select"]["x"][:rows]
    cap = int(max(cu[1:] - cu[:-1])) + args.decode + 1
    kv = _lib.kv_cache(cfg, B, cap, dev)
    wu = unembed(w.dec, args.vocab, w.seed, dev)
    fn = torch.ones(cfg.d, dtype=torch.float32, device=dev)
    emb = normal_bf16((args.vocab, cfg.d), w.seed, 4800, 0.02, device=dev)   # token embedding table
    _lib.prefill_kv(cfg, None, cu, x, codes, kv, weight_table=pipe.wtable)
    lens = (cu[1:] - cu[:-1]).astype(np.int32)
    tok = torch.zeros(B, dtype=torch.int64, device=dev)
    ws = _lib.decode_workspace(cfg, B, cap, args.vocab, dev)
    # untimed warm-up steps (first launches of the decode kernels); the timed
    # steps then rewrite the same cache positions from the same first token
    for t in range(3):
        _lib.decode_step(cfg, None, lens + t, emb[tok], kv, fn, wu, weight_table=pipe.wtable, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for t in range(args.decode):
        _, _, nxt = _lib.decode_step(cfg, None, lens + t, emb[tok], kv, fn, wu, weight_table=pipe.wtable,
                                     workspace=ws)
        tok = nxt.long()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.decode
    return {"steps": args.decode, "ms_per_step": ms, "tokens_per_s": B / (ms * 1e-3), "batch": B,
            "cache_rows_per_sample": [int(v) for v in (cu[1:] - cu[:-1])], "vocab": args.vocab,
            "weights_bytes_per_step": 2 * (w.dec.L * (4 * w.dec.d ** 2 + 3 * w.dec.d * w.dec.d_ff)
                                           + args.vocab * w.dec.d)}


def colmean_sweep(dev):
    """spider_anchor_colmean over G tiles of [16, n, n] fp32 maps: time per call (HIP events
    around its two launches) and the algorithmic bytes (every map element read once, the
    scores written once) over that time."""
    from synth.vision import attention_maps
    from paper_2609_34977_amd import _lib

    H = 16
    for n in (576, 1024):
        for G in (1, 8, 64):
            A = attention_maps(G, H, n, seed=0, device=dev)
            out = torch.empty(G, n, dtype=torch.float32, device=dev)
            for _ in range(3):
                _lib.anchor_colmean(A, out)
            torch.cuda.synchronize()
            _lib.profile_mask(["anchor_colmean"])
            _lib.profile_enable(True)
            iters = 20
            t0 = time.perf_counter()
            for _ in range(iters):
                _lib.anchor_colmean(A, out)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            prof = _lib.profile_read()["anchor_colmean"]
            _lib.profile_enable(False)
            _lib.profile_mask(None)
            us = prof[1] * 1e3 / iters
            byts = G * H * n * n * 4 + G * n * 4
            ach = byts / (us * 1e-6) / 1e9
            print(json.dumps({"mode": "colmean_sweep", "tiles": G, "heads": H, "patches": n,
                              "us_per_call": us, "wall_us_per_call": (t1 - t0) * 1e6 / iters,
                              "algorithmic_bytes": byts, "achieved_GBs": ach,
                              "frac_of_hbm_peak": ach / HBM_PEAK_GBS}), flush=True)
            del A, out
            torch.cuda.empty_cache()


HEADLINE = {"workload": "stress", "keep": 288, "skip_p": 0.25}


def run_step(w, args, dev, weights=None, online=False, projector_on=False, decode=0,
             cpu=True, copy_probe_mib=0):
    """Times `args.steps` whole steps of workload `w` and returns its result record
    (without the contract's top-level fields).  `weights` reuses device weights
    already generated for the same decoder and seed."""
    from paper_2609_34977_amd import _lib
    from paper_2609_34977_amd.pipeline import Pipeline
    from paper_2609_34977_amd.profiling import recorded_traffic

    t_setup = time.perf_counter()
    attn, feats, src, text, W, pol = build_inputs(w, dev, weights)
    if online:
        pol = online_policy(w, dev, args.vocab)
    sc, dec = w.score, w.dec
    cfg = _lib.decoder_cfg(dec.L, dec.d, dec.H, dec.d_ff,
                           _lib.BF16 if dec.dtype == "bf16" else _lib.F32, dec.eps, dec.theta)
    projector = None
    if projector_on:
        from synth.decoder_inputs import projector_inputs, projector_weights
        projector = projector_weights(w, dev)
        src = projector_inputs(w, dev)
    pipe = Pipeline(G=sc.G, n=sc.n, K=sc.K, keep=sc.keep, r_num=sc.r_num, r_den=sc.r_den,
                    kmeans_iter=sc.kmeans_iter, tiles_per_sample=w.tiles_per_sample,
                    n_text=w.n_text, quota_mode=w.quota_mode, dec=cfg, weights=W, device=dev,
                    projector=projector)
    torch.cuda.synchronize()
    print(f"# {w.name}: setup {time.perf_counter() - t_setup:.1f} s", file=sys.stderr, flush=True)

    out = None
    for i in range(args.warmup):
        out = pipe.step(attn, feats, src, text, pol)
    torch.cuda.synchronize()
    print(f"# {w.name}: warmup done", file=sys.stderr, flush=True)
    if copy_probe_mib > 0:
        a = torch.empty(copy_probe_mib << 20, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # per-class breakdown (events around every launch) from a separate pass
    n_full = max(2, min(args.steps, 5))
    _lib.profile_mask(None)
    _lib.profile_enable(True)
    for i in range(n_full):
        out = pipe.step(attn, feats, src, text, pol)
    torch.cuda.synchronize()
    full = _lib.profile_read()
    _lib.profile_enable(False)
    dom = max((k for k, v in full.items() if v[0]), key=lambda k: full[k][1])

    # timed region: events only around the dominant kernel class
    _lib.profile_mask([dom])
    _lib.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        out = pipe.step(attn, feats, src, text, pol)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = _lib.profile_read()
    _lib.profile_enable(False)
    _lib.profile_mask(None)
    print(f"# {w.name}: timed steps done", file=sys.stderr, flush=True)

    ms = (t1 - t0) * 1e3 / args.steps
    cu, codes = out["cu"], out["codes"]
    rows = int(cu[-1])
    B = w.B
    admit = out.get("admit")
    alg = algorithmic(w, cu, codes, admit, args.vocab)
    kernel_ms = {k: v[1] / n_full for k, v in full.items() if v[0]}
    launches = {k: v[0] // n_full for k, v in full.items() if v[0]}
    per_step_ms = prof[dom][1] / args.steps
    bf16 = dec.dtype == "bf16"
    if dom in alg:
        byts, flops = alg[dom]
        intensity = flops / max(byts, 1.0)
        ridge = (BF16_PEAK_TFLOPS if bf16 else FP32_PEAK_TFLOPS) * 1e12 / (HBM_PEAK_GBS * 1e9)
        if dom != "attention" and intensity < ridge:
            ach = byts / (per_step_ms * 1e-3) / 1e9
            roof = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": ach / HBM_PEAK_GBS}
        else:
            pk = BF16_PEAK_TFLOPS if bf16 else FP32_PEAK_TFLOPS
            ach = flops / (per_step_ms * 1e-3) / 1e12
            roof = {"bound": "mfma", "achieved": ach, "peak": pk, "unit": "TFLOP/s", "frac": ach / pk}
    else:
        roof = {"bound": "hbm", "achieved": None, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": None}
    workload = (f"{w.name}_keep{sc.keep}" + (f"_skip{w.skip['p']:g}" if w.skip.get("kind") == "random_layer"
                                               and w.name == "stress" else "")
                + ("_online" if online else "") + ("_projector" if projector_on else ""))
    roof.update({"kernel": dom, "launches_per_step": prof[dom][0] // args.steps,
                 "avg_launch_us": prof[dom][1] * 1e3 / max(prof[dom][0], 1),
                 "traffic": recorded_traffic(os.path.join(ROOT, "profiles", f"{dom}_traffic_{workload}.json"),
                                             dom, workload, rows)})
    prefill_flops = sum(v[1] for v in alg.values())
    res = {
        "value": rows / (ms * 1e-3),
        "unit": "tokens/s",
        "ms_per_step": ms,
        "dtype": dec.dtype,
        "config": {"workload": workload,
                   "batch": B, "tiles": sc.G,
                   "visual_tokens_per_tile": sc.n, "keep_per_tile": sc.keep,
                   "text_tokens": w.n_text, "decoder_rows": rows, "decoder_layers": dec.L,
                   "d_model": dec.d, "heads": dec.H, "d_ff": dec.d_ff,
                   "skip": "online" if online else w.skip.get("kind"),
                   "skip_p": None if online else w.skip.get("p"),
                   "skipped_sublayer_slots": float((codes[:, :rows] != 0).mean()),
                   "parallelism": "single GPU"},
        "ms_per_sample": ms / B,
        "effective_tokens_per_s": B * (sc.n * w.tiles_per_sample + w.n_text) / (ms * 1e-3),
        "prefill_tflop_per_step": prefill_flops / 1e12,
        "online": None if admit is None else {
            "vocab": args.vocab, "w1": pol.w1, "w2": pol.w2, "T_skip": pol.T_skip,
            "admitted_visual_rows": int(np.sum(admit >= 0)),
            "visual_rows": int(sum(cu[b + 1] - cu[b] - w.n_text for b in range(B)))},
        "roofline": roof,
        "kernel_ms_per_step": {k: round(v, 4) for k, v in kernel_ms.items()},
        "launches_per_step": launches,
    }
    if decode > 0:
        res["decode"] = decode_latency(w, pipe, out, dev, args)
    if cpu:
        print(f"# {w.name}: cpu baseline", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w, min(args.cpu_layers, dec.L), W)
    return res, W


GEMM_SHAPES = ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down")


def vendor_gemm(args, dev):
    """Context for the decoder GEMMs.  For each workload the prefill runs without
    skipping (every sub-layer over every row, so each launch has M = the decoder
    rows) and its per-launch time per GEMM class is read from the profiled pre-pass;
    beside it torch.nn.functional.linear (hipBLASLt) runs the same products in bf16:
    QKV [M, 3d], O [M, d], gate and up stacked [M, 2 d_ff] (plain products: no SwiGLU,
    bf16 outputs), down [M, d] over K = d_ff.  Both read cold weights: the prefill
    streams 32+ layers of distinct weights, the library call cycles through copies
    totalling more than the 256 MB last-level cache.  Up to 256 rows the library's
    classes end with fp32 split-K partials whose sum happens in the next kernel (the
    norm, or the QKV finalize), which is not counted here."""
    import torch.nn.functional as F
    from synth import get_workload
    for name, keep in (("stress", 576), ("stress", 288), ("llava15_13b", None), ("llava_next_7b", 128),
                       ("llava15_7b", 128)):
        w = get_workload(name, keep=keep, L=args.layers, skip_p=0.0)
        res, _ = run_step(w, args, dev, cpu=False)
        M = res["config"]["decoder_rows"]
        d, dff = w.dec.d, w.dec.d_ff
        shapes = {"gemm_qkv": (3 * d, d), "gemm_o": (d, d), "gemm_gateup": (2 * dff, d), "gemm_down": (d, dff)}
        km, ln = res["kernel_ms_per_step"], res["launches_per_step"]
        ours = {c: 1e3 * km[c] / ln[c] for c in GEMM_SHAPES if ln.get(c)}
        vend = {}
        for c in GEMM_SHAPES:
            N, K = shapes[c]
            a = torch.randn(M, K, device=dev, dtype=torch.bfloat16)
            copies = max(2, -(-(1 << 30) // (N * K * 2)))
            ws = [torch.randn(N, K, device=dev, dtype=torch.bfloat16) for _ in range(copies)]
            for i in range(copies):
                F.linear(a, ws[i])
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            n = 4 * copies
            e0.record()
            for i in range(n):
                F.linear(a, ws[i % copies])
            e1.record()
            torch.cuda.synchronize()
            vend[c] = 1e3 * e0.elapsed_time(e1) / n
            del a, ws
            torch.cuda.empty_cache()
        tf = {c: 2.0 * M * shapes[c][0] * shapes[c][1] / 1e6 for c in GEMM_SHAPES}  # flop / us -> TFLOP/s
        print(json.dumps({"mode": "vendor_gemm", "workload": res["config"]["workload"], "rows": M, "d": d,
                          "d_ff": dff, "ours_us": ours, "hipblaslt_us": vend,
                          "ours_tflops": {c: tf[c] / ours[c] for c in ours},
                          "hipblaslt_tflops": {c: tf[c] / vend[c] for c in vend}}), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(see the sharding notes in DESIGN.md); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    from synth import get_workload

    headline = args.workload is None
    name = HEADLINE["workload"] if headline else args.workload
    keep = args.keep if args.keep is not None or not headline else HEADLINE["keep"]
    skip_p = args.skip_p if args.skip_p is not None or not headline else HEADLINE["skip_p"]
    w = get_workload(name, keep=keep, L=args.layers, skip_p=skip_p)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.score_sweep:
        score_sweep(w, dev, args)
        return
    if args.colmean_sweep:
        colmean_sweep(dev)
        return
    if args.select_sweep:
        select_sweep(w, dev, args)
        return
    if args.curve:
        curve(args, dev)
        return
    if args.vendor_gemm:
        vendor_gemm(args, dev)
        return
    cpu = not args.no_cpu_baseline and not args.online and not args.projector
    res, W = run_step(w, args, dev, online=args.online, projector_on=args.projector, decode=args.decode,
                      cpu=cpu, copy_probe_mib=args.copy_probe_mib)
    line = {"metric": METRIC, "value": res.pop("value"), "unit": res.pop("unit"), "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": res.pop("ms_per_step"),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": res.pop("dtype"),
            "data": "synthetic", "config": res.pop("config")}
    line.update(res)
    if headline and not args.no_secondary and not args.online and not args.projector:
        w2 = get_workload("llava15_7b", L=args.layers)
        same = w2.dec == w.dec and w2.seed == w.seed
        r2, _ = run_step(w2, args, dev, weights=W if same else None, cpu=False)
        line[r2["config"]["workload"]] = {k: r2[k] for k in ("value", "unit", "ms_per_step", "ms_per_sample",
                                                             "effective_tokens_per_s", "roofline",
                                                             "kernel_ms_per_step", "config")}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
