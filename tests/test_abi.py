"""C ABI checks that need no GPU: symbols, host-only entry points, argument validation.

Every validation case below passes arguments that are rejected before the
library makes any HIP call, so on a machine without a GPU the documented
status comes back (a HIP call would instead give SPIDER_ERR_HIP).
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import asl_skip as ak
from oracle import msv_prune as mp
from synth import get_workload
from synth.skip_inputs import adaptive_scores, policy_lists, slc_tables

lib_mod = pytest.importorskip("paper_2609_34977_amd._lib")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

OK, INVALID, SHAPE, UNSUPPORTED, WORKSPACE, HIP = 0, 1, 2, 3, 4, 5


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lib_mod._LIB_PATH):
        pytest.skip("libspider.so not built")
    return lib_mod.lib()


def test_every_header_symbol_is_exported(L):
    hdr = open(os.path.join(ROOT, "include", "spider.h")).read()
    names = set(re.findall(r"\b(spider_[a-z_]+)\s*\(", hdr))
    assert len(names) >= 14
    for n in names:
        assert hasattr(L, n), n
    assert names == set(lib_mod.exported_symbols())
    assert L.spider_version() >= 100


@pytest.mark.parametrize("keep", [0, 1, 16, 64, 128, 192, 576, 1440, 2880])
def test_budget_matches_oracle(L, keep):
    assert lib_mod.budget(keep) == mp.budget(keep)
    assert lib_mod.budget(keep, 1, 2) == mp.budget(keep, 1, 2)


def test_budget_rejects_bad_ratio(L):
    a, c = ctypes.c_int(), ctypes.c_int()
    assert L.spider_budget(10, 11, 10, ctypes.byref(a), ctypes.byref(c)) == INVALID
    assert b"r_num" in L.spider_last_error()
    assert L.spider_budget(-1, 7, 10, ctypes.byref(a), ctypes.byref(c)) == INVALID


@pytest.mark.parametrize("name", ["llava15_7b", "llava_next_7b", "synthetic_40"])
def test_slc_policy_bit_exact_with_oracle(L, name):
    n_layers = 40 if name == "synthetic_40" else 32
    sa, sf = slc_tables(policy_lists(name, n_layers), n_layers)
    sel, tgt = lib_mod.slc_policy(sa, sf, 1e-8)
    na, nf = ak.slc_normalize(sa, sf, 1e-8)
    m, osel = ak.skip_targets(na, nf)
    assert np.array_equal(tgt, m)
    assert np.array_equal(sel, osel)          # same doubles, bit for bit


@pytest.mark.parametrize("wl", ["llava_next_7b", "llava15_13b"])
def test_plan_skips_bit_exact_with_oracle(L, wl):
    w = get_workload(wl)
    n_layers = w.dec.L
    sa, sf = slc_tables(policy_lists(w.skip["policy"], n_layers), n_layers)
    na, nf = ak.slc_normalize(sa, sf)
    m, sel = ak.skip_targets(na, nf)
    S = adaptive_scores(w, 300)
    for b in range(w.B):
        codes, admit = lib_mod.plan_skips(S[b], sel, m, w.skip["w1"], w.skip["w2"],
                                          w.skip["T_skip"], n_layers)
        oc, oadmit, _ = ak.plan(S[b], sel, m, w.skip["w1"], w.skip["w2"], w.skip["T_skip"], n_layers)
        assert np.array_equal(codes, oc)
        assert np.array_equal(admit, oadmit)
    frac = (oadmit >= 0).mean()
    assert 0.2 < frac < 0.7


def test_plan_skips_threshold_ties_and_window(L):
    S = np.array([[1.0, 0.2, 0.0], [0.0, 0.9, 0.3]], np.float32)
    codes, admit = lib_mod.plan_skips(S, np.array([0.5, 0.5, 1.0, 1.0]), np.array([0, 1, 0, 0], np.uint8),
                                      1.0, 1.0, 1.5, 4)
    assert codes.tolist() == [[1, 0, 0], [1, 2, 0], [1, 2, 0], [1, 2, 0]]
    assert admit.tolist() == [0, 1, -1]


def test_plan_skips_validation(L):
    sel = np.zeros(4)
    tgt = np.array([0, 1, 2, 0], np.uint8)
    S = np.zeros((2, 3), np.float32)
    codes = np.zeros((4, 3), np.uint8)
    st = L.spider_plan_skips(4, 3, S.ctypes.data, 3, sel.ctypes.data, tgt.ctypes.data, 1.0, 1.0,
                             1.0, codes.ctypes.data, 3, None)
    assert st == INVALID and b"target" in L.spider_last_error()
    st = L.spider_plan_skips(4, 3, S.ctypes.data, 2, sel.ctypes.data, sel.ctypes.data, 1.0, 1.0,
                             1.0, codes.ctypes.data, 3, None)
    assert st == SHAPE


def _score_call(L, **kw):
    args = dict(G=1, n=576, H=16, d_v=1024, n_layers=2, attn=0x1000, asg=16 * 577, ash=577,
                col0=1, dt=1, fsg=577 * 1024, fsr=1024, row0=1, n_anchor=89, K=4, it=10,
                a=0x1000, cl=0x1000, s=0x1000, m=None, ws=0x100000, wsb=1 << 30)
    args.update(kw)
    fp = (ctypes.c_void_p * 8)(*([0x2000] * 8))
    if kw.get("null_feat"):
        fp[1] = None
    return L.spider_score(args["G"], args["n"], args["H"], args["d_v"], args["n_layers"],
                          args["attn"], args["asg"], args["ash"], args["col0"], fp, args["dt"],
                          args["fsg"], args["fsr"], args["row0"], args["n_anchor"], args["K"],
                          args["it"], args["a"], args["cl"], args["s"], args["m"], args["ws"],
                          args["wsb"], None)


def test_score_validation_before_any_hip_call(L):
    assert _score_call(L, G=0) == INVALID
    assert _score_call(L, n=5000, asg=16 * 5001, ash=5001, fsg=5001 * 1024) == UNSUPPORTED
    assert _score_call(L, K=9) == UNSUPPORTED
    assert _score_call(L, n_anchor=577) == SHAPE
    assert _score_call(L, it=0) == INVALID
    assert _score_call(L, a=None) == INVALID
    assert _score_call(L, null_feat=True) == INVALID
    assert _score_call(L, ash=100) == SHAPE
    assert _score_call(L, fsr=1000, fsg=577 * 1000) == SHAPE
    assert _score_call(L, d_v=1020, fsr=1024) == UNSUPPORTED
    assert _score_call(L, wsb=16) == WORKSPACE
    assert b"workspace" in L.spider_last_error()
    assert _score_call(L, ws=0x100010) == WORKSPACE  # misaligned
    assert L.spider_score_workspace_size(1, 576, 1024, 2, 4) > 0
    assert L.spider_score_workspace_size(0, 576, 1024, 2, 4) == 0


def test_score_noalloc_rejects_sizes_beyond_its_scratch_before_any_hip_call(L):
    def call(G, n=576, d_v=1024, K=4):
        feats = (ctypes.c_void_p * 2)(0x1000, 0x1000)
        return L.spider_score_noalloc(G, n, 16, d_v, 2, 0x1000, 16 * (n + 1), n + 1, 1, feats, 1,
                                      (n + 1) * d_v, d_v, 1, 89, K, 10, 0x1000, 0x1000, 0x1000, None, None)
    limit = 32 << 20
    per_tile = L.spider_score_workspace_size(1, 576, 1024, 2, 4)
    too_many = limit // per_tile + 8
    assert L.spider_score_workspace_size(too_many, 576, 1024, 2, 4) > limit
    assert call(too_many) == WORKSPACE
    assert b"static scratch" in L.spider_last_error()
    assert call(0) == INVALID


def _select_call(L, **kw):
    a = dict(G=1, n=576, cl=0x1000, s=0x1000, na=89, nc=39, K=4, qm=0, idx=0x1000, cnt=0x1000,
             cap=132, tps=1, src=None, ssg=0, dm=0, dt=1, text=None, nt=0, x=None, cu=None)
    a.update(kw)
    return L.spider_select(a["G"], a["n"], a["cl"], a["s"], a["na"], a["nc"], a["K"], a["qm"],
                           a["idx"], a["cnt"], a["cap"], a["tps"], a["src"], a["ssg"], a["dm"],
                           a["dt"], a["text"], a["nt"], a["x"], a["cu"], None)


def test_select_validation_before_any_hip_call(L):
    assert _select_call(L, G=0) == INVALID
    assert _select_call(L, cap=131) == SHAPE
    assert _select_call(L, qm=2) == INVALID
    assert _select_call(L, K=0) == UNSUPPORTED
    assert _select_call(L, na=600) == SHAPE
    assert _select_call(L, G=5, tps=2) == SHAPE
    assert _select_call(L, cl=None) == INVALID
    # assembly arguments
    assert _select_call(L, src=0x2000, ssg=576 * 4096, dm=4096, x=None, cu=0x1000) == INVALID
    assert _select_call(L, src=0x2000, ssg=100, dm=4096, x=0x3000, cu=0x1000) == SHAPE
    assert _select_call(L, src=0x2000, ssg=576 * 4100, dm=4100, x=0x3000, cu=0x1000) == UNSUPPORTED
    assert _select_call(L, src=0x2000, ssg=576 * 4096, dm=4096, x=0x3000, cu=0x1000, nt=5) == INVALID


def _prefill_call(L, cfg, cu, codes, ws_bytes=1 << 40, ws=0x100000, x=0x1000, null_w=False):
    W = (lib_mod.LayerWeights * cfg.L)()
    for i in range(cfg.L):
        W[i] = lib_mod.LayerWeights(*([0x1000] * 9))
    if null_w:
        W[cfg.L - 1].wd = None
    cu = np.ascontiguousarray(cu, np.int32)
    codes = np.ascontiguousarray(codes, np.uint8)
    return L.spider_prefill(ctypes.byref(cfg), W, len(cu) - 1, cu.ctypes.data, x, codes.ctypes.data,
                            0x1000, ws, ws_bytes, None)


def test_prefill_validation_before_any_hip_call(L):
    bf = lib_mod.decoder_cfg(2, 4096, 32, 11008, lib_mod.BF16)
    codes = np.zeros((2, 10), np.uint8)
    assert _prefill_call(L, lib_mod.decoder_cfg(2, 4096, 64, 11008, lib_mod.BF16), [0, 10], codes) == UNSUPPORTED
    assert _prefill_call(L, lib_mod.decoder_cfg(2, 4096, 30, 11008, lib_mod.BF16), [0, 10], codes) == SHAPE
    assert _prefill_call(L, lib_mod.decoder_cfg(0, 4096, 32, 11008, lib_mod.BF16), [0, 10], codes) == INVALID
    assert _prefill_call(L, lib_mod.decoder_cfg(2, 4096, 32, 11000, lib_mod.BF16), [0, 10], codes) == UNSUPPORTED
    assert _prefill_call(L, lib_mod.decoder_cfg(2, 96, 32, 100, lib_mod.F32), [0, 10], codes) == SHAPE
    assert _prefill_call(L, bf, [1, 10], codes) == SHAPE
    assert _prefill_call(L, bf, [0, 6, 5], np.zeros((2, 5), np.uint8)) == SHAPE
    bad = codes.copy()
    bad[1, 3] = 4
    assert _prefill_call(L, bf, [0, 10], bad) == INVALID
    assert _prefill_call(L, bf, [0, 10], codes, null_w=True) == INVALID
    assert _prefill_call(L, bf, [0, 10], codes, ws_bytes=100) == WORKSPACE
    assert _prefill_call(L, bf, [0, 10], codes, x=0x1001) == UNSUPPORTED
    # an empty batch is a no-op
    assert _prefill_call(L, bf, [0, 0], np.zeros((2, 0), np.uint8)) == OK
    assert lib_mod.prefill_workspace_size(bf, 1, 192) > 0


def _online_call(L, cfg, cu, n_text=4, V=32000, wu=0x1000, sel=None, tgt=None, w1=1.0, T=1.0,
                 ws_bytes=1 << 40):
    W = (lib_mod.LayerWeights * cfg.L)()
    for i in range(cfg.L):
        W[i] = lib_mod.LayerWeights(*([0x1000] * 9))
    cu = np.ascontiguousarray(cu, np.int32)
    rows = int(cu[-1])
    sel = np.zeros(cfg.L, np.float64) if sel is None else np.ascontiguousarray(sel, np.float64)
    tgt = np.zeros(cfg.L, np.uint8) if tgt is None else np.ascontiguousarray(tgt, np.uint8)
    codes = np.zeros((cfg.L, max(rows, 1)), np.uint8)
    return L.spider_prefill_online(ctypes.byref(cfg), W, len(cu) - 1, cu.ctypes.data, 0x1000, n_text,
                                   wu, V, sel.ctypes.data, tgt.ctypes.data, w1, 0.5, T,
                                   codes.ctypes.data, None, None, 0x1000, 0x100000, ws_bytes, None)


def test_prefill_online_validation_before_any_hip_call(L):
    bf = lib_mod.decoder_cfg(4, 4096, 32, 11008, lib_mod.BF16)
    f32 = lib_mod.decoder_cfg(4, 128, 4, 344, lib_mod.F32)
    assert _online_call(L, bf, [0, 10], n_text=0) == INVALID
    assert _online_call(L, bf, [0, 10, 13], n_text=4) == SHAPE       # sample 1 shorter than n_text
    assert _online_call(L, bf, [0, 10], V=32001) == UNSUPPORTED      # bf16 GEMM needs V % 64 == 0
    assert _online_call(L, bf, [0, 10], V=1) == INVALID
    assert _online_call(L, bf, [0, 10], wu=None) == INVALID
    assert _online_call(L, bf, [0, 10], wu=0x1008) == UNSUPPORTED
    assert _online_call(L, bf, [0, 10], tgt=[0, 2, 0, 0]) == INVALID
    assert _online_call(L, bf, [0, 10], sel=[0.0, np.nan, 0, 0]) == INVALID
    assert _online_call(L, bf, [0, 10], T=np.inf) == INVALID
    assert _online_call(L, bf, [0, 10], ws_bytes=100) == WORKSPACE
    assert _online_call(L, bf, [0, 10, 10], n_text=4) == SHAPE       # empty sample
    # any V for fp32; entries past the window are not read
    assert _online_call(L, f32, [0, 10], V=1001, tgt=[0, 1, 7, 7], ws_bytes=100) == WORKSPACE
    assert lib_mod.prefill_online_workspace_size(bf, 1, 192, 32000) > lib_mod.prefill_workspace_size(bf, 1, 192)


def test_prefill_online_ablation_validation_before_any_hip_call(L):
    """The ablation entry point: unknown bits are rejected first, the other
    checks are those of spider_prefill_online."""
    bf = lib_mod.decoder_cfg(4, 4096, 32, 11008, lib_mod.BF16)
    W = (lib_mod.LayerWeights * bf.L)()
    for i in range(bf.L):
        W[i] = lib_mod.LayerWeights(*([0x1000] * 9))
    cu = np.array([0, 10], np.int32)
    sel = np.zeros(bf.L, np.float64)
    tgt = np.zeros(bf.L, np.uint8)
    codes = np.zeros((bf.L, 10), np.uint8)

    def call(bits, n_text=4, ws_bytes=1 << 40):
        return L.spider_prefill_online_ablation(ctypes.byref(bf), W, 1, cu.ctypes.data, 0x1000, n_text, 0x1000,
                                                32000, sel.ctypes.data, tgt.ctypes.data, 1.0, 0.5, 1.0, bits,
                                                codes.ctypes.data, None, None, 0x1000, 0x100000, ws_bytes, None)
    assert call(16) == INVALID and b"ablation" in L.spider_last_error()
    assert call(0x80000000) == INVALID
    assert call(1 | 8, n_text=0) == INVALID
    for bits in (0, 1, 2, 4, 8, 15):
        assert call(bits, ws_bytes=100) == WORKSPACE


@pytest.mark.parametrize("n,num,den", [(576, 1, 2), (1000, 2, 5), (7, 1, 2), (1369, 1, 2), (50, 1, 1), (50, 0, 3)])
def test_budget_ratio_matches_oracle(L, n, num, den):
    assert lib_mod.budget_ratio(n, num, den) == mp.budget_ratio(n, num, den)
    assert lib_mod.budget_ratio(n, num, den, 1, 2) == mp.budget_ratio(n, num, den, 1, 2)


def test_budget_ratio_rejects_bad_arguments(L):
    k, a, c = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    for args in [(-1, 1, 2), (10, 3, 2), (10, 1, 0), (10, -1, 2)]:
        assert L.spider_budget_ratio(*args, 7, 10, ctypes.byref(k), ctypes.byref(a), ctypes.byref(c)) == INVALID
    assert L.spider_budget_ratio(10, 1, 2, 11, 10, ctypes.byref(k), ctypes.byref(a), ctypes.byref(c)) == INVALID


def _colmean_call(L, G=2, H=16, n=576, attn=0x1000, sg=None, sh=None, sr=None, ws=0x100000, wsb=1 << 40):
    sr = n if sr is None else sr
    sh = n * sr if sh is None else sh
    sg = H * sh if sg is None else sg
    return L.spider_anchor_colmean(G, H, n, attn, sg, sh, sr, 0x2000, ws, wsb, None)


def test_anchor_colmean_validation_before_any_hip_call(L):
    assert _colmean_call(L, G=0) == INVALID
    assert _colmean_call(L, n=4100) == UNSUPPORTED
    assert _colmean_call(L, H=2000) == UNSUPPORTED
    assert _colmean_call(L, attn=None) == INVALID
    assert _colmean_call(L, sr=500) == SHAPE
    assert _colmean_call(L, n=574) == UNSUPPORTED          # n % 4
    assert _colmean_call(L, attn=0x1004) == UNSUPPORTED    # 16-byte alignment
    assert _colmean_call(L, wsb=100) == WORKSPACE
    assert _colmean_call(L, ws=0x100010) == WORKSPACE
    assert lib_mod.anchor_colmean.__doc__
    assert L.spider_anchor_colmean_workspace_size(1, 16, 576) == 16 * 5 * 576 * 4


def test_score_with_given_anchor_scores_validation(L):
    feats = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    # H must be 0 when cls_attn is NULL, >= 1 otherwise
    assert L.spider_score(1, 576, 16, 1024, 2, None, 0, 0, 0, feats, lib_mod.BF16, 577 * 1024, 1024, 1,
                          89, 4, 10, 0x3000, 0x4000, 0x5000, None, 0x100000, 1 << 40, None) == INVALID
    assert L.spider_score(1, 576, 0, 1024, 2, 0x1000, 577, 577, 1, feats, lib_mod.BF16, 577 * 1024, 1024, 1,
                          89, 4, 10, 0x3000, 0x4000, 0x5000, None, 0x100000, 1 << 40, None) == INVALID
    assert L.spider_score(1, 576, 0, 1024, 2, None, 0, 0, 0, feats, lib_mod.BF16, 577 * 1024, 1024, 1,
                          89, 4, 10, 0x3000, 0x4000, 0x5000, None, 0x100000, 100, None) == WORKSPACE


def test_cls_attention_validation_before_any_hip_call(L):
    def call(G=1, H=16, dh=64, T=577, q=0x1000, sqg=None, k=0x2000, skg=None, skr=None, dt=lib_mod.BF16, sc=0.125):
        sqg = H * dh if sqg is None else sqg
        skr = H * dh if skr is None else skr
        skg = T * skr if skg is None else skg
        return L.spider_cls_attention(G, H, dh, T, q, sqg, k, skg, skr, dt, sc, 0x3000, None)
    assert call(G=0) == INVALID
    assert call(q=None) == INVALID
    assert call(dt=7) == INVALID
    assert call(sc=float("nan")) == INVALID
    assert call(dh=512) == UNSUPPORTED
    assert call(T=5000) == UNSUPPORTED
    assert call(skr=100) == SHAPE
    assert call(dh=62) == UNSUPPORTED
    assert call(q=0x1004) == UNSUPPORTED      # bf16 needs 8-byte alignment
    assert call(q=0x1008, dt=lib_mod.F32) == UNSUPPORTED


def test_prefill_kv_and_decode_validation_before_any_hip_call(L):
    bf = lib_mod.decoder_cfg(2, 4096, 32, 11008, lib_mod.BF16)
    W = (lib_mod.LayerWeights * 2)()
    for i in range(2):
        W[i] = lib_mod.LayerWeights(*([0x1000] * 9))
    cu = np.array([0, 10], np.int32)
    codes = np.zeros((2, 10), np.uint8)
    kv = lib_mod.KVCache(0x10000, 0x20000, 16)
    call = lambda kvp, ws=1 << 40: L.spider_prefill_kv(ctypes.byref(bf), W, 1, cu.ctypes.data, 0x1000,
                                                       codes.ctypes.data, 0x1000, kvp, 0x100000, ws, None)
    assert call(None) == INVALID
    assert call(ctypes.byref(lib_mod.KVCache(0x10000, 0x20000, 8))) == SHAPE      # sample longer than cap
    assert call(ctypes.byref(lib_mod.KVCache(0x10008, 0x20000, 16))) == UNSUPPORTED
    assert call(ctypes.byref(kv), ws=100) == WORKSPACE
    dcall = lambda ln, wu=0x3000, V=32000, fn=0x4000, ws=1 << 40: L.spider_decode_step(
        ctypes.byref(bf), W, len(ln), ln.ctypes.data, 0x1000, ctypes.byref(kv), fn, wu, V, 0x5000, None, None,
        0x100000, ws, None)
    assert dcall(np.array([5, 16], np.int32)) == SHAPE        # position past the cache
    assert dcall(np.array([-1], np.int32)) == SHAPE
    assert dcall(np.array([3], np.int32), V=32001) == UNSUPPORTED
    assert dcall(np.array([3], np.int32), fn=None) == INVALID
    assert dcall(np.array([3], np.int32), ws=100) == WORKSPACE
    # the decode attention reads cached rows as 16-byte vectors
    kv_odd = lib_mod.KVCache(0x10008, 0x20000, 16)
    f32 = lib_mod.decoder_cfg(2, 4096, 32, 11008, lib_mod.F32)
    assert L.spider_decode_step(ctypes.byref(f32), W, 1, np.array([3], np.int32).ctypes.data, 0x1000,
                                ctypes.byref(kv_odd), None, None, 0, 0x5000, None, None, 0x100000, 1 << 40,
                                None) == UNSUPPORTED
    f32_dh30 = lib_mod.decoder_cfg(2, 120, 4, 344, lib_mod.F32)     # dh = 30: not a multiple of 4 floats
    assert L.spider_decode_step(ctypes.byref(f32_dh30), W, 1, np.array([3], np.int32).ctypes.data, 0x1000,
                                ctypes.byref(kv), None, None, 0, 0x5000, None, None, 0x100000, 1 << 40,
                                None) == UNSUPPORTED
    assert L.spider_decode_workspace_size(ctypes.byref(bf), 2, 16, 32000) > \
        L.spider_decode_workspace_size(ctypes.byref(bf), 2, 16, 0) > 0


def test_profiler_host_side(L):
    lib_mod.profile_enable(True)
    d = lib_mod.profile_read()
    assert "gemm_gateup" in d and all(v == (0, 0.0) for v in d.values())
    lib_mod.profile_enable(False)
    assert L.spider_profile_read(99, ctypes.byref(ctypes.c_int64()), ctypes.byref(ctypes.c_double())) == INVALID
