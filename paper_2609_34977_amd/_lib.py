"""ctypes binding of libspider (the C ABI declared in include/spider.h).

Argument marshalling only: tensors are passed as device pointers, outputs and
workspaces are allocated with torch on the tensors' device, and every call is
enqueued on torch's current stream.  No computation happens here; if the
library is missing the import of any function raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspider.so")
_lib = None

F32, BF16 = 0, 1


class SpiderError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"spider status {status}: {msg}")
        self.status = status


class DecoderCfg(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int), ("d", ctypes.c_int), ("H", ctypes.c_int),
                ("d_ff", ctypes.c_int), ("eps", ctypes.c_float), ("theta", ctypes.c_float),
                ("dtype", ctypes.c_int)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")]


class KVCache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("cap", ctypes.c_int)]


_VP, _I, _I64, _SZ, _F, _D = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t,
                              ctypes.c_float, ctypes.c_double)

_SIGS = {
    "spider_last_error": ([], ctypes.c_char_p),
    "spider_version": ([], _I),
    "spider_budget": ([_I, _I, _I, ctypes.POINTER(_I), ctypes.POINTER(_I)], _I),
    "spider_budget_ratio": ([_I, _I, _I, _I, _I, ctypes.POINTER(_I), ctypes.POINTER(_I), ctypes.POINTER(_I)], _I),
    "spider_anchor_colmean_workspace_size": ([_I, _I, _I], _SZ),
    "spider_anchor_colmean": ([_I, _I, _I, _VP, _I64, _I64, _I64, _VP, _VP, _SZ, _VP], _I),
    "spider_cls_attention": ([_I, _I, _I, _I, _VP, _I64, _VP, _I64, _I64, _I, _F, _VP, _VP], _I),
    "spider_project_kept_workspace_size": ([_I, _I, _I, _I, _I], _SZ),
    "spider_project_kept": ([_I, _I, _I, _VP, _VP, _VP, _I64, _I64, _I, _I, _VP, _VP, _I, _VP, _VP, _I, _I, _I,
                             _VP, _VP, _SZ, _VP], _I),
    "spider_score_workspace_size": ([_I, _I, _I, _I, _I], _SZ),
    "spider_score": ([_I, _I, _I, _I, _I, _VP, _I64, _I64, _I, ctypes.POINTER(_VP), _I, _I64, _I64,
                      _I, _I, _I, _I, _VP, _VP, _VP, _VP, _VP, _SZ, _VP], _I),
    "spider_score_noalloc": ([_I, _I, _I, _I, _I, _VP, _I64, _I64, _I, ctypes.POINTER(_VP), _I, _I64, _I64,
                              _I, _I, _I, _I, _VP, _VP, _VP, _VP, _VP], _I),
    "spider_select": ([_I, _I, _VP, _VP, _I, _I, _I, _I, _VP, _VP, _I, _I, _VP, _I64, _I, _I, _VP,
                       _I, _VP, _VP, _VP], _I),
    "spider_slc_policy": ([_I, _VP, _VP, _D, _VP, _VP], _I),
    "spider_plan_skips": ([_I, _I, _VP, _I, _VP, _VP, _D, _D, _D, _VP, _I, _VP], _I),
    "spider_prefill_workspace_size": ([ctypes.POINTER(DecoderCfg), _I, _I], _SZ),
    "spider_prefill": ([ctypes.POINTER(DecoderCfg), ctypes.POINTER(LayerWeights), _I, _VP, _VP,
                        _VP, _VP, _VP, _SZ, _VP], _I),
    "spider_prefill_online_workspace_size": ([ctypes.POINTER(DecoderCfg), _I, _I, _I], _SZ),
    "spider_prefill_online": ([ctypes.POINTER(DecoderCfg), ctypes.POINTER(LayerWeights), _I, _VP, _VP,
                               _I, _VP, _I, _VP, _VP, _D, _D, _D, _VP, _VP, _VP, _VP, _VP, _SZ, _VP],
                              _I),
    "spider_prefill_online_ablation": ([ctypes.POINTER(DecoderCfg), ctypes.POINTER(LayerWeights), _I, _VP,
                                        _VP, _I, _VP, _I, _VP, _VP, _D, _D, _D, ctypes.c_uint32, _VP, _VP,
                                        _VP, _VP, _VP, _SZ, _VP], _I),
    "spider_prefill_kv": ([ctypes.POINTER(DecoderCfg), ctypes.POINTER(LayerWeights), _I, _VP, _VP, _VP, _VP,
                           ctypes.POINTER(KVCache), _VP, _SZ, _VP], _I),
    "spider_decode_workspace_size": ([ctypes.POINTER(DecoderCfg), _I, _I, _I], _SZ),
    "spider_decode_step": ([ctypes.POINTER(DecoderCfg), ctypes.POINTER(LayerWeights), _I, _VP, _VP,
                            ctypes.POINTER(KVCache), _VP, _VP, _I, _VP, _VP, _VP, _VP, _SZ, _VP], _I),
    "spider_profile_enable": ([_I], _I),
    "spider_profile_mask": ([ctypes.c_uint32], _I),
    "spider_profile_classes": ([], _I),
    "spider_profile_class_name": ([_I], ctypes.c_char_p),
    "spider_profile_read": ([_I, ctypes.POINTER(_I64), ctypes.POINTER(_D)], _I),
}


def lib() -> ctypes.CDLL:
    """Load libspider.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_34977_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def exported_symbols():
    return list(_SIGS)


def _check(status: int):
    if status != 0:
        raise SpiderError(status, lib().spider_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ws(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256) + 256, dtype=torch.uint8, device=device)


def _aligned(buf: torch.Tensor):
    p = buf.data_ptr()
    return ctypes.c_void_p((p + 255) // 256 * 256)


# ----------------------------------------------------------------- host-only calls
def budget(keep: int, r_num: int = 7, r_den: int = 10):
    a, c = _I(), _I()
    _check(lib().spider_budget(keep, r_num, r_den, ctypes.byref(a), ctypes.byref(c)))
    return a.value, c.value


def budget_ratio(n: int, rv_num: int, rv_den: int, r_num: int = 7, r_den: int = 10):
    """(keep, n_anchor, n_cmp) for a retention ratio rv_num / rv_den of n tokens."""
    k, a, c = _I(), _I(), _I()
    _check(lib().spider_budget_ratio(n, rv_num, rv_den, r_num, r_den, ctypes.byref(k), ctypes.byref(a),
                                     ctypes.byref(c)))
    return k.value, a.value, c.value


def slc_policy(slc_attn, slc_ffn, eps: float = 1e-8):
    sa = np.ascontiguousarray(slc_attn, dtype=np.float32)
    sf = np.ascontiguousarray(slc_ffn, dtype=np.float32)
    L = len(sa)
    sel = np.zeros(L, np.float64)
    tgt = np.zeros(L, np.uint8)
    _check(lib().spider_slc_policy(L, sa.ctypes.data, sf.ctypes.data, eps, sel.ctypes.data,
                                   tgt.ctypes.data))
    return sel, tgt


def plan_skips(s_sa, slc_sel, target, w1: float, w2: float, T_skip: float, L: int):
    """s_sa [L//2, n_vis] float32 -> (codes [L, n_vis] uint8, admit [n_vis] int32)."""
    s = np.ascontiguousarray(s_sa, dtype=np.float32)
    n_vis = s.shape[1] if s.ndim == 2 else 0
    sel = np.ascontiguousarray(slc_sel, dtype=np.float64)
    tgt = np.ascontiguousarray(target, dtype=np.uint8)
    codes = np.zeros((L, n_vis), np.uint8)
    admit = np.zeros(n_vis, np.int32)
    _check(lib().spider_plan_skips(L, n_vis, s.ctypes.data if s.size else None, max(n_vis, 1) if s.ndim == 2 else 0,
                                   sel.ctypes.data, tgt.ctypes.data, w1, w2, T_skip,
                                   codes.ctypes.data if codes.size else None, n_vis,
                                   admit.ctypes.data if admit.size else None))
    return codes, admit


# ----------------------------------------------------------------- device calls
def anchor_colmean(attn: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Anchor scores without [CLS]: attn [G, H, n, n] fp32 (any strides with unit column
    stride) -> a [G, n] fp32, the mean over heads and query rows."""
    G, H, n, n2 = attn.shape
    if n2 != n or attn.stride(3) != 1:
        raise ValueError("attn must be [G, H, n, n] with contiguous rows")
    dev = attn.device
    if out is None:
        out = torch.empty(G, n, dtype=torch.float32, device=dev)
    L = lib()
    wsz = L.spider_anchor_colmean_workspace_size(G, H, n)
    ws = _ws(wsz, dev)
    _check(L.spider_anchor_colmean(G, H, n, _ptr(attn), attn.stride(0), attn.stride(1), attn.stride(2),
                                   _ptr(out), _aligned(ws), wsz, _stream(dev)))
    return out


def cls_attention(q: torch.Tensor, k: torch.Tensor, scale: float, out: Optional[torch.Tensor] = None):
    """[CLS] attention rows from q [G, H, dh] and keys k [G, T, H, dh] (last two dims
    contiguous) -> [G, H, T] fp32."""
    G, H, dh = q.shape
    T = k.shape[1]
    if k.shape != (G, T, H, dh) or q.stride(2) != 1 or q.stride(1) != dh or k.stride(3) != 1 or k.stride(2) != dh:
        raise ValueError("q must be [G, H, dh] and k [G, T, H, dh] with contiguous heads")
    if out is None:
        out = torch.empty(G, H, T, dtype=torch.float32, device=q.device)
    _check(lib().spider_cls_attention(G, H, dh, T, _ptr(q), q.stride(0), _ptr(k), k.stride(0), k.stride(1),
                                      _dt(q), scale, _ptr(out), _stream(q.device)))
    return out


def score(cls_attn: Optional[torch.Tensor], feats: Sequence[torch.Tensor], n_anchor: int, K: int = 4,
          max_iter: int = 10, attn_col0: int = 1, feat_row0: int = 1, n: Optional[int] = None,
          a: Optional[torch.Tensor] = None, noalloc: bool = False):
    """MSV-Prune scoring of G tiles.  cls_attn [G,H,T] fp32, feats list of [G,T,d_v];
    or cls_attn None and a [G, n] fp32 given anchor scores (encoders without [CLS]).
    With noalloc the call goes to spider_score_noalloc (the library's static scratch
    instead of a workspace)."""
    f0 = feats[0]
    d_v = f0.shape[-1]
    if cls_attn is None:
        if a is None:
            raise ValueError("give cls_attn or the anchor scores a")
        G, n = a.shape
        H, T = 0, 0
        dev = a.device
    else:
        G, H, T = cls_attn.shape
        n = T - attn_col0 if n is None else n
        dev = cls_attn.device
    for f in feats:
        if f.dtype != f0.dtype or f.shape != f0.shape or f.stride() != f0.stride():
            raise ValueError("all tapped layers must share dtype, shape and strides")
    # given scores are copied: the library reads them from (and leaves them in) a_out
    a = a.float().contiguous().clone() if cls_attn is None else torch.empty(G, n, dtype=torch.float32,
                                                                            device=dev)
    cl = torch.empty(G, n, dtype=torch.int32, device=dev)
    s = torch.empty(G, n, dtype=torch.float32, device=dev)
    m = torch.empty(G, n, dtype=torch.float32, device=dev)
    L = lib()
    fptr = (ctypes.c_void_p * len(feats))(*[f.data_ptr() for f in feats])
    if noalloc:
        _check(L.spider_score_noalloc(G, n, H, d_v, len(feats), _ptr(cls_attn),
                                      cls_attn.stride(0) if cls_attn is not None else 0,
                                      cls_attn.stride(1) if cls_attn is not None else 0, attn_col0, fptr,
                                      _dt(f0), f0.stride(0), f0.stride(1), feat_row0, n_anchor, K, max_iter,
                                      _ptr(a), _ptr(cl), _ptr(s), _ptr(m), _stream(dev)))
        return {"a": a, "cluster": cl, "s": s, "m": m}
    wsz = L.spider_score_workspace_size(G, n, d_v, len(feats), K)
    ws = _ws(wsz, dev)
    _check(L.spider_score(G, n, H, d_v, len(feats), _ptr(cls_attn),
                          cls_attn.stride(0) if cls_attn is not None else 0,
                          cls_attn.stride(1) if cls_attn is not None else 0, attn_col0, fptr, _dt(f0),
                          f0.stride(0), f0.stride(1),
                          feat_row0, n_anchor, K, max_iter, _ptr(a), _ptr(cl), _ptr(s), _ptr(m),
                          _aligned(ws), wsz, _stream(dev)))
    return {"a": a, "cluster": cl, "s": s, "m": m}


def select(cluster: torch.Tensor, s: torch.Tensor, n_anchor: int, n_cmp: int, K: int = 4,
           quota_mode: int = 0, cap: Optional[int] = None, tiles_per_sample: int = 1,
           src: Optional[torch.Tensor] = None, text: Optional[torch.Tensor] = None,
           text_only: bool = False, x_out: Optional[torch.Tensor] = None):
    """Quotas + selection (+ optional assembly of [kept visual | text] rows).  With
    text_only (and text given, src None) only the text rows and the boundaries are
    placed; spider_project_kept then writes the kept rows."""
    G, n = cluster.shape
    dev = cluster.device
    if cap is None:
        cap = min(n, n_anchor + n_cmp + K)
    idx = torch.empty(G, cap, dtype=torch.int32, device=dev)
    cnt = torch.empty(G, dtype=torch.int32, device=dev)
    x = cu = None
    d_model = n_text = 0
    dt = F32
    if src is not None or text_only:
        ref = src if src is not None else text
        d_model = ref.shape[-1]
        dt = _dt(ref)
        B = G // tiles_per_sample
        n_text = 0 if text is None else text.shape[1]
        x = x_out if x_out is not None else torch.empty(B * (tiles_per_sample * cap + n_text), d_model,
                                                          dtype=ref.dtype, device=dev)
        cu = torch.empty(B + 1, dtype=torch.int32, device=dev)
    _check(lib().spider_select(G, n, _ptr(cluster), _ptr(s), n_anchor, n_cmp, K, quota_mode,
                               _ptr(idx), _ptr(cnt), cap, tiles_per_sample, _ptr(src),
                               src.stride(0) if src is not None else 0, d_model, dt, _ptr(text),
                               n_text, _ptr(x), _ptr(cu), _stream(dev)))
    return {"idx": idx, "count": cnt, "x": x, "cu_seqlens": cu}


def project_kept(sel: dict, feats: torch.Tensor, proj: dict, tiles_per_sample: int = 1, n_text: int = 0,
                 feat_row0: int = 1, workspace: Optional[torch.Tensor] = None):
    """Projects the kept rows of ``sel`` (from select(..., text_only=True)) into sel["x"].
    feats [G, T, d_in]; proj = {"w1" [d_hid, d_in], "b1" [d_hid] fp32 or None, "w2", "b2"}."""
    idx, cnt, x = sel["idx"], sel["count"], sel["x"]
    G, cap = idx.shape
    w1, w2 = proj["w1"], proj["w2"]
    d_hid, d_in = w1.shape
    d_out = w2.shape[0]
    dev = feats.device
    L = lib()
    wsz = L.spider_project_kept_workspace_size(G, cap, d_hid, d_out, _dt(feats))
    if workspace is None or workspace.numel() < wsz + 256:
        workspace = _ws(wsz, dev)
    _check(L.spider_project_kept(G, tiles_per_sample, cap, _ptr(idx), _ptr(cnt), _ptr(feats), feats.stride(0),
                                 feats.stride(1), feat_row0, d_in, _ptr(w1), _ptr(proj.get("b1")), d_hid,
                                 _ptr(w2), _ptr(proj.get("b2")), d_out, n_text, _dt(feats), _ptr(x),
                                 _aligned(workspace), wsz, _stream(dev)))
    return x


def decoder_cfg(L: int, d: int, H: int, d_ff: int, dtype: int, eps: float = 1e-5,
                theta: float = 10000.0) -> DecoderCfg:
    return DecoderCfg(L, d, H, d_ff, eps, theta, dtype)


def layer_weights(weights: Sequence[dict]):
    arr = (LayerWeights * len(weights))()
    for i, w in enumerate(weights):
        arr[i] = LayerWeights(*[w[k].data_ptr() for k in
                                ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")])
    return arr


def prefill_workspace_size(cfg: DecoderCfg, B: int, rows: int) -> int:
    return lib().spider_prefill_workspace_size(ctypes.byref(cfg), B, rows)


def prefill(cfg: DecoderCfg, weights, cu_seqlens, x: torch.Tensor, codes,
            out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
            weight_table=None) -> torch.Tensor:
    """Skip-aware decoder prefill; returns h [rows, d] fp32 on x's device."""
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    B = len(cu) - 1
    rows = int(cu[-1])
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    if c.shape != (cfg.L, rows):
        raise ValueError(f"codes must be [L={cfg.L}, rows={rows}], got {c.shape}")
    dev = x.device
    if out is None:
        out = torch.empty(rows, cfg.d, dtype=torch.float32, device=dev)
    wsz = prefill_workspace_size(cfg, B, rows)
    if workspace is None or workspace.numel() < wsz + 256:
        workspace = _ws(wsz, dev)
    wt = weight_table if weight_table is not None else layer_weights(weights)
    _check(lib().spider_prefill(ctypes.byref(cfg), wt, B, cu.ctypes.data, _ptr(x),
                                c.ctypes.data if c.size else None, _ptr(out), _aligned(workspace),
                                wsz, _stream(dev)))
    return out


def prefill_online_workspace_size(cfg: DecoderCfg, B: int, rows: int, V: int) -> int:
    return lib().spider_prefill_online_workspace_size(ctypes.byref(cfg), B, rows, V)


# skip-rule ablation bits of spider_prefill_online_ablation
ONLINE_NO_EII, ONLINE_NO_FITC, ONLINE_NO_ACCUM, ONLINE_WHOLE_LAYER = 1, 2, 4, 8


def prefill_online(cfg: DecoderCfg, weights, cu_seqlens, x: torch.Tensor, n_text: int,
                   w_unembed: torch.Tensor, slc_sel, target, w1: float, w2: float, T_skip: float,
                   s_sa: bool = True, out: Optional[torch.Tensor] = None,
                   workspace: Optional[torch.Tensor] = None, weight_table=None, ablation: int = 0):
    """Prefill driven by the online skip controller (``ablation``: SPIDER_ONLINE_* bits,
    0 = the paper's rule through spider_prefill_online).

    Returns (h [rows, d] fp32, codes [L, rows] uint8, admit [rows] int32,
    S_sa [L//2, rows] fp32 or None)."""
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    B = len(cu) - 1
    rows = int(cu[-1])
    dev = x.device
    V = int(w_unembed.shape[0])
    if out is None:
        out = torch.empty(rows, cfg.d, dtype=torch.float32, device=dev)
    W = cfg.L // 2
    s_out = torch.empty(W, rows, dtype=torch.float32, device=dev) if (s_sa and W > 0) else None
    sel = np.ascontiguousarray(slc_sel, dtype=np.float64)
    tgt = np.ascontiguousarray(target, dtype=np.uint8)
    codes = np.zeros((cfg.L, rows), np.uint8)
    admit = np.full(rows, -1, np.int32)
    wsz = prefill_online_workspace_size(cfg, B, rows, V)
    if workspace is None or workspace.numel() < wsz + 256:
        workspace = _ws(wsz, dev)
    wt = weight_table if weight_table is not None else layer_weights(weights)
    head = (ctypes.byref(cfg), wt, B, cu.ctypes.data, _ptr(x), n_text, _ptr(w_unembed), V,
            sel.ctypes.data, tgt.ctypes.data, w1, w2, T_skip)
    tail = (codes.ctypes.data if codes.size else None, admit.ctypes.data if admit.size else None,
            _ptr(s_out), _ptr(out), _aligned(workspace), wsz, _stream(dev))
    if ablation:
        _check(lib().spider_prefill_online_ablation(*head, ablation, *tail))
    else:
        _check(lib().spider_prefill_online(*head, *tail))
    return out, codes, admit, s_out


def kv_cache(cfg: DecoderCfg, B: int, cap: int, device, dtype=None):
    """Allocates a KV cache [L][B][cap][d] (keys, values) and its descriptor."""
    dt = dtype or (torch.bfloat16 if cfg.dtype == BF16 else torch.float32)
    k = torch.zeros(cfg.L, B, cap, cfg.d, dtype=dt, device=device)
    v = torch.zeros_like(k)
    return {"k": k, "v": v, "desc": KVCache(k.data_ptr(), v.data_ptr(), cap)}


def prefill_kv(cfg: DecoderCfg, weights, cu_seqlens, x: torch.Tensor, codes, kv: dict,
               out: Optional[torch.Tensor] = None, weight_table=None) -> torch.Tensor:
    """spider_prefill that also fills the KV cache ``kv`` (from kv_cache())."""
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    B = len(cu) - 1
    rows = int(cu[-1])
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    dev = x.device
    if out is None:
        out = torch.empty(rows, cfg.d, dtype=torch.float32, device=dev)
    wsz = prefill_workspace_size(cfg, B, rows)
    ws = _ws(wsz, dev)
    wt = weight_table if weight_table is not None else layer_weights(weights)
    _check(lib().spider_prefill_kv(ctypes.byref(cfg), wt, B, cu.ctypes.data, _ptr(x),
                                   c.ctypes.data if c.size else None, _ptr(out), ctypes.byref(kv["desc"]),
                                   _aligned(ws), wsz, _stream(dev)))
    return out


def decode_workspace(cfg: DecoderCfg, B: int, cap: int, V: int, device) -> torch.Tensor:
    return _ws(lib().spider_decode_workspace_size(ctypes.byref(cfg), B, cap, V), device)


def decode_step(cfg: DecoderCfg, weights, lens, x: torch.Tensor, kv: dict, final_norm=None, w_unembed=None,
                weight_table=None, workspace: Optional[torch.Tensor] = None):
    """One decode step: x [B, d] new-token rows at positions lens (host ints).
    Returns (h [B, d] fp32, logits [B, V] fp32 or None, next ids [B] int32 or None)."""
    ln = np.ascontiguousarray(lens, dtype=np.int32)
    B = len(ln)
    dev = x.device
    V = int(w_unembed.shape[0]) if w_unembed is not None else 0
    h = torch.empty(B, cfg.d, dtype=torch.float32, device=dev)
    logits = torch.empty(B, V, dtype=torch.float32, device=dev) if V else None
    nxt = torch.empty(B, dtype=torch.int32, device=dev) if V else None
    wsz = lib().spider_decode_workspace_size(ctypes.byref(cfg), B, kv["desc"].cap, V)
    if workspace is None or workspace.numel() < wsz + 256:
        workspace = _ws(wsz, dev)
    wt = weight_table if weight_table is not None else layer_weights(weights)
    _check(lib().spider_decode_step(ctypes.byref(cfg), wt, B, ln.ctypes.data, _ptr(x), ctypes.byref(kv["desc"]),
                                    _ptr(final_norm), _ptr(w_unembed), V, _ptr(h), _ptr(logits), _ptr(nxt),
                                    _aligned(workspace), wsz, _stream(dev)))
    return h, logits, nxt


# ----------------------------------------------------------------- profiler
def profile_enable(on: bool = True):
    _check(lib().spider_profile_enable(1 if on else 0))


def profile_mask(classes=None):
    """Record only the named kernel classes (None = all)."""
    L = lib()
    if classes is None:
        m = 0xFFFFFFFF
    else:
        names = [L.spider_profile_class_name(c).decode() for c in range(L.spider_profile_classes())]
        m = 0
        for c in classes:
            m |= 1 << names.index(c)
    _check(L.spider_profile_mask(m))


def profile_read() -> dict:
    L = lib()
    out = {}
    for c in range(L.spider_profile_classes()):
        n, ms = _I64(), _D()
        _check(L.spider_profile_read(c, ctypes.byref(n), ctypes.byref(ms)))
        out[L.spider_profile_class_name(c).decode()] = (n.value, ms.value)
    return out
