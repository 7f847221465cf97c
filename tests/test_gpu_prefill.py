"""GPU decoder prefill (spider_prefill) against the oracle decoder.

Bars (per sample): max|h_gpu - h_oracle| / max|h_oracle| <= 1e-4 for the fp32
path and <= 2e-2 for the bf16 path (oracle with the bf16 rounding recipe);
bypassed rows bit-identical to their input; two runs bitwise identical.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as odec
from synth import get_workload
from synth.decoder_inputs import all_weights, layer_weights, MATS
from synth.vision import rng
from gpu_common import need_gpu, rel_err, log


def _cfg(L, dec, n_layers=None):
    return L.decoder_cfg(n_layers or dec.L, dec.d, dec.H, dec.d_ff,
                         L.BF16 if dec.dtype == "bf16" else L.F32, dec.eps, dec.theta)


def _codes(n_layers, cu, n_text, seed, p_attn, p_ffn, per_row):
    r = rng(seed, 950)
    rows = cu[-1]
    codes = np.zeros((n_layers, rows), np.uint8)
    for b in range(len(cu) - 1):
        n_vis = max(0, int(cu[b + 1] - cu[b]) - n_text)
        for l in range(n_layers):
            if per_row:
                ca = r.random(n_vis) < p_attn
                cf = r.random(n_vis) < p_ffn
            else:
                ca = np.full(n_vis, r.random() < p_attn)
                cf = np.full(n_vis, r.random() < p_ffn)
            codes[l, cu[b]:cu[b] + n_vis] = ca.astype(np.uint8) | (cf.astype(np.uint8) << 1)
    return codes


def _oracle_weights(dec, n_layers, seed=0):
    def get(l):
        lw = layer_weights(dec, l, seed, "cpu")
        return {k: v.float().numpy() for k, v in lw.items()}
    return get


def _run(L, dec, n_layers, cu, codes, x_cpu, seed=0):
    W = [layer_weights(dec, l, seed, "cuda") for l in range(n_layers)]
    cfg = _cfg(L, dec, n_layers)
    h = L.prefill(cfg, W, cu, x_cpu.cuda(), codes)
    torch.cuda.synchronize()
    return h.cpu().numpy(), W, cfg


def _x(dec, rows, seed):
    from synth.counter_rng import normal_bf16
    if dec.dtype == "bf16":
        return normal_bf16((rows, dec.d), seed, 4100, 0.5)
    return torch.from_numpy((rng(seed, 4100).standard_normal((rows, dec.d)) * 0.5).astype(np.float32))


PARITY = {
    # name: (workload, layers, cu_seqlens, n_text, p_attn, p_ffn, per_row)
    "tiny_mask": ("tiny", 2, [0, 48], 32, None, None, False),
    "tiny_ragged_rows": ("tiny", 2, [0, 37, 37, 90], 32, 0.4, 0.3, True),
    "tiny_dense": ("tiny", 2, [0, 48], 32, 0.0, 0.0, False),
    "7b_192_rows": ("llava15_7b", 2, [0, 192], 64, 0.5, 0.5, True),
    "7b_dense": ("llava15_7b", 2, [0, 192], 64, 0.0, 0.0, False),
    "7b_two_samples_ragged": ("llava15_7b", 2, [0, 131, 324], 64, 0.3, 0.3, True),
    "7b_704_rows_layer_mask": ("llava_next_7b", 2, [0, 704], 64, 0.5, 0.5, False),
    "7b_256_rows": ("llava15_7b", 1, [0, 256], 64, 0.3, 0.3, True),
    "7b_97_rows_dense": ("llava15_7b", 1, [0, 97], 64, 0.0, 0.0, False),
    # 257..384 rows (just past the streaming kernel's bound): 128-row tiles of the
    # large-row GEMM with split tail tiles in the SwiGLU launch
    "7b_300_rows_every_ffn": ("llava15_7b", 1, [0, 300], 64, 0.3, 0.0, True),
    "7b_two_samples_384_rows_dense": ("llava15_7b", 1, [0, 190, 384], 64, 0.0, 0.0, False),
    "13b_two_samples": ("llava15_13b", 1, [0, 256, 512], 128, 0.4, 0.2, True),
    # three ragged samples (the middle one text only) with a third of the visual
    # rows bypassing attention: query blocks of the shared-tile attention kernel
    # and row tiles of the large-row GEMM straddle sample boundaries
    "7b_three_ragged_1537_rows": ("llava15_7b", 1, [0, 1000, 1037, 1537], 64, 0.35, 0.2, True),
    # 3000 rows: the unsplit QKV GEMM applies RoPE and stores bf16 Q, K and V^T in its own
    # epilogue, here with 256-row tiles (the 1537-row case above takes 192-row tiles)
    "7b_three_ragged_3000_rows": ("llava15_7b", 1, [0, 1500, 1560, 3000], 64, 0.4, 0.2, True),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(PARITY))
def test_prefill_parity(case):
    L = need_gpu()
    wl, n_layers, cu, n_text, pa, pf, per_row = PARITY[case]
    w = get_workload(wl)
    dec = w.dec
    cu = np.array(cu, np.int32)
    rows = int(cu[-1])
    log(f"[prefill] case={case} L={n_layers} d={dec.d} rows={rows}")
    if pa is None:   # the tiny workload's own mask: attention of layer 1 off for visual rows
        codes = np.zeros((n_layers, rows), np.uint8)
        codes[1, :rows - n_text] = 1
    else:
        codes = _codes(n_layers, cu, n_text, 5, pa, pf, per_row)
    x = _x(dec, rows, 1)
    h, _, _ = _run(L, dec, n_layers, cu, codes, x)
    recipe = "bf16" if dec.dtype == "bf16" else "f32"
    ref = odec.prefill(x.float().numpy(), _oracle_weights(dec, n_layers), cu, codes, dec,
                       recipe=recipe, dtype=np.float64,
                       n_layers=n_layers)
    tol = 2e-2 if recipe == "bf16" else 1e-4
    for b in range(len(cu) - 1):
        if cu[b + 1] == cu[b]:
            continue
        e = rel_err(h[cu[b]:cu[b + 1]], ref[cu[b]:cu[b + 1]])
        log(f"  sample {b}: max rel err {e:.2e}")
        assert e <= tol, f"sample {b}: {e}"
    full = np.all(codes == 3, axis=0)
    assert np.array_equal(h[full], x.float().numpy()[full])


@pytest.mark.gpu
def test_bypassed_rows_keep_input_bits_and_runs_are_deterministic():
    L = need_gpu()
    w = get_workload("llava15_7b")
    dec = w.dec
    cu = np.array([0, 192], np.int32)
    codes = _codes(2, cu, 64, 9, 0.3, 0.3, True)
    codes[:, 10:20] = 3
    x = _x(dec, 192, 2)
    h1, W, cfg = _run(L, dec, 2, cu, codes, x)
    h2 = L.prefill(cfg, W, cu, x.cuda(), codes).cpu().numpy()
    assert np.array_equal(h1, h2)
    assert np.array_equal(h1[10:20], x.float().numpy()[10:20])


@pytest.mark.gpu
@pytest.mark.parametrize("wl,cu", [("llava_next_7b", [0, 705]), ("llava15_7b", [0, 1000, 1037, 1537]),
                                   ("llava15_7b", [0, 1500, 1560, 3000])])
def test_large_row_paths_are_deterministic(wl, cu):
    """More than 256 rows: tile GEMMs (the 705-row SwiGLU launch splits its last wave's tiles along k)
    and the shared-tile attention; two runs give the same bits.  Without a KV cache the unsplit QKV
    GEMM applies RoPE and stores bf16 Q, K and V^T in its epilogue; with one it writes fp32 sums and
    a separate kernel does that: both must give the same bits."""
    L = need_gpu()
    dec = get_workload(wl).dec
    cu = np.array(cu, np.int32)
    rows = int(cu[-1])
    log(f"[prefill] deterministic large rows: {wl} rows={rows}")
    codes = _codes(2, cu, 64, 11, 0.3, 0.2, True)
    x = _x(dec, rows, 4)
    h1, W, cfg = _run(L, dec, 2, cu, codes, x)
    h2 = L.prefill(cfg, W, cu, x.cuda(), codes).cpu().numpy()
    assert np.array_equal(h1, h2)
    assert np.all(np.isfinite(h1))
    kv = L.kv_cache(cfg, len(cu) - 1, int(max(cu[1:] - cu[:-1])), "cuda")
    h3 = L.prefill_kv(cfg, W, cu, x.cuda(), codes, kv).cpu().numpy()
    assert np.array_equal(h1, h3)


@pytest.mark.gpu
def test_all_rows_bypass_everything_is_identity():
    L = need_gpu()
    w = get_workload("llava15_7b")
    cu = np.array([0, 100], np.int32)
    codes = np.full((2, 100), 3, np.uint8)
    x = _x(w.dec, 100, 3)
    h, _, _ = _run(L, w.dec, 2, cu, codes, x)
    assert np.array_equal(h, x.float().numpy())


@pytest.mark.gpu
def test_full_depth_7b_properties():
    """32 layers at the benchmark shape (192 rows): finite, bypass identity, deterministic."""
    L = need_gpu()
    w = get_workload("llava15_7b")
    cu = np.array([0, 192], np.int32)
    codes = _codes(32, cu, 64, 13, 0.25, 0.25, False)
    codes[:, 0:4] = 3
    x = _x(w.dec, 192, 4)
    log("[prefill] full depth 7B, 192 rows")
    h1, W, cfg = _run(L, w.dec, 32, cu, codes, x)
    h2 = L.prefill(cfg, W, cu, x.cuda(), codes).cpu().numpy()
    assert np.all(np.isfinite(h1))
    assert np.array_equal(h1, h2)
    assert np.array_equal(h1[0:4], x.float().numpy()[0:4])
