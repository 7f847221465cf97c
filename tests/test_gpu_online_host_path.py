"""spider_prefill_online with its bookkeeping on the host at small row counts.

Up to 256 rows the online controller keeps admissions, codes and row lists on
the device, except where fewer than five text rows bound each sub-layer's row
count (B * n_text < 5), which would let the static prefill take the decode-row
GEMM; those calls build the row lists on the host.  These cases take that
path (one sample, n_text = 2), in fp32 and in bf16 with the fused lens, and
hold it to the same bars as test_gpu_online.py: admission layers and mask
identical to the oracle's, S_sa and h within the prefill bars, and h equal to
spider_prefill run with the mask the call built, bit for bit.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import asl_skip as ak
from oracle.online import prefill_online
from synth import get_workload
from synth.decoder_inputs import layer_weights
from synth.online_inputs import decoder_rows, unembed
from gpu_common import need_gpu, rel_err, log
from test_gpu_online import W1, W2, _layer_margins, _policy, _thresholds

CASES = {
    # name: (workload, layers, cu_seqlens, n_text, V)
    "tiny_fp32_two_text_rows": ("tiny", 4, [0, 70], 2, 1000),
    "7b_bf16_two_text_rows_fused_lens": ("llava15_7b", 2, [0, 130], 2, 32000),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_online_host_bookkeeping(case):
    L = need_gpu()
    wl, n_layers, cu, n_text, V = CASES[case]
    dec = get_workload(wl).dec
    bf16 = dec.dtype == "bf16"
    recipe = "bf16" if bf16 else "f32"
    cu = np.array(cu, np.int32)
    rows = int(cu[-1])
    Wn = n_layers // 2
    log(f"[online-host] case={case} L={n_layers} rows={rows} n_text={n_text}")
    x = decoder_rows(dec, cu, n_text, seed=5)
    wu_cpu = unembed(dec, V, seed=6)
    vis_rows = [r for b in range(len(cu) - 1) for r in range(int(cu[b]), int(cu[b + 1]) - n_text)]

    sa, sf = _policy(n_layers)
    na, nf = ak.slc_normalize(sa, sf)
    m, sel = ak.skip_targets(na, nf)
    cfg_o = dataclasses.replace(dec, L=n_layers)
    wts = lambda l: {k: v.float().numpy() for k, v in layer_weights(dec, l, 0, "cpu").items()}
    xo = x.float().numpy()
    wuo = wu_cpu.float().numpy()

    def oracle(T):
        return prefill_online(xo, wts, cu, n_text, wuo, sel, m, W1, W2, T, cfg_o, recipe=recipe)

    _, _, _, S_free = oracle(np.inf)
    margin_need = [1e-3] + [2e-2 if bf16 else 1e-3] * (Wn - 1)
    chosen = None
    for T in _thresholds(S_free, sel, vis_rows):
        ref = oracle(T)
        mg = _layer_margins(ref[3], ref[2], sel, T, vis_rows)
        if all(v >= need for v, need in zip(mg, margin_need)):
            chosen = (T, ref)
            break
    assert chosen is not None, "no threshold keeps the oracle's decisions clear of it"
    T, (h_o, codes_o, admit_o, S_o) = chosen
    log(f"  T_skip={T:.6f}: admitted {int((admit_o[vis_rows] >= 0).sum())} of {len(vis_rows)} visual rows")

    sel_g, tgt_g = L.slc_policy(sa, sf, 1e-8)
    W = [layer_weights(dec, l, 0, "cuda") for l in range(n_layers)]
    cfg = L.decoder_cfg(n_layers, dec.d, dec.H, dec.d_ff, L.BF16 if bf16 else L.F32, dec.eps, dec.theta)
    h, codes, admit, S = L.prefill_online(cfg, W, cu, x.cuda(), n_text, wu_cpu.cuda(), sel_g, tgt_g, W1, W2, T)
    hs = L.prefill(cfg, W, cu, x.cuda(), codes)
    torch.cuda.synchronize()
    assert torch.equal(h, hs)
    S = S.cpu().numpy()
    for l in range(Wn):
        cand = [r for r in vis_rows if admit_o[r] < 0 or admit_o[r] >= l]
        e = float(np.max(np.abs(S[l, cand] - S_o[l, cand]))) if cand else 0.0
        log(f"  layer {l}: {len(cand)} scored, max |dS_sa| {e:.2e}")
        assert e <= (1e-4 if (l == 0 or not bf16) else 1e-2), (l, e)
    assert np.array_equal(admit, admit_o.astype(np.int32))
    assert np.array_equal(codes, codes_o)
    e = rel_err(h.cpu().numpy(), h_o)
    log(f"  max rel err {e:.2e}")
    assert e <= (2e-2 if bf16 else 1e-4)
