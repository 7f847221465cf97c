"""GPU KV cache of the prefill (spider_prefill_kv) and decode steps with the LM
head (spider_decode_step) against the oracle (a decode step is the skip-aware
prefill over the extended sequence, read at the new rows).

Bars: the prefill's h equals spider_prefill's bit for bit; cached keys and
values within 1e-2 (bf16: both sides round the same fp32-accumulated values,
a rounding flip moves one element by one bf16 step) / 1e-5 (fp32) of the
oracle relative to the layer's largest entry, slots past a sample untouched;
decode states within the prefill bars (2e-2 / 1e-4) per step; logits within
2e-2 / 1e-4 of the oracle relative to the largest logit; the greedy token
equal wherever the oracle's two best logits are further apart than that bar.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import decode as od
from oracle import decoder as odec
from synth import get_workload
from synth.decoder_inputs import layer_weights
from synth.online_inputs import unembed
from synth.vision import rng
from gpu_common import need_gpu, rel_err, log

CASES = {
    # name: (workload, layers, cu_seqlens, n_text, V, steps)
    "tiny_fp32": ("tiny", 2, [0, 40, 77], 32, 1000, 3),
    "7b_two_samples": ("llava15_7b", 2, [0, 150, 342], 64, 32000, 3),
    # one sample: the 1-row GEMVs with the fused RMSNorm and residual adds
    "7b_one_sample": ("llava15_7b", 2, [0, 192], 64, 32000, 3),
    # three samples: the 4-row GEMVs with one zero-padded row
    "7b_three_samples": ("llava15_7b", 2, [0, 100, 180, 290], 64, 32000, 2),
    # five samples: more than 4 rows, split-K GEMMs with separate norm kernels
    "7b_five_samples": ("llava15_7b", 1, [0, 70, 140, 210, 280, 350], 64, 32000, 2),
}


def _x(dec, rows, seed):
    from synth.counter_rng import normal_bf16
    if dec.dtype == "bf16":
        return normal_bf16((rows, dec.d), seed, 4700, 0.5)
    return torch.from_numpy((rng(seed, 4700).standard_normal((rows, dec.d)) * 0.5).astype(np.float32))


def _codes(L, cu, n_text, seed):
    r = rng(seed, 4701)
    rows = int(cu[-1])
    codes = np.zeros((L, rows), np.uint8)
    for b in range(len(cu) - 1):
        n_vis = int(cu[b + 1] - cu[b]) - n_text
        codes[:, cu[b]:cu[b] + n_vis] = (r.random((L, n_vis)) < 0.3) | ((r.random((L, n_vis)) < 0.3) << 1)
    codes[L - 1, :] |= 1       # last layer: no row is a query, the cache still needs its keys and values
    return codes


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_prefill_cache_and_decode_steps(case):
    L = need_gpu()
    wl, n_layers, cu, n_text, V, steps = CASES[case]
    dec = dataclasses.replace(get_workload(wl).dec, L=n_layers)
    bf16 = dec.dtype == "bf16"
    recipe = "bf16" if bf16 else "f32"
    cu = np.array(cu, np.int32)
    B, rows = len(cu) - 1, int(cu[-1])
    log(f"[decode] case={case} L={n_layers} d={dec.d} rows={rows} steps={steps}")
    x = _x(dec, rows, 1)
    codes = _codes(n_layers, cu, n_text, 2)
    new = [_x(dec, steps, 10 + b) for b in range(B)]
    wu = unembed(dec, V, seed=3)
    fn = torch.ones(dec.d, dtype=torch.float32)
    W = [layer_weights(dec, l, 0, "cuda") for l in range(n_layers)]
    cfg = L.decoder_cfg(n_layers, dec.d, dec.H, dec.d_ff, L.BF16 if bf16 else L.F32, dec.eps, dec.theta)
    cap = int(max(cu[1:] - cu[:-1])) + steps + 5
    kv = L.kv_cache(cfg, B, cap, "cuda")
    h_kv = L.prefill_kv(cfg, W, cu, x.cuda(), codes, kv)
    h_plain = L.prefill(cfg, W, cu, x.cuda(), codes)
    lens = (cu[1:] - cu[:-1]).astype(np.int32)
    outs = []
    for t in range(steps):
        xt = torch.stack([new[b][t] for b in range(B)]).cuda()
        h, logits, nxt = L.decode_step(cfg, W, lens, xt, kv, fn.cuda(), wu.cuda())
        outs.append((h.cpu().numpy(), logits.cpu().numpy(), nxt.cpu().numpy()))
        lens = lens + 1
    torch.cuda.synchronize()
    assert torch.equal(h_kv, h_plain)

    # oracle: the prefill over the extended sequences, its keys and values, the LM head
    wts = lambda l: {k: v.float().numpy() for k, v in layer_weights(dec, l, 0, "cpu").items()}
    kvo = []
    h_new, (xe, cue, ce, where) = od.decode(x.float().numpy(), wts, cu, codes,
                                            [new[b].float().numpy() for b in range(B)], dec, recipe=recipe,
                                            kv=kvo)
    tol_kv = 1e-2 if bf16 else 1e-5
    tol_h = 2e-2 if bf16 else 1e-4
    Kc, Vc = kv["k"].float().cpu().numpy(), kv["v"].float().cpu().numpy()
    for l in range(n_layers):
        Ko, Vo = kvo[l]
        for b in range(B):
            n_b = int(cue[b + 1] - cue[b])
            for name, C, O in (("K", Kc, Ko), ("V", Vc, Vo)):
                e = rel_err(C[l, b, :n_b], O[cue[b]:cue[b + 1]])
                assert e <= tol_kv, f"layer {l} sample {b} cached {name}: {e}"
                assert np.all(C[l, b, n_b:] == 0.0), f"layer {l} sample {b}: slots past the sample written"
    wuo = wu.float().numpy()
    for t in range(steps):
        hg, lg, ng = outs[t]
        ho = np.stack([h_new[b][t] for b in range(B)])
        lo = od.lm_head(ho, fn.numpy(), wuo, dec.eps, recipe)
        eh = rel_err(hg, ho)
        el = float(np.max(np.abs(lg - lo)) / np.max(np.abs(lo)))
        log(f"  step {t}: h err {eh:.2e}, logits err {el:.2e}, tokens {list(ng)} / {list(od.next_tokens(lo))}")
        assert eh <= tol_h and el <= tol_h, (t, eh, el)
        for b in range(B):
            top = np.sort(lo[b])[::-1]
            if top[0] - top[1] > 2 * tol_h * np.max(np.abs(lo)):
                assert ng[b] == od.next_tokens(lo)[b], f"step {t} sample {b}: greedy token"


@pytest.mark.gpu
def test_decode_is_deterministic_and_leaves_other_slots():
    L = need_gpu()
    dec = dataclasses.replace(get_workload("llava15_7b").dec, L=2)
    cfg = L.decoder_cfg(2, dec.d, dec.H, dec.d_ff, L.BF16, dec.eps, dec.theta)
    W = [layer_weights(dec, l, 0, "cuda") for l in range(2)]
    cu = np.array([0, 100], np.int32)
    x = _x(dec, 100, 5).cuda()
    codes = np.zeros((2, 100), np.uint8)
    outs = []
    for _ in range(2):
        kv = L.kv_cache(cfg, 1, 128, "cuda")
        L.prefill_kv(cfg, W, cu, x, codes, kv)
        h, _, _ = L.decode_step(cfg, W, [100], _x(dec, 1, 6).cuda(), kv)
        torch.cuda.synchronize()
        outs.append((h.clone(), kv["k"].clone(), kv["v"].clone()))
    assert all(torch.equal(a, b) for a, b in zip(outs[0], outs[1]))
    assert torch.count_nonzero(outs[0][1][:, 0, 101:]) == 0
