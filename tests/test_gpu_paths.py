"""GPU parity on decoder paths that the workload-shaped tests do not take.

Found by tracing the GPU suite with rocprofv3's kernel statistics against the
kernel instantiations the library holds; each case makes one of those paths
run against the oracle, with the bars of test_gpu_prefill:

* the LDS-staged GEMM kernel: a bf16 decoder whose widths are not multiples of
  the large-row kernel's tiles (d = 384, three heads of 128; d_ff = 704) over
  more than 256 rows, so QKV (fp32 partials plus the finalize), O and down run
  as 128 x 128 tiles and the SwiGLU launch as 128 x 64; the same decoder at 200
  rows stays on the streaming kernel;
* the fp32 RMSNorm for rows wider than 4096 (d = 4224, 33 heads of 128).
"""
import dataclasses

import numpy as np
import pytest

from oracle import decoder as odec
from synth import get_workload
from gpu_common import need_gpu, rel_err, log
from test_gpu_prefill import _codes, _oracle_weights, _run, _x

CASES = {
    # name: (decoder overrides, layers, cu_seqlens, n_text, p_attn, p_ffn)
    "bf16_d384_dff704_200_rows": (("llava15_7b", dict(d=384, H=3, d_ff=704)), 2, [0, 200], 64, 0.3, 0.3),
    "bf16_d384_dff704_300_rows": (("llava15_7b", dict(d=384, H=3, d_ff=704)), 2, [0, 300], 64, 0.3, 0.3),
    "bf16_d384_dff704_two_samples_700_rows": (("llava15_7b", dict(d=384, H=3, d_ff=704)), 2, [0, 420, 700], 64,
                                              0.3, 0.2),
    "fp32_d4224_40_rows": (("tiny", dict(d=4224, H=33, d_ff=512)), 1, [0, 40], 16, 0.3, 0.3),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_prefill_uncommon_widths(case):
    L = need_gpu()
    (wl, over), n_layers, cu, n_text, pa, pf = CASES[case]
    dec = dataclasses.replace(get_workload(wl).dec, L=n_layers, **over)
    cu = np.array(cu, np.int32)
    rows = int(cu[-1])
    log(f"[prefill paths] case={case} d={dec.d} H={dec.H} d_ff={dec.d_ff} {dec.dtype} rows={rows}")
    codes = _codes(n_layers, cu, n_text, 7, pa, pf, True)
    x = _x(dec, rows, 3)
    h, _, _ = _run(L, dec, n_layers, cu, codes, x)
    recipe = "bf16" if dec.dtype == "bf16" else "f32"
    ref = odec.prefill(x.float().numpy(), _oracle_weights(dec, n_layers), cu, codes, dec,
                       recipe=recipe, dtype=np.float64, n_layers=n_layers)
    tol = 2e-2 if recipe == "bf16" else 1e-4
    for b in range(len(cu) - 1):
        e = rel_err(h[cu[b]:cu[b + 1]], ref[cu[b]:cu[b + 1]])
        log(f"  sample {b}: max rel err {e:.2e}")
        assert e <= tol, f"sample {b}: {e}"
    full = np.all(codes == 3, axis=0)
    assert np.array_equal(h[full], x.float().numpy()[full])
