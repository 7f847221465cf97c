"""Whole hot path (score -> select/assemble -> skip plan -> prefill) vs the oracle pipeline.

Bars: kept indices, sample boundaries and skip codes identical; the final
residual per sample within 1e-4 (fp32 workload) or 2e-2 (bf16 recipe) of the
float64 oracle, relative to the sample's largest magnitude.  These cases run
at most 8 layers; the full-depth bf16 workloads are checked layer by layer in
test_gpu_depth.py (teacher-forced at the same 2e-2), where the end-to-end
drift over all layers is also logged.
"""
import pytest

from e2e import run_end_to_end, run_tiny_end_to_end
from gpu_common import need_gpu, log


@pytest.mark.gpu
@pytest.mark.parametrize("keep", [16, 30, 49])
def test_tiny_end_to_end(keep):
    need_gpu()
    log(f"[e2e] tiny keep={keep}")
    r = run_tiny_end_to_end(keep=keep)
    assert r["idx_equal"] and r["cu_equal"] and r["codes_equal"], r
    assert r["rel_err"] <= 1e-4, r


CASES = {
    # name: (workload, keep, layers, skip_p)
    # the LLaVA-1.5-7B configuration over its first 8 layers (own random mask for 8 layers)
    "llava15_7b_keep128_8_layers": ("llava15_7b", None, 8, None),
    # eight samples, 2049 rows (the tile GEMM path), one layer
    "llava15_13b_batch8_one_layer": ("llava15_13b", None, 1, 0.3),
}


@pytest.mark.gpu
@pytest.mark.parametrize("case", list(CASES))
def test_end_to_end(case):
    need_gpu()
    name, keep, layers, p = CASES[case]
    log(f"[e2e] {case}")
    r = run_end_to_end(name, keep=keep, n_layers=layers, skip_p=p)
    log(f"  rows {r['rows']} skipped {r['skipped_fraction']:.3f} max rel err {max(r['rel_err']):.2e}")
    assert r["idx_equal"] and r["cu_equal"] and r["codes_equal"], r
    assert max(r["rel_err"]) <= 2e-2, r
