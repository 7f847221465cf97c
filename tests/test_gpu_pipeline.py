"""Whole hot path on the tiny fp32 workload vs the oracle pipeline."""
import pytest

from e2e import run_tiny_end_to_end
from gpu_common import need_gpu, log


@pytest.mark.gpu
@pytest.mark.parametrize("keep", [16, 30, 49])
def test_tiny_end_to_end(keep):
    need_gpu()
    log(f"[e2e] tiny keep={keep}")
    r = run_tiny_end_to_end(keep=keep)
    assert r["idx_equal"] and r["cu_equal"] and r["codes_equal"], r
    assert r["rel_err"] <= 1e-4, r
