"""Shared pieces of the GPU parity tests: device checks and oracle references."""
import os
import sys

import numpy as np
import pytest
import torch

from oracle import msv_prune as mp


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34977_amd import _lib
    if not os.path.exists(_lib._LIB_PATH):
        raise RuntimeError("libspider.so is not built; the GPU tests need the HIP library")
    return _lib


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_tiles(attn, feats, keep, r_num=7, r_den=10, K=4, iters=10, mode="literal"):
    """Run the oracle MSV-Prune on every tile; inputs are CPU torch tensors."""
    A = attn.numpy()
    F = [f.float().numpy() for f in feats]
    return [mp.prune_tile(A[g], [f[g] for f in F], keep, r_num, r_den, K, iters, mode)
            for g in range(A.shape[0])]


def rel_err(g: np.ndarray, o: np.ndarray) -> float:
    return float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-30))
