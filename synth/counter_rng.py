"""Counter-based generator for large synthetic tensors (CPU and GPU identical).

Element ``i`` of tensor ``tensor_id`` under ``seed`` takes the 64-bit counter
``(seed << 56) | (tensor_id << 40) | i`` and hashes it with SplitMix64
(Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
OOPSLA 2014; the finaliser constants are those of that publication).  The
64-bit output is split into four 16-bit uniforms whose sum (Irwin-Hall of
order 4) is centred and scaled to the requested standard deviation.  Every
step up to the final scale is exact integer arithmetic and the scale is one
IEEE fp32 multiply, so CPU and GPU produce bit-identical values.  The
distribution is a close approximation of N(0, std^2) bounded at about
+-3.46 std.

bf16 values are produced by round-to-nearest-even on the fp32 bit pattern
(integer arithmetic), again identical on every device.
"""
from __future__ import annotations

import torch

_GOLDEN = 0x9E3779B97F4A7C15
_C1 = 0xBF58476D1CE4E5B9
_C2 = 0x94D049BB133111EB


def _s64(v: int) -> int:
    """Unsigned 64-bit constant -> the int64 with the same bits."""
    return v - (1 << 64) if v >= (1 << 63) else v


_GOLDEN_S, _C1_S, _C2_S = _s64(_GOLDEN), _s64(_C1), _s64(_C2)
# sqrt(var) of the centred sum of four independent U{0..65535}: 65536/sqrt(3)
_IH4_STD = 37837.23112659009
_CHUNK = 1 << 20          # CPU chunk (cache-sized temporaries)
_CHUNK_GPU = 1 << 26


def _chunk(device) -> int:
    return _CHUNK_GPU if torch.device(device).type == "cuda" else _CHUNK


def _lsr(z: torch.Tensor, k: int) -> torch.Tensor:
    """Logical right shift of int64 bits."""
    return (z >> k) & ((1 << (64 - k)) - 1)


def _splitmix64(c: torch.Tensor) -> torch.Tensor:
    z = c + _GOLDEN_S
    z = (z ^ _lsr(z, 30)) * _C1_S
    z = (z ^ _lsr(z, 27)) * _C2_S
    return z ^ _lsr(z, 31)


def _normal_chunk(seed: int, tensor_id: int, start: int, n: int, std: float,
                  device) -> torch.Tensor:
    idx = torch.arange(start, start + n, dtype=torch.int64, device=device)
    c = idx | ((seed << 56) | (tensor_id << 40))
    z = _splitmix64(c)
    s = (z & 0xFFFF) + ((z >> 16) & 0xFFFF) + ((z >> 32) & 0xFFFF) + ((z >> 48) & 0xFFFF)
    s = (s - 2 * 65535).to(torch.float32)          # exact: |s| <= 131070
    scale = torch.tensor(std / _IH4_STD, dtype=torch.float32, device=device)
    return s * scale


def _check(seed: int, tensor_id: int, numel: int) -> None:
    if not (0 <= seed < 128):
        raise ValueError("seed must be in [0, 128)")
    if not (0 <= tensor_id < (1 << 16)):
        raise ValueError("tensor_id must be in [0, 65536)")
    if numel >= (1 << 40):
        raise ValueError("tensor too large for the counter layout")


def normal_f32(shape, seed: int, tensor_id: int, std: float = 0.02,
               device="cpu") -> torch.Tensor:
    """fp32 tensor of approximately N(0, std^2) values."""
    numel = 1
    for s in shape:
        numel *= int(s)
    _check(seed, tensor_id, numel)
    out = torch.empty(numel, dtype=torch.float32, device=device)
    ch = _chunk(device)
    for st in range(0, numel, ch):
        n = min(ch, numel - st)
        out[st:st + n] = _normal_chunk(seed, tensor_id, st, n, std, device)
    return out.view(*shape)


def f32_to_bf16_rne(x: torch.Tensor) -> torch.Tensor:
    """Round fp32 -> bf16 (nearest-even) with integer ops; finite inputs only."""
    b = x.contiguous().view(torch.int32)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return r.to(torch.int16).view(torch.bfloat16)


def normal_bf16(shape, seed: int, tensor_id: int, std: float = 0.02,
                device="cpu") -> torch.Tensor:
    """bf16 tensor of approximately N(0, std^2) values (RNE from fp32)."""
    numel = 1
    for s in shape:
        numel *= int(s)
    _check(seed, tensor_id, numel)
    out = torch.empty(numel, dtype=torch.bfloat16, device=device)
    ch = _chunk(device)
    for st in range(0, numel, ch):
        n = min(ch, numel - st)
        out[st:st + n] = f32_to_bf16_rne(_normal_chunk(seed, tensor_id, st, n, std, device))
    return out.view(*shape)
