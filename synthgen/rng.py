"""Counter-based random numbers that give the same bits on any device.

Every tensor is a pure function of (seed, tensor id, element index):

* key = mix64(mix64(seed) XOR tensor_id)
* raw[i] = mix64(key + (i + 1) * 0x9E3779B97F4A7C15 mod 2^64)

which is the i-th output of Vigna's splitmix64 generator started from
state ``key`` (the finaliser ``mix64`` is the published splitmix64 one).
All of it is 64-bit integer work, done with torch int64 tensors (two's
complement wrap-around, logical shifts emulated with masks), so a CPU and a
GPU produce identical integers.

Floats are derived with at most one float multiply:

* uniform_f64: the top 53 bits times 2^-53;
* normal_f32: an Irwin-Hall sum of the four 16-bit fields of raw[i],
  centred exactly in integers, then one fp32 multiply by
  fp32(sigma * sqrt(3) / 65536) (variance of a U(0,1) sum of four is 1/3).
"""
from __future__ import annotations

import math

import torch

_M64 = (1 << 64) - 1


def _i64(c: int) -> int:
    c &= _M64
    return c - (1 << 64) if c >= (1 << 63) else c


GOLDEN = 0x9E3779B97F4A7C15
_MUL1 = 0xBF58476D1CE4E5B9
_MUL2 = 0x94D049BB133111EB


def mix64_int(x: int) -> int:
    """splitmix64 finaliser on a Python int (mod 2^64)."""
    x &= _M64
    x = ((x ^ (x >> 30)) * _MUL1) & _M64
    x = ((x ^ (x >> 27)) * _MUL2) & _M64
    return x ^ (x >> 31)


def key_for(seed: int, tensor_id: int) -> int:
    return mix64_int(mix64_int(seed) ^ (tensor_id & _M64))


def _srl(x: torch.Tensor, s: int) -> torch.Tensor:
    # logical right shift of an int64 tensor
    return (x >> s) & ((1 << (64 - s)) - 1)


def _mix64_t(x: torch.Tensor) -> torch.Tensor:
    x = x ^ _srl(x, 30)
    x = x * _i64(_MUL1)
    x = x ^ _srl(x, 27)
    x = x * _i64(_MUL2)
    return x ^ _srl(x, 31)


def splitmix64_stream(seed: int, tensor_id: int, start: int, count: int,
                      device="cpu") -> torch.Tensor:
    """raw[start .. start+count) as an int64 tensor (bit pattern of u64)."""
    key = key_for(seed, tensor_id)
    idx = torch.arange(start + 1, start + 1 + count, dtype=torch.int64,
                       device=device)
    state = idx * _i64(GOLDEN) + _i64(key)
    return _mix64_t(state)


_CHUNK = 1 << 25


def uniform_f64(seed: int, tensor_id: int, count: int, device="cpu",
                start: int = 0) -> torch.Tensor:
    """U[0,1) in float64: top 53 bits of raw[i] times 2^-53."""
    raw = splitmix64_stream(seed, tensor_id, start, count, device)
    return _srl(raw, 11).to(torch.float64) * (2.0 ** -53)


def uniform_u64_key(seed: int, tensor_id: int, count: int) -> torch.Tensor:
    """The top 63 bits of raw[i] as non-negative int64 (sort keys)."""
    return _srl(splitmix64_stream(seed, tensor_id, 0, count), 1)


def normal_f32(seed: int, tensor_id: int, shape, sigma: float,
               device="cpu", start: int = 0) -> torch.Tensor:
    """N(0, sigma^2)-shaped fp32 draws (Irwin-Hall of four 16-bit fields)."""
    count = 1
    for s in shape:
        count *= int(s)
    scale = torch.tensor(sigma * math.sqrt(3.0) / 65536.0,
                         dtype=torch.float32).item()
    out = torch.empty(count, dtype=torch.float32, device=device)
    pos = 0
    while pos < count:
        n = min(_CHUNK, count - pos)
        raw = splitmix64_stream(seed, tensor_id, start + pos, n, device)
        s = (raw & 0xFFFF) + (_srl(raw, 16) & 0xFFFF) \
            + (_srl(raw, 32) & 0xFFFF) + _srl(raw, 48)
        centred = (s - 131070).to(torch.float32)  # exact: |.| < 2^24
        out[pos:pos + n] = centred * scale
        pos += n
    return out.view(*shape)


def permutation(seed: int, tensor_id: int, n: int) -> torch.Tensor:
    """A seeded permutation of range(n) (argsort of distinct 63-bit keys)."""
    keys = uniform_u64_key(seed, tensor_id, n)
    return torch.argsort(keys, stable=True)
