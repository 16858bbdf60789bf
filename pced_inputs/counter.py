"""Counter-based seeded value streams shared by every side of the PCED test harness.

This module produces *input bits only*: cache contents, queries, LM-head weights.
It holds none of the decoding method's arithmetic. Both the GPU path and the CPU
oracle receive identical bits from it, so any disagreement between them is a
disagreement in the method, never in the inputs.

Generator
---------
SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014): the state advances by the golden-ratio increment
``G = 0x9E3779B97F4A7C15`` and each output is the finaliser ``mix`` applied to the
state. The i-th output (i = 0, 1, ...) of a stream seeded with ``k`` is therefore
``mix(k + (i + 1) * G)``, which makes element ``i`` of a tensor computable on its
own (counter-based), on the host or on the device, in any order.

Stream keys
-----------
``key(seed, f1, f2, ...)`` folds integer fields into a 64-bit key with
``k <- mix((k ^ f) + G)``, starting from ``k = seed``.

Values
------
A 64-bit output ``h`` is split into four 16-bit fields ``u0..u3``. Their sum ``U``
is an Irwin-Hall(4) draw on the integer grid; ``U - 131070`` is centred and, being
an integer of magnitude <= 131070, exactly representable in float32. The value is
``float32(U - 131070) * float32(scale * sqrt(3) / 65536)``: one IEEE float32
multiply, so every implementation gets identical bits. Its variance is
``scale**2 * (1 - 2**-32)``, close to N(0, scale**2) and bounded by
``|x| <= 3.46 * scale``. Values destined for bf16 storage are rounded to nearest
even from that float32 value.
"""
from __future__ import annotations

import math

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
MIX_M1 = 0xBF58476D1CE4E5B9
MIX_M2 = 0x94D049BB133111EB
IH_CENTER = 131070  # 4 * 65535 / 2


def mix64(z: int) -> int:
    """SplitMix64 finaliser on a Python int (mod 2**64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX_M1) & MASK64
    z = ((z ^ (z >> 27)) * MIX_M2) & MASK64
    return z ^ (z >> 31)


def splitmix64_sequence(seed: int, n: int) -> list[int]:
    """The first ``n`` outputs of SplitMix64 seeded with ``seed``."""
    out, state = [], seed & MASK64
    for _ in range(n):
        state = (state + GOLDEN) & MASK64
        out.append(mix64(state))
    return out


def key(seed: int, *fields: int) -> int:
    """Fold integer fields into a 64-bit stream key."""
    k = seed & MASK64
    for f in fields:
        k = mix64(((k ^ (f & MASK64)) + GOLDEN) & MASK64)
    return k


def value_scale(scale: float) -> np.float32:
    """The float32 multiplier that maps the centred Irwin-Hall integer to a value."""
    return np.float32(scale * math.sqrt(3.0) / 65536.0)


# ----------------------------------------------------------------- numpy (host)

def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * np.uint64(MIX_M1)
    z = z ^ (z >> np.uint64(27))
    z = z * np.uint64(MIX_M2)
    return z ^ (z >> np.uint64(31))


def hashes_np(k: int, start: int, count: int) -> np.ndarray:
    """Outputs ``start .. start+count-1`` of the SplitMix64 stream seeded with ``k``."""
    idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        state = np.uint64(k) + idx * np.uint64(GOLDEN)
        return _mix64_np(state)


def values_f32_np(k: int, start: int, count: int, scale: float) -> np.ndarray:
    """float32 values ``start .. start+count-1`` of stream ``k``."""
    h = hashes_np(k, start, count)
    m = np.uint64(0xFFFF)
    u = (h & m) + ((h >> np.uint64(16)) & m) + ((h >> np.uint64(32)) & m) + (h >> np.uint64(48))
    centred = (u.astype(np.int64) - IH_CENTER).astype(np.float32)
    return centred * value_scale(scale)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16, nearest-even, returned as uint16 bit patterns.

    Inputs here are finite (the generator never makes inf/NaN)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def values_np(k: int, start: int, count: int, scale: float, dtype: str, offset: float = 0.0) -> np.ndarray:
    """Values as stored: uint16 bf16 bits for ``dtype='bf16'``, float32 for ``'f32'``.
    A non-zero ``offset`` is added in float32 before the rounding to storage
    (distributions centred away from 0, such as norm weights around 1)."""
    v = values_f32_np(k, start, count, scale)
    if offset:
        v = v + np.float32(offset)
    if dtype == "bf16":
        return f32_to_bf16_bits(v)
    if dtype == "f32":
        return v
    raise ValueError(f"unknown dtype {dtype!r}")


# ------------------------------------------------------------- torch (device)

def _as_i64(x: int) -> int:
    x &= MASK64
    return x - (1 << 64) if x >= (1 << 63) else x


def _mix64_torch(z):
    import torch

    def lsr(v, s):  # logical shift right on int64 bit patterns
        return (v >> s) & ((1 << (64 - s)) - 1)

    z = z ^ lsr(z, 30)
    z = z * torch.tensor(_as_i64(MIX_M1), dtype=torch.int64, device=z.device)
    z = z ^ lsr(z, 27)
    z = z * torch.tensor(_as_i64(MIX_M2), dtype=torch.int64, device=z.device)
    return z ^ lsr(z, 31)


def values_torch(k: int, start: int, count: int, scale: float, dtype: str, device, offset: float = 0.0):
    """Same bits as :func:`values_np`, computed on ``device`` with int64 torch ops.

    int64 multiply wraps modulo 2**64 in two's complement, which gives the same bit
    pattern as the unsigned product; shifts are made logical by masking."""
    import torch

    idx = torch.arange(start + 1, start + count + 1, dtype=torch.int64, device=device)
    state = idx * torch.tensor(_as_i64(GOLDEN), dtype=torch.int64, device=device)
    state = state + torch.tensor(_as_i64(k), dtype=torch.int64, device=device)
    h = _mix64_torch(state)
    del state, idx
    m = 0xFFFF
    u = (h & m) + ((h >> 16) & m) + ((h >> 32) & m) + ((h >> 48) & m)
    del h
    v = (u - IH_CENTER).to(torch.float32) * float(value_scale(scale))
    del u
    if offset:
        v = v + float(np.float32(offset))
    if dtype == "f32":
        return v
    if dtype == "bf16":
        bits = v.view(torch.int32)
        lsb = (bits >> 16) & 1
        r = ((bits + 0x7FFF + lsb) >> 16) & 0xFFFF
        r = r - ((r >> 15) & 1) * 65536  # reinterpret as signed so the int16 cast is exact
        return r.to(torch.int16)  # same 16-bit pattern as the numpy uint16 result
    raise ValueError(f"unknown dtype {dtype!r}")
