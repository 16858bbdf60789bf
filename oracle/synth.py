"""The oracle's own implementation of the synthetic model stand-in used by multi-step
generation.

TEST INFRASTRUCTURE ONLY (see ``pced_oracle``).

In a real deployment the query vector and the new K/V row of step t come out of
the model's projections applied to the previous token. Here they are drawn from
a counter-based generator keyed by that token, so a run is fully determined by
(seed, first token) and the chosen tokens feed back into the inputs exactly as
in autoregressive decoding.

Definition (SplitMix64, Steele, Lea and Flood, OOPSLA 2014):
  G = 0x9E3779B97F4A7C15
  mix(z): z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
          z *= 0x94D049BB133111EB; z ^= z >> 31          (all mod 2**64)
  fold(seed, f1, ..., fn): k = seed; for each f: k = mix((k ^ f) + G)
  out(k, i) = mix(k + (i + 1) * G)
  value(k, i) = float32(U - 131070) * float32(sqrt(3) / 65536), where U is the sum
      of the four 16-bit fields of out(k, i); rounded to nearest-even bf16 when
      the storage type is bf16.
For step t, sequence s (global index), layer l and the query's previous token y
(the given first token at t = 0):
  q[s, l]     = value(fold(seed, 0x51, t, s, l, y), i), i < Hq * D
  k_new[s, l] = value(fold(seed, 0x4B, t, s, l, y), i), i < Hkv * D
  v_new[s, l] = value(fold(seed, 0x56, t, s, l, y), i), i < Hkv * D
"""
from __future__ import annotations

import math

import numpy as np

_M = (1 << 64) - 1
_G = 0x9E3779B97F4A7C15
TAG_Q, TAG_K, TAG_V = 0x51, 0x4B, 0x56


def _mix(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M
    return z ^ (z >> 31)


def fold(seed: int, *fields: int) -> int:
    k = seed & _M
    for f in fields:
        k = _mix(((k ^ (f & _M)) + _G) & _M)
    return k


def stream_values(k: int, n: int, dtype: str) -> np.ndarray:
    """n stored values of stream k: uint16 bf16 bits or float32."""
    outs = []
    for i in range(n):
        h = _mix((k + (i + 1) * _G) & _M)
        u = (h & 0xFFFF) + ((h >> 16) & 0xFFFF) + ((h >> 32) & 0xFFFF) + (h >> 48)
        outs.append(u - 131070)
    vals = np.array(outs, dtype=np.float32) * np.float32(math.sqrt(3.0) / 65536.0)
    if dtype == "f32":
        return vals
    bits = vals.view(np.uint32).astype(np.uint64)
    rounded = (bits + 0x7FFF + ((bits >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def step_inputs(seed, t, prev_tokens, n_experts, n_layers, n_q_heads, n_kv_heads, head_dim, dtype):
    """(q [S,L,Hq,D], k_new [S,L,Hkv,D], v_new [S,L,Hkv,D]) for step t."""
    S = sum(n + 1 for n in n_experts)
    store = np.uint16 if dtype == "bf16" else np.float32
    q = np.empty((S, n_layers, n_q_heads * head_dim), dtype=store)
    kn = np.empty((S, n_layers, n_kv_heads * head_dim), dtype=store)
    vn = np.empty_like(kn)
    s = 0
    for b, n in enumerate(n_experts):
        y = int(prev_tokens[b])
        for _ in range(n + 1):
            for l in range(n_layers):
                q[s, l] = stream_values(fold(seed, TAG_Q, t, s, l, y), n_q_heads * head_dim, dtype)
                kn[s, l] = stream_values(fold(seed, TAG_K, t, s, l, y), n_kv_heads * head_dim, dtype)
                vn[s, l] = stream_values(fold(seed, TAG_V, t, s, l, y), n_kv_heads * head_dim, dtype)
            s += 1
    return (q.reshape(S, n_layers, n_q_heads, head_dim),
            kn.reshape(S, n_layers, n_kv_heads, head_dim),
            vn.reshape(S, n_layers, n_kv_heads, head_dim))
