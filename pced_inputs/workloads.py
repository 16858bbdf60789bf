"""Seeded synthetic PCED decode workloads (shapes and value distributions only).

Each workload describes one batch of queries. A query has N document experts and
one amateur (sequence 0 of the query, holding only the query tokens); every
sequence owns its own precomputed, ragged KV cache. Tensors are never stored in
a workload: they are *streams* of the counter generator in ``counter.py`` and are
materialised on demand, on the host (numpy / torch-CPU) or on the device
(torch), with identical bits.

Stream layout (element index = flat C-order index of the tensor shape given):

* ``kcache(s)`` / ``vcache(s)``: ``[L][len_s][Hkv][D]``, scale 1.0
* ``lm_head``: ``[V][hidden]``, scale 0.02
* ``q(t)``: ``[S][L][Hq][D]``, scale 1.0 (step t's query vectors)
* ``knew(t)`` / ``vnew(t)``: ``[S][L][Hkv][D]``, scale 1.0 (step t's new K/V row)

Small per-query quantities (cache lengths, retrieval scores, the page
permutation) come from numpy's PCG64 under ``SeedSequence(seed)``.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from . import counter

# stream tags (arbitrary distinct constants)
TAG_KCACHE, TAG_VCACHE, TAG_LMHEAD, TAG_Q, TAG_KNEW, TAG_VNEW = 11, 12, 13, 14, 15, 16


@dataclasses.dataclass(frozen=True)
class Geometry:
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    hidden: int
    vocab: int
    dtype: str  # 'bf16' | 'f32'

    @property
    def kv_bytes_per_token(self) -> int:
        """K and V bytes of one token over all layers."""
        esize = 2 if self.dtype == "bf16" else 4
        return 2 * self.n_layers * self.n_kv_heads * self.head_dim * esize


LLAMA3_8B = dict(n_q_heads=32, n_kv_heads=8, head_dim=128, hidden=4096, vocab=128256)


@dataclasses.dataclass
class Workload:
    name: str
    geom: Geometry
    seed: int
    n_experts: list          # per query
    cache_len: np.ndarray    # int32 [S], query-major, amateur first in each query
    relevance: np.ndarray    # float32 [sum N], retrieval scores in [0, 1]
    steps: int
    gamma: float = 2.5
    beta: Optional[np.ndarray] = None   # fixed per-expert beta, or None = dynamic
    page_size: int = 16
    shuffle_pages: bool = False

    # ---------------------------------------------------------------- layout
    @property
    def n_queries(self) -> int:
        return len(self.n_experts)

    @property
    def n_seqs(self) -> int:
        return int(sum(n + 1 for n in self.n_experts))

    @property
    def seq_offsets(self) -> np.ndarray:
        """First sequence (the amateur) of each query, plus the total."""
        return np.concatenate([[0], np.cumsum([n + 1 for n in self.n_experts])]).astype(np.int64)

    def pages_needed(self, extra_tokens: int) -> np.ndarray:
        """Pages per sequence to hold the cache plus ``extra_tokens`` appended tokens."""
        P = self.page_size
        return (self.cache_len.astype(np.int64) + extra_tokens + P - 1) // P

    def page_table(self, extra_tokens: int, max_pages_per_seq: int) -> np.ndarray:
        """[S][max_pages_per_seq] physical page ids (-1 unused).

        In order unless ``shuffle_pages``, in which case physical pages are a
        seeded random permutation of the pool, so logically adjacent pages of a
        sequence are scattered."""
        need = self.pages_needed(extra_tokens)
        total = int(need.sum())
        phys = np.arange(total, dtype=np.int64)
        if self.shuffle_pages:
            phys = _rng(self.seed, 4).permutation(total)
        pt = np.full((self.n_seqs, max_pages_per_seq), -1, dtype=np.int32)
        off = 0
        for s, n in enumerate(need):
            if n > max_pages_per_seq:
                raise ValueError("max_pages_per_seq too small for this workload")
            pt[s, :n] = phys[off:off + n]
            off += n
        return pt

    # ------------------------------------------------------------- streams
    def stream_key(self, tag: int, *fields: int) -> int:
        return counter.key(self.seed, tag, *fields)

    def cache_shape(self, s: int) -> tuple:
        g = self.geom
        return (g.n_layers, int(self.cache_len[s]), g.n_kv_heads, g.head_dim)

    def kcache_host(self, s: int, layer: Optional[int] = None) -> np.ndarray:
        return self._cache_host(TAG_KCACHE, s, layer)

    def vcache_host(self, s: int, layer: Optional[int] = None) -> np.ndarray:
        return self._cache_host(TAG_VCACHE, s, layer)

    def _cache_host(self, tag, s, layer):
        L, T, H, D = self.cache_shape(s)
        k = self.stream_key(tag, s)
        if layer is None:
            return host_values(k, 0, L * T * H * D, 1.0, self.geom.dtype).reshape(L, T, H, D)
        per = T * H * D
        return host_values(k, layer * per, per, 1.0, self.geom.dtype).reshape(T, H, D)

    def kcache_device(self, s: int, device):
        return self._cache_device(TAG_KCACHE, s, device)

    def vcache_device(self, s: int, device):
        return self._cache_device(TAG_VCACHE, s, device)

    def _cache_device(self, tag, s, device):
        L, T, H, D = self.cache_shape(s)
        k = self.stream_key(tag, s)
        return device_values(k, 0, L * T * H * D, 1.0, self.geom.dtype, device).reshape(L, T, H, D)

    def lm_head_host(self, rows: Optional[np.ndarray] = None) -> np.ndarray:
        """[V][hidden] (or only the listed vocab rows)."""
        g = self.geom
        k = self.stream_key(TAG_LMHEAD)
        if rows is None:
            return host_values(k, 0, g.vocab * g.hidden, 0.02, g.dtype).reshape(g.vocab, g.hidden)
        return np.stack([host_values(k, int(r) * g.hidden, g.hidden, 0.02, g.dtype) for r in rows])

    def lm_head_device(self, device):
        g = self.geom
        k = self.stream_key(TAG_LMHEAD)
        return device_values(k, 0, g.vocab * g.hidden, 0.02, g.dtype, device).reshape(g.vocab, g.hidden)

    def step_shapes(self):
        g = self.geom
        S = self.n_seqs
        return ((S, g.n_layers, g.n_q_heads, g.head_dim), (S, g.n_layers, g.n_kv_heads, g.head_dim))

    def step_inputs_host(self, t: int):
        """(q, k_new, v_new) of step t as stored values."""
        qs, ks = self.step_shapes()
        n_q, n_k = int(np.prod(qs)), int(np.prod(ks))
        dt = self.geom.dtype
        q = host_values(self.stream_key(TAG_Q, t), 0, n_q, 1.0, dt).reshape(qs)
        kn = host_values(self.stream_key(TAG_KNEW, t), 0, n_k, 1.0, dt).reshape(ks)
        vn = host_values(self.stream_key(TAG_VNEW, t), 0, n_k, 1.0, dt).reshape(ks)
        return q, kn, vn

    def step_inputs_device(self, t: int, device):
        qs, ks = self.step_shapes()
        n_q, n_k = int(np.prod(qs)), int(np.prod(ks))
        dt = self.geom.dtype
        q = device_values(self.stream_key(TAG_Q, t), 0, n_q, 1.0, dt, device).reshape(qs)
        kn = device_values(self.stream_key(TAG_KNEW, t), 0, n_k, 1.0, dt, device).reshape(ks)
        vn = device_values(self.stream_key(TAG_VNEW, t), 0, n_k, 1.0, dt, device).reshape(ks)
        return q, kn, vn


# -------------------------------------------------------------- materialise

_TORCH_HOST_THRESHOLD = 1 << 20
_CHUNK = 1 << 24


def host_values(k: int, start: int, count: int, scale: float, dtype: str, offset: float = 0.0) -> np.ndarray:
    """Host array of stored values (uint16 bf16 bits or float32)."""
    if count <= _TORCH_HOST_THRESHOLD:
        return counter.values_np(k, start, count, scale, dtype, offset)
    import torch  # multi-threaded CPU path, bit-identical to the numpy one

    out = np.empty(count, dtype=np.uint16 if dtype == "bf16" else np.float32)
    for c0 in range(0, count, _CHUNK):
        n = min(_CHUNK, count - c0)
        v = counter.values_torch(k, start + c0, n, scale, dtype, "cpu", offset).numpy()
        out[c0:c0 + n] = v.view(out.dtype)
    return out


def device_values(k: int, start: int, count: int, scale: float, dtype: str, device, offset: float = 0.0):
    """Device tensor of stored values: torch.int16 holding bf16 bits, or float32."""
    import torch

    out = torch.empty(count, dtype=torch.int16 if dtype == "bf16" else torch.float32, device=device)
    for c0 in range(0, count, _CHUNK):
        n = min(_CHUNK, count - c0)
        out[c0:c0 + n] = counter.values_torch(k, start + c0, n, scale, dtype, device, offset)
    return out


# ------------------------------------------------------------------ configs

def _rng(seed: int, *spawn: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=spawn)))


def _layout(n_experts, expert_lens, amateur_len):
    lens = []
    off = 0
    for n in n_experts:
        lens.append(amateur_len)
        lens.extend(int(x) for x in expert_lens[off:off + n])
        off += n
    return np.asarray(lens, dtype=np.int32)


def config1(seed: int = 0) -> Workload:
    """Tiny fp32: 1 layer, 4 q-heads / 2 kv-heads, head_dim 64, hidden 256, vocab 1000;
    N=4 experts with 128-token caches plus a 16-token query-only amateur; 8 steps;
    retrieval scores ~ U(0,1)."""
    g = Geometry(1, 4, 2, 64, 256, 1000, "f32")
    n = [4]
    r = _rng(seed, 1).random(4).astype(np.float32)
    return Workload("tiny-fp32", g, seed, n, _layout(n, [128] * 4, 16), r, steps=8)


def config2(seed: int = 0) -> Workload:
    """Llama-3-8B shapes, bf16, one layer, one step: N=8 experts of 2048 + 64 query
    tokens; 64-token amateur; retrieval scores ~ U(0,1)."""
    g = Geometry(1, **LLAMA3_8B, dtype="bf16")
    n = [8]
    r = _rng(seed, 1).random(8).astype(np.float32)
    return Workload("llama8b-n8-1layer", g, seed, n, _layout(n, [2048 + 64] * 8, 64), r, steps=1)


def config3(seed: int = 0) -> Workload:
    """Llama-3-8B shapes, bf16, 32 layers: N=32 experts with cache lengths
    ~ U{512..2048}; 64-token amateur; 128 generated tokens; scores ~ Beta(2,5)."""
    g = Geometry(32, **LLAMA3_8B, dtype="bf16")
    n = [32]
    lens = _rng(seed, 2).integers(512, 2048, size=32, endpoint=True)
    r = _rng(seed, 1).beta(2.0, 5.0, size=32).astype(np.float32)
    return Workload("llama8b-n32-32layer", g, seed, n, _layout(n, lens, 64), r, steps=128)


def config4(seed: int = 0) -> Workload:
    """Many-document shape, bf16, one layer: N=100 experts, lengths ~ U{256..1536};
    5 experts (seeded positions) score U[0.7,1], the other 95 score U[0,0.3]."""
    g = Geometry(1, **LLAMA3_8B, dtype="bf16")
    n = [100]
    lens = _rng(seed, 2).integers(256, 1536, size=100, endpoint=True)
    rg = _rng(seed, 1)
    r = rg.uniform(0.0, 0.3, size=100)
    hi = rg.choice(100, size=5, replace=False)
    r[hi] = rg.uniform(0.7, 1.0, size=5)
    return Workload("llama8b-n100-1layer", g, seed, n, _layout(n, lens, 64), r.astype(np.float32), steps=1)


def config5(seed: int = 0) -> Workload:
    """Concurrent queries, bf16, one layer: 16 queries x (16 experts with lengths
    ~ U{256..4096} + 64-token amateur), 16-token pages in one pool assigned by a
    seeded permutation; per-query scores ~ U(0,1); 64 decode steps."""
    g = Geometry(1, **LLAMA3_8B, dtype="bf16")
    n = [16] * 16
    lens = _rng(seed, 2).integers(256, 4096, size=256, endpoint=True)
    r = _rng(seed, 1).random(256).astype(np.float32)
    return Workload("llama8b-16q-n16-paged", g, seed, n, _layout(n, lens, 64), r, steps=64,
                    shuffle_pages=True)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


def custom(geom: Geometry, n_experts, expert_lens, amateur_len, steps, seed=0, relevance=None,
           beta=None, gamma=2.5, shuffle_pages=False, name="custom") -> Workload:
    """A workload of arbitrary shape (tests: small tiles, ragged tails, edge cases)."""
    n_total = int(sum(n_experts))
    if relevance is None:
        relevance = _rng(seed, 1).random(n_total).astype(np.float32)
    return Workload(name, geom, seed, list(n_experts), _layout(n_experts, expert_lens, amateur_len),
                    np.asarray(relevance, dtype=np.float32), steps=steps, gamma=gamma,
                    beta=None if beta is None else np.asarray(beta, dtype=np.float32),
                    shuffle_pages=shuffle_pages)
