"""Seeded random-init weights of a Llama-3-style decoder stack (shapes and value
distributions only) and seeded token streams for the query suffix.

Like ``workloads.py`` this module materialises counter-generator streams and
holds none of the decoding method's arithmetic. Every tensor is a stream of
``counter.py`` keyed by (seed, tag, layer); element i is the i-th element of the
tensor in C order:

* ``embed``: ``[V][hidden]``, scale 1.0
* ``final_norm``, ``attn_norm[l]``, ``mlp_norm[l]``: ``[hidden]``, 1 + values of scale 0.1
* ``wq[l]``: ``[Hq*D][hidden]``, ``wk[l]`` / ``wv[l]``: ``[Hkv*D][hidden]``,
  ``wo[l]``: ``[hidden][Hq*D]``, ``w_gate[l]`` / ``w_up[l]``: ``[F][hidden]``,
  ``w_down[l]``: ``[hidden][F]``; scale 0.02 (the usual initialiser width)

All are stored as bf16 bit patterns (the model path computes in bf16 with fp32
accumulation).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from . import counter
from .workloads import Geometry, device_values, host_values

TAGS = {"embed": 21, "final_norm": 22, "attn_norm": 23, "wq": 24, "wk": 25, "wv": 26, "wo": 27,
        "mlp_norm": 28, "w_gate": 29, "w_up": 30, "w_down": 31}
TAG_SUFFIX = 32
LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")
PROJ_SCALE, EMBED_SCALE, NORM_JITTER = 0.02, 1.0, 0.1


@dataclasses.dataclass(frozen=True)
class ModelSpec:
    geom: Geometry
    ffn_dim: int
    rope_theta: float = 500000.0
    seed: int = 0

    def shape(self, name: str) -> tuple:
        g = self.geom
        H, qd, kd, F = g.hidden, g.n_q_heads * g.head_dim, g.n_kv_heads * g.head_dim, self.ffn_dim
        return {"embed": (g.vocab, H), "final_norm": (H,), "attn_norm": (H,), "mlp_norm": (H,),
                "wq": (qd, H), "wk": (kd, H), "wv": (kd, H), "wo": (H, qd),
                "w_gate": (F, H), "w_up": (F, H), "w_down": (H, F)}[name]

    def _params(self, name: str):
        if name.endswith("norm"):
            return NORM_JITTER, 1.0
        return (EMBED_SCALE if name == "embed" else PROJ_SCALE), 0.0

    def _key(self, name: str, layer: int) -> int:
        return counter.key(self.seed, TAGS[name], layer)

    def host(self, name: str, layer: int = 0, rows: Optional[np.ndarray] = None) -> np.ndarray:
        """Stored bf16 bits of one tensor (or of the listed rows of a matrix)."""
        shp = self.shape(name)
        scale, off = self._params(name)
        k = self._key(name, layer)
        if rows is None:
            return host_values(k, 0, int(np.prod(shp)), scale, "bf16", off).reshape(shp)
        n = shp[1]
        return np.stack([host_values(k, int(r) * n, n, scale, "bf16", off) for r in rows])

    def device(self, name: str, layer: int, device):
        shp = self.shape(name)
        scale, off = self._params(name)
        return device_values(self._key(name, layer), 0, int(np.prod(shp)), scale, "bf16", device,
                             off).reshape(shp)


def suffix_tokens(seed: int, n_queries: int, n_tokens: int, vocab: int) -> np.ndarray:
    """[B][n_tokens] int32 query-suffix token ids, uniform over the vocabulary."""
    h = counter.hashes_np(counter.key(seed, TAG_SUFFIX), 0, n_queries * n_tokens)
    return (h % np.uint64(vocab)).astype(np.int32).reshape(n_queries, n_tokens)
