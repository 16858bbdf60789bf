"""Plain CPU oracle for the decoder layers around the PCED decode step: the
batched forward pass of the N+1 experts that produces each step's queries, new
K/V rows and final hidden states (paper, Section 3: the experts run in one
batched forward pass, the query is processed into every expert's cache, and the
chosen token joins every expert's history).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or execute
this module; only the tests and the benchmark's CPU baseline use it. NumPy
float64, the plain definitions, contiguous caches, one token at a time.

The paper does not restate the language model. Readings used (a Llama-3-style
decoder, the shape of the 8B model the workloads use):

* h = E[y] (the token's embedding row), then per layer
      a = RMSNorm(h) * g_attn;  q, k, v = a Wq^T, a Wk^T, a Wv^T
      q, k <- RoPE(q, pos), RoPE(k, pos);  (k, v) appended to the layer's cache
      h <- h + Attn(q, K, V) Wo^T
      b = RMSNorm(h) * g_mlp;  h <- h + (silu(b Wg^T) * (b Wu^T)) Wd^T
  and the logits are RMSNorm(h) * g_final W_lm^T.
* RMSNorm(h) = h / sqrt(mean(h^2) + 1e-5).
* RoPE rotates the pairs (x[2i], x[2i+1]) of every head by the angle
  pos * theta^(-2i/D) (the original complex-pair form; it differs from the
  half-split form only by a fixed permutation of the q/k weight rows).
* Positions: every expert's cache was encoded from position 0, so the token
  appended to sequence s sits at position len_s, its own cache length before the
  append (each expert, and the amateur, has its own positions).
* Grouped-query attention as in the decode step: q-head h reads kv-head
  h // (Hq / Hkv), scale 1/sqrt(D).

Precision contract (bf16 weights; the GPU computes in fp32 with bf16 operands):
* the residual stream h is kept unrounded (float64 here, fp32 there);
* a normalised product is rho * (bf16(h * g) W^T) with rho = 1/sqrt(mean(h^2) + eps)
  taken from the unrounded h: the element-wise product h * g is rounded to bf16
  and the row scale applied to the product (equal to RMSNorm(h) * g W^T in exact
  arithmetic);
* q, k, v are rounded to bf16 after RoPE (the stored cache rows and the
  attention's query); the attention output is rounded to bf16 before Wo; the
  MLP activation silu(gate) * up is rounded to bf16 before Wd.
"""
from __future__ import annotations

from typing import Callable, Optional, Sequence

import numpy as np

from .pced_oracle import (RMS_EPS, StepResult, attention, decode_stored, dynamic_beta, fuse_query,
                          round_to_bf16)


def rope(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate the pairs (x[..., 2i], x[..., 2i+1]) by pos * theta^(-2i/D)."""
    D = x.shape[-1]
    i = np.arange(D // 2, dtype=np.float64)
    ang = float(pos) * np.power(float(theta), -2.0 * i / D)
    c, s = np.cos(ang), np.sin(ang)
    x0, x1 = x[..., 0::2], x[..., 1::2]
    out = np.empty(x.shape, dtype=np.float64)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


def rms_rho(h: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    """1/sqrt(mean(h^2) + eps) per row."""
    return 1.0 / np.sqrt(np.mean(np.square(h), axis=-1) + eps)


def normed_product(h: np.ndarray, g: np.ndarray, W: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    """RMSNorm(h) * g W^T under the precision contract: rho * (bf16(h * g) W^T)."""
    a = round_to_bf16(h * g[None, :])
    return rms_rho(h, eps)[:, None] * (a @ W.T)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


class ModelOracle:
    """Stateful multi-step PCED decoding with the decoder stack producing each
    step's q / k / v from the shared token (one token at a time).

    ``weights(name, layer)`` returns a layer tensor as stored bf16 bits (names:
    attn_norm, wq, wk, wv, wo, mlp_norm, w_gate, w_up, w_down); ``embed(rows)``
    the listed embedding rows; ``final_norm`` and ``lm_head`` stored bits.
    ``cache_k(s, l)`` / ``cache_v(s, l)`` are the preloaded caches [T, Hkv, D].
    """

    def __init__(self, *, n_layers, n_q_heads, n_kv_heads, head_dim, vocab, rope_theta,
                 n_experts: Sequence[int], cache_k: Callable, cache_v: Callable, weights: Callable,
                 embed: Callable, final_norm, lm_head, relevance, gamma: float = 2.5, beta=None,
                 aggregation: str = "max", beta_scalar: bool = False):
        self.L, self.Hq, self.Hkv, self.D, self.V = n_layers, n_q_heads, n_kv_heads, head_dim, vocab
        self.theta = float(rope_theta)
        self.n_experts = list(n_experts)
        self.seq_off = np.concatenate([[0], np.cumsum([n + 1 for n in self.n_experts])]).astype(int)
        self.S = int(self.seq_off[-1])
        self.seq_query = np.repeat(np.arange(len(self.n_experts)), [n + 1 for n in self.n_experts])
        self._weights, self._embed = weights, embed
        self.final_norm = decode_stored(final_norm, "bf16")
        self.lm_head = lm_head if lm_head.dtype == np.float64 else decode_stored(lm_head, "bf16")
        self.relevance = np.asarray(relevance, dtype=np.float64)
        self.gamma = float(gamma)
        self.fixed_beta = None if beta is None else np.asarray(beta, dtype=np.float64)
        self.frozen_beta = None
        self.aggregation, self.beta_scalar = aggregation, bool(beta_scalar)
        # contiguous caches per (sequence, layer), stored values decoded
        self.K = [[decode_stored(cache_k(s, l), "bf16") for l in range(self.L)] for s in range(self.S)]
        self.Vc = [[decode_stored(cache_v(s, l), "bf16") for l in range(self.L)] for s in range(self.S)]
        self._wcache = {}

    def weight(self, name: str, l: int) -> np.ndarray:
        key = (name, l)
        if key not in self._wcache:
            self._wcache[key] = decode_stored(self._weights(name, l), "bf16")
        return self._wcache[key]

    def lengths(self):
        return [self.K[s][0].shape[0] for s in range(self.S)]

    # ---- the stages of one decoder layer (each takes its inputs explicitly, so a
    # test can feed any stage the values another implementation produced)

    def qkv(self, l: int, h: np.ndarray, positions) -> tuple:
        """Layer l's q [S, Hq, D], k, v [S, Hkv, D] for residual rows h at the given
        positions: normalised products, RoPE on q and k, all rounded to bf16."""
        S, Hq, Hkv, D = h.shape[0], self.Hq, self.Hkv, self.D
        g = self.weight("attn_norm", l)
        q = normed_product(h, g, self.weight("wq", l)).reshape(S, Hq, D)
        k = normed_product(h, g, self.weight("wk", l)).reshape(S, Hkv, D)
        v = normed_product(h, g, self.weight("wv", l)).reshape(S, Hkv, D)
        qs = np.empty_like(q)
        ks = np.empty_like(k)
        for s in range(S):
            qs[s] = round_to_bf16(rope(q[s], positions[s], self.theta))
            ks[s] = round_to_bf16(rope(k[s], positions[s], self.theta))
        return qs, ks, round_to_bf16(v)

    def o_residual(self, l: int, h: np.ndarray, o: np.ndarray) -> np.ndarray:
        """h + bf16(o) Wo^T for the attention output o [S, Hq*D] (or [S, Hq, D])."""
        return h + round_to_bf16(o.reshape(h.shape[0], self.Hq * self.D)) @ self.weight("wo", l).T

    def mlp_act(self, l: int, h: np.ndarray) -> np.ndarray:
        """bf16(silu(b Wg^T) * (b Wu^T)) with b the MLP norm's product of h."""
        g = self.weight("mlp_norm", l)
        gate = normed_product(h, g, self.weight("w_gate", l))
        up = normed_product(h, g, self.weight("w_up", l))
        return round_to_bf16(silu(gate) * up)

    def down_residual(self, l: int, h: np.ndarray, act: np.ndarray) -> np.ndarray:
        """h + act Wd^T."""
        return h + act @ self.weight("w_down", l).T

    def logits_of(self, h: np.ndarray) -> np.ndarray:
        """Final norm and LM head: RMSNorm(h) g_final W_lm^T."""
        return normed_product(h, self.final_norm, self.lm_head)

    def append_rows(self, l: int, k: np.ndarray, v: np.ndarray):
        """Append one K/V row per sequence (decoded values [S, Hkv, D]) to layer l."""
        for s in range(self.S):
            self.K[s][l] = np.concatenate([self.K[s][l], k[s][None]], axis=0)
            self.Vc[s][l] = np.concatenate([self.Vc[s][l], v[s][None]], axis=0)

    def attend(self, l: int, q: np.ndarray) -> np.ndarray:
        """Every sequence's attention over its layer-l cache: [S, Hq, D]."""
        return np.stack([attention(q[s], self.K[s][l], self.Vc[s][l]) for s in range(self.S)])

    def layer(self, l: int, h: np.ndarray, kv_rows: Optional[Callable] = None):
        """One decoder layer for the new token of every sequence; appends its K/V
        rows. ``kv_rows(l)``, if given, returns the rows [S, Hkv, D] to append in
        place of the layer's own (a cache taught by another implementation).
        Returns (h after the layer, attention output [S, Hq, D], own (q, k, v))."""
        pos = [self.K[s][l].shape[0] for s in range(self.S)]
        q, k, v = self.qkv(l, h, pos)
        ka, va = (k, v) if kv_rows is None else kv_rows(l)
        self.append_rows(l, ka, va)
        o = self.attend(l, q)
        h = self.o_residual(l, h, o)
        h = self.down_residual(l, h, self.mlp_act(l, h))
        return h, o, (q, k, v)

    def forward(self, in_tokens: np.ndarray, kv_rows: Optional[Callable] = None):
        """Embed each query's token into all its sequences and run every layer.
        Returns (final residual stream h [S, hidden], {layer: attention output},
        {layer: own (q, k, v)})."""
        toks = np.asarray(in_tokens)[self.seq_query]
        h = decode_stored(self._embed(toks), "bf16")
        attn, own = {}, {}
        for l in range(self.L):
            h, attn[l], own[l] = self.layer(l, h, kv_rows)
        return h, attn, own

    def prefill(self, tokens: np.ndarray, kv_rows: Optional[Callable] = None):
        """Append the query-suffix tokens [B][n] to every sequence of each query,
        one token at a time (causal by construction); no logits. ``kv_rows(i, l)``
        optionally supplies suffix token i's rows at layer l (see ``layer``).
        Returns {(i, l): own (q, k, v)}."""
        tokens = np.asarray(tokens)
        own = {}
        for i in range(tokens.shape[1]):
            rows = None if kv_rows is None else (lambda l, i=i: kv_rows(i, l))
            _, _, o = self.forward(tokens[:, i], rows)
            for l, x in o.items():
                own[(i, l)] = x
        return own

    def select(self, logits: np.ndarray) -> StepResult:
        """Dynamic beta at the first call (frozen afterwards) and Eq. 2 / Eq. 3 per
        query over the logits of every sequence."""
        if self.fixed_beta is not None:
            beta = self.fixed_beta
        else:
            if self.frozen_beta is None:
                self.frozen_beta = np.concatenate([
                    dynamic_beta(logits[self.seq_off[b]:self.seq_off[b + 1]], self.beta_scalar)
                    for b in range(len(self.n_experts))])
            beta = self.frozen_beta
        sels = []
        e0 = 0
        for b, n in enumerate(self.n_experts):
            rows = logits[self.seq_off[b]:self.seq_off[b + 1]]
            sels.append(fuse_query(rows, self.relevance[e0:e0 + n], self.gamma, beta[e0:e0 + n],
                                   rule=self.aggregation))
            e0 += n
        return StepResult(
            tokens=np.array([x.token for x in sels]), winners=np.array([x.winner for x in sels]),
            top1=np.array([x.top1 for x in sels]), top2=np.array([x.top2 for x in sels]),
            beta=np.array(beta, copy=True), logits=logits, hidden=None, attn={})

    def step(self, in_tokens: np.ndarray) -> StepResult:
        """One decode step: append the queries' previous tokens, logits of every
        sequence, dynamic beta at the first step, Eq. 2 / Eq. 3 per query."""
        h, attn, _ = self.forward(in_tokens)
        r = self.select(self.logits_of(h))
        r.hidden, r.attn = h, attn
        return r


def causal_block_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, n_new: int) -> np.ndarray:
    """Attention of the last ``n_new`` positions of K/V, all at once, with a causal
    mask: query i (0-based among the new ones) sees the T - n_new cached rows and
    new rows 0..i. Q: [n_new, Hq, D]; K, V: [T, Hkv, D]. The matrix form of a
    multi-token prefill, used to pin the one-token-at-a-time path."""
    T = K.shape[0]
    nq, Hq, D = Q.shape
    G = Hq // K.shape[1]
    out = np.empty((nq, Hq, D))
    for h in range(Hq):
        Kh, Vh = K[:, h // G, :], V[:, h // G, :]
        z = Q[:, h, :] @ Kh.T / np.sqrt(D)                       # [nq, T]
        mask = np.arange(T)[None, :] > (T - n_new + np.arange(nq))[:, None]
        z = np.where(mask, -np.inf, z)
        z = z - z.max(axis=1, keepdims=True)
        p = np.exp(z)
        p /= p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ Vh
    return out
