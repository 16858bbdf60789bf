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

    def layer(self, l: int, h: np.ndarray):
        """One decoder layer for the new token of every sequence; appends its K/V
        rows. Returns (h after the layer, attention output [S, Hq, D])."""
        S, Hq, Hkv, D = self.S, self.Hq, self.Hkv, self.D
        w = lambda n: self.weight(n, l)  # noqa: E731
        g_attn, g_mlp = w("attn_norm"), w("mlp_norm")
        q = normed_product(h, g_attn, w("wq")).reshape(S, Hq, D)
        k = normed_product(h, g_attn, w("wk")).reshape(S, Hkv, D)
        v = normed_product(h, g_attn, w("wv")).reshape(S, Hkv, D)
        o = np.empty((S, Hq, D))
        for s in range(S):
            pos = self.K[s][l].shape[0]
            qs = round_to_bf16(rope(q[s], pos, self.theta))
            ks = round_to_bf16(rope(k[s], pos, self.theta))
            vs = round_to_bf16(v[s])
            self.K[s][l] = np.concatenate([self.K[s][l], ks[None]], axis=0)
            self.Vc[s][l] = np.concatenate([self.Vc[s][l], vs[None]], axis=0)
            o[s] = attention(qs, self.K[s][l], self.Vc[s][l])
        h = h + round_to_bf16(o.reshape(S, Hq * D)) @ w("wo").T
        gate = normed_product(h, g_mlp, w("w_gate"))
        up = normed_product(h, g_mlp, w("w_up"))
        act = round_to_bf16(silu(gate) * up)
        h = h + act @ w("w_down").T
        return h, o

    def forward(self, in_tokens: np.ndarray):
        """Embed each query's token into all its sequences and run every layer.
        Returns (final residual stream h [S, hidden], {layer: attention output})."""
        toks = np.asarray(in_tokens)[self.seq_query]
        h = decode_stored(self._embed(toks), "bf16")
        attn = {}
        for l in range(self.L):
            h, attn[l] = self.layer(l, h)
        return h, attn

    def prefill(self, tokens: np.ndarray):
        """Append the query-suffix tokens [B][n] to every sequence of each query,
        one token at a time (causal by construction); no logits."""
        tokens = np.asarray(tokens)
        for i in range(tokens.shape[1]):
            self.forward(tokens[:, i])

    def step(self, in_tokens: np.ndarray) -> StepResult:
        """One decode step: append the queries' previous tokens, logits of every
        sequence, dynamic beta at the first step, Eq. 2 / Eq. 3 per query."""
        h, attn = self.forward(in_tokens)
        logits = normed_product(h, self.final_norm, self.lm_head)
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
            beta=np.array(beta, copy=True), logits=logits, hidden=h, attn=attn)


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
