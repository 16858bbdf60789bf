"""Convenience layer over the C ABI: allocates the caller-owned device buffers
(KV pools, workspace, outputs) with torch and forwards every call to libpced.

Nothing here computes any part of the decode step.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from . import _lib


def _torch():
    import torch
    return torch


class PcedSession:
    """A context plus its two KV pools for one model geometry and capacity."""

    def __init__(self, *, n_layers, n_q_heads, n_kv_heads, head_dim, vocab, dtype, max_queries,
                 max_seqs, max_pages, max_pages_per_seq, norm="rms", device="cuda", poison=False,
                 max_attn_chunks=0, aggregation="max", beta_scalar=False, ffn_dim=0, rope_theta=500000):
        torch = _torch()
        self.dtype = dtype
        self.device = device
        self.geom = dict(n_layers=n_layers, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads,
                         head_dim=head_dim, vocab=vocab)
        self.ffn_dim = ffn_dim
        self.cfg = _lib.make_config(n_layers=n_layers, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads,
                                    head_dim=head_dim, vocab=vocab, dtype=dtype, max_queries=max_queries,
                                    max_seqs=max_seqs, max_pages=max_pages,
                                    max_pages_per_seq=max_pages_per_seq, norm=norm,
                                    max_attn_chunks=max_attn_chunks, aggregation=aggregation,
                                    beta_scalar=beta_scalar, ffn_dim=ffn_dim, rope_theta=rope_theta)
        self.ctx = _lib.Context(self.cfg, device=device)
        pool = _lib.pced_pool_bytes(self.cfg)
        self.k_pool = torch.empty(pool, dtype=torch.uint8, device=device)
        self.v_pool = torch.empty(pool, dtype=torch.uint8, device=device)
        if poison:  # all-ones bytes: NaN in bf16 and f32, to expose reads of unwritten memory
            for t in (self.k_pool, self.v_pool, self.ctx.workspace):
                t.fill_(255)
        self.n_experts: list = []
        self.S = 0
        self.B = 0
        self.NE = 0

    def pack_lm_head(self, w):
        """Packed copy (device) of row-major [V][hidden] LM-head weights."""
        torch = _torch()
        out = torch.empty(_lib.pced_lm_head_bytes(self.cfg), dtype=torch.uint8, device=self.device)
        _lib.pced_pack_lm_head(self.cfg, w, out)
        return out

    def pack_model(self, layer_tensors, embed, final_norm):
        """Packed decoder-stack weights (device). ``layer_tensors(l)`` returns the 9
        bf16 device tensors of layer l in pced_pack_model_layer order."""
        torch = _torch()
        out = torch.empty(_lib.pced_model_bytes(self.cfg), dtype=torch.uint8, device=self.device)
        for l in range(self.geom["n_layers"]):
            ts = layer_tensors(l)
            _lib.pced_pack_model_layer(self.cfg, l, ts, out)
            torch.cuda.current_stream().synchronize()  # the sources may be dropped after the copy
            del ts
        _lib.pced_pack_model_globals(self.cfg, embed, final_norm, out)
        torch.cuda.current_stream().synchronize()
        return out

    def model_step(self, model, lm_head, in_tokens, want=("logits", "winner", "top1", "top2", "beta_used")):
        torch = _torch()
        tokens = torch.empty(self.B, dtype=torch.int32, device=self.device)
        extra = self.out_buffers(want) if want else None
        self.ctx.pced_model_step(model, lm_head, in_tokens, tokens, extra)
        out = dict(extra or {})
        out["tokens"] = tokens
        return out

    # ------------------------------------------------------------------ load
    def load(self, n_experts: Sequence[int], cache_len: Sequence[int], src_k, src_v, relevance,
             gamma=2.5, beta=None, page_table=None, reserve_tokens=0):
        self.n_experts = list(n_experts)
        self.B = len(self.n_experts)
        self.S = int(sum(n + 1 for n in self.n_experts))
        self.NE = int(sum(self.n_experts))
        self.ctx.pced_load_caches(n_experts, cache_len, src_k, src_v, self.k_pool, self.v_pool, relevance,
                                  gamma=gamma, beta=beta, page_table=page_table,
                                  reserve_tokens=reserve_tokens)

    # ----------------------------------------------------------------- steps
    def out_buffers(self, want=("logits", "winner", "top1", "top2", "beta_used")):
        torch = _torch()
        g = self.geom
        f32, i32 = torch.float32, torch.int32
        shapes = {
            "attn_out": ((self.S, g["n_layers"], g["n_q_heads"], g["head_dim"]), f32),
            "logits": ((self.S, g["vocab"]), f32),
            "winner": ((self.B,), i32),
            "top1": ((self.B,), f32),
            "top2": ((self.B,), f32),
            "beta_used": ((self.NE,), f32),
            "hidden": ((self.S, g["n_q_heads"] * g["head_dim"]), f32),
        }
        if self.ffn_dim:
            L, H, D = g["n_layers"], g["n_q_heads"] * g["head_dim"], g["head_dim"]
            qkv = (g["n_q_heads"] + 2 * g["n_kv_heads"]) * D
            shapes["resid_trace"] = ((L, 2, self.S, H), f32)
            shapes["qkv_trace"] = ((L, self.S, qkv), torch.int16)
            shapes["act_trace"] = ((L, self.S, self.ffn_dim), torch.int16)
        return {k: torch.empty(shapes[k][0], dtype=shapes[k][1], device=self.device) for k in want}

    def step(self, q, k_new, v_new, lm_head, want=("logits", "winner", "top1", "top2", "beta_used")):
        torch = _torch()
        tokens = torch.empty(self.B, dtype=torch.int32, device=self.device)
        extra = self.out_buffers(want) if want else None
        self.ctx.pced_step(q, k_new, v_new, lm_head, tokens, extra)
        out = dict(extra or {})
        out["tokens"] = tokens
        return out

    def generate(self, n_steps, seed, first_token, lm_head, want=()):
        torch = _torch()
        tokens = torch.empty((self.B, n_steps), dtype=torch.int32, device=self.device)
        extra = self.out_buffers(want) if want else None
        self.ctx.pced_generate(n_steps, seed, first_token, lm_head, tokens, extra)
        out = dict(extra or {})
        out["tokens"] = tokens
        return out

    def lengths(self):
        return self.ctx.pced_get_lengths(self.S)

    def read_cache(self, seq, layer, start, count):
        """(k, v) rows [count][Hkv][D] of one sequence and layer, read out of the
        pool (int16 bf16 bits or float32), on the session's device."""
        torch = _torch()
        g = self.geom
        dt = torch.int16 if self.dtype == "bf16" else torch.float32
        k = torch.empty((count, g["n_kv_heads"], g["head_dim"]), dtype=dt, device=self.device)
        v = torch.empty_like(k)
        self.ctx.pced_read_cache(seq, layer, start, count, k, v)
        return k, v


def session_for_workload(wl, device="cuda", extra_tokens: Optional[int] = None, norm="rms",
                         load_now=True, max_queries=None, poison=False, max_attn_chunks=0, aggregation="max",
                         beta_scalar=False, ffn_dim=0, rope_theta=500000):
    """Build a session sized for a synthetic workload (duck-typed: any object with
    the attributes of ``pced_inputs.workloads.Workload``) and load its caches,
    materialised on ``device``."""
    g = wl.geom
    extra = wl.steps if extra_tokens is None else extra_tokens
    need = wl.pages_needed(extra)
    maxpps = int(need.max())
    sess = PcedSession(n_layers=g.n_layers, n_q_heads=g.n_q_heads, n_kv_heads=g.n_kv_heads,
                       head_dim=g.head_dim, vocab=g.vocab, dtype=g.dtype,
                       max_queries=max_queries or wl.n_queries, max_seqs=wl.n_seqs,
                       max_pages=int(need.sum()), max_pages_per_seq=maxpps, norm=norm, device=device,
                       poison=poison, max_attn_chunks=max_attn_chunks, aggregation=aggregation,
                       beta_scalar=beta_scalar, ffn_dim=ffn_dim, rope_theta=rope_theta)
    sess.workload_page_table = wl.page_table(extra, maxpps)
    if load_now:
        load_workload(sess, wl)
    return sess


def load_workload(sess: PcedSession, wl, src=None):
    """(Re)load the workload's caches into the session; ``src`` optionally reuses
    already materialised (k, v) device tensors."""
    torch = _torch()
    if src is None:
        src_k = [wl.kcache_device(s, sess.device) for s in range(wl.n_seqs)]
        src_v = [wl.vcache_device(s, sess.device) for s in range(wl.n_seqs)]
    else:
        src_k, src_v = src
    sess.load(wl.n_experts, wl.cache_len.tolist(), src_k, src_v, wl.relevance.tolist(), gamma=wl.gamma,
              beta=None if wl.beta is None else np.asarray(wl.beta).tolist(),
              page_table=sess.workload_page_table)
    torch.cuda.current_stream().synchronize()
    return src_k, src_v
