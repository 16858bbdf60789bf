"""Glue between the synthetic workloads, the GPU path (through the C ABI) and the
CPU oracle, for the parity tests. Inputs come only from ``pced_inputs``; no
expected value comes from the GPU path."""
from __future__ import annotations

import functools

import numpy as np

from oracle import pced_oracle as O
from pced_inputs import workloads as W

# tolerances of the parity contract: per-row max-abs error relative to the
# row's max-abs reference value
REL_TOL = {"bf16": 2e-2, "f32": 1e-5}
GAP_EXEMPT = 1e-3


def rel_err_rows(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, dtype=np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    den = np.abs(ref).max(axis=1)
    den[den == 0] = 1.0
    return float((np.abs(got - ref).max(axis=1) / den).max())


@functools.lru_cache(maxsize=2)
def lm_head_host(seed: int, vocab: int, hidden: int, dtype: str) -> np.ndarray:
    """Decoded float64 LM head of a workload (shared by every config with this
    seed and shape, so it is generated once per test session)."""
    wl = W.custom(W.Geometry(1, 1, 1, hidden, hidden, vocab, dtype), [1], [1], 1, 1, seed=seed)
    return O.decode_stored(wl.lm_head_host(), dtype)


def make_oracle(wl: W.Workload, layers=None, seqs=None, norm="rms") -> O.Oracle:
    """Oracle over the workload's caches, generated lazily per (sequence, layer)."""
    g = wl.geom
    cache = {}

    def get(kind, s, l):
        key = (kind, s, l)
        if key not in cache:
            cache[key] = (wl.kcache_host if kind == "k" else wl.vcache_host)(s, l)
        return cache[key]

    return O.Oracle(n_layers=g.n_layers, n_q_heads=g.n_q_heads, n_kv_heads=g.n_kv_heads,
                    head_dim=g.head_dim, vocab=g.vocab, dtype=g.dtype, n_experts=wl.n_experts,
                    cache_k=lambda s, l: get("k", s, l), cache_v=lambda s, l: get("v", s, l),
                    relevance=wl.relevance, gamma=wl.gamma, beta=wl.beta, norm=norm)


def beta_tol(logits, ref_logits, wl) -> np.ndarray:
    """Per-expert bound on |beta_gpu - beta_ref| from the logits' errors. beta_k =
    JSD(softmax s_k || softmax s_0) in bits; the gradient of the JSD with respect
    to either logit row has L1 norm at most sum_v p(v) |log2(p(v)/m(v))| <=
    1 + 1/(e ln 2) < 1.6 (p/m <= 2 above the mixture m; x log2(1/x) <= 1/(e ln 2)
    below it), so to first order |d beta_k| <= 1.6 (e_k + e_0), e_r = max_v
    |d s_r(v)|. Floor 1e-4 for the fp32 sums over the vocabulary. ``wl``: any
    object with ``n_experts`` and ``seq_offsets`` of the rows' queries."""
    e = np.abs(np.asarray(logits, np.float64) - ref_logits).max(axis=1)
    tol = []
    for b, n in enumerate(wl.n_experts):
        r0 = wl.seq_offsets[b]
        tol += [max(1e-4, 1.6 * (e[r0 + k] + e[r0])) for k in range(1, n + 1)]
    return np.array(tol)


def score_tol(logits, ref_logits, wl, beta_gpu, beta_ref, top1_ref) -> np.ndarray:
    """Per-query bound on |top_gpu - top_ref| for the fused scores of Eq. 2. A
    score (1 + b) s_k - b s_0 + c moves by at most (1 + 2 b) e with e the query's
    max logit error, plus |d b| |s_k - s_0| from the difference in beta, plus
    the fp32 evaluation of Eq. 2 (a few ulp of the score, taken as 1e-5 of it);
    top-1 and top-2 are maxima of such scores, so they move by at most as much."""
    lg = np.asarray(logits, np.float64)
    out = []
    e0 = 0
    for b, n in enumerate(wl.n_experts):
        r0, r1 = wl.seq_offsets[b], wl.seq_offsets[b + 1]
        e = float(np.abs(lg[r0:r1] - ref_logits[r0:r1]).max())
        bb = np.asarray(beta_ref[e0:e0 + n], np.float64)
        db = float(np.abs(np.asarray(beta_gpu[e0:e0 + n], np.float64) - bb).max())
        spread = float(np.abs(ref_logits[r0 + 1:r1] - ref_logits[r0][None, :]).max())
        out.append((1 + 2 * float(bb.max())) * e + db * spread + 1e-5 * max(1.0, abs(float(top1_ref[b]))))
        e0 += n
    return np.array(out)


def fused_best(logits_query, relevance, gamma, beta):
    """S(v) = max over experts of Eq. 2 (oracle, float64)."""
    return O.contrastive_scores(logits_query, beta, O.prior_term(relevance, gamma)).max(axis=0)


def check_tokens(gpu_tokens, ref_logits, wl: W.Workload, beta, ref_sel_tokens, ref_gaps, rule="max"):
    """Token contract: identical unless the oracle's top-2 gap is below 1e-3; in
    that case the GPU token must score within 1e-3 of the oracle's best (under
    the selection rule: Eq. 3's max, or the MoE / PoE aggregation).
    Returns the number of exempted queries."""
    exempt = 0
    off = wl.seq_offsets
    e0 = 0
    for b, n in enumerate(wl.n_experts):
        rows = ref_logits[off[b]:off[b + 1]]
        if int(gpu_tokens[b]) != int(ref_sel_tokens[b]):
            assert ref_gaps[b] < GAP_EXEMPT, (
                f"query {b}: gpu token {gpu_tokens[b]} != oracle {ref_sel_tokens[b]} with gap {ref_gaps[b]}")
            if rule == "max":
                S = fused_best(rows, wl.relevance[e0:e0 + n], wl.gamma, beta[e0:e0 + n])
            else:
                S = O.aggregate_scores(rows, wl.relevance[e0:e0 + n], wl.gamma, beta[e0:e0 + n], rule)[0]
            assert S[int(gpu_tokens[b])] >= S.max() - GAP_EXEMPT
            exempt += 1
        e0 += n
    return exempt
