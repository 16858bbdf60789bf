"""Plain CPU oracle for one PCED decode step (Parallel Context-of-Experts Decoding,
arXiv 2601.08670).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or execute
this module; only the tests, the package's smoke check and the benchmark's CPU
baseline leg use it. It is deliberately slow: NumPy float64, the plain
definitions, no blocking, no fusion, no paging (caches are contiguous arrays).

What one step computes (Section 3, "Parallel Context-of-Experts" and
"Retrieval-aware contrastive decoding"):

1. Shared history: the token chosen at the previous step is appended to *every*
   expert's cache, so each sequence's cache grows by one K/V row per layer and the
   new row is attended by the query of this step (Section 3, last sentence).
2. Each of the N+1 sequences of a query (amateur k=0 with no document, experts
   k=1..N with one document each) attends over its own cache with its own query
   (Section 3, Eq. 1 datastore and the batched forward pass). The paper does not
   restate attention; it is standard scaled dot-product attention with grouped
   query heads: head h reads kv-head h // (Hq / Hkv).
3. Each sequence's final hidden state is projected to full-vocabulary logits s_k.
   Reading used: the hidden state is the last layer's attention output,
   concatenated over heads, rounded to the storage precision (bf16, or fp32 for
   fp32 workloads) and, with ``norm='rms'``, scaled by 1/sqrt(mean(x^2) + 1e-5).
4. Eq. 2: s_hat_k = (1 + beta_k) s_k - beta_k s_0 + gamma log r_k for k = 1..N,
   with r clipped to [1e-8, 1 - 1e-8] (Appendix B clips away from 0 and below 1,
   epsilon = 1e-8) and the natural logarithm.
5. beta: either given per expert, or dynamic: at the first generated token of the
   query beta_k = JSD(softmax s_k || softmax s_0) in bits (AdaCAD's divergence
   between the with-context and the no-context distributions), then kept fixed
   (Section 3, text after Eq. 2).
6. Eq. 3: y = argmax_v max_{k=1..N} s_hat_k(v); the amateur is not a candidate.
   Ties: lowest token id; the reported expert is the lowest k attaining the max.
   Also reported: the best score and the best score over all other tokens (top-2
   of distinct tokens), whose difference is the top-2 gap.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Optional, Sequence

import numpy as np

RELEVANCE_EPS = 1e-8
RMS_EPS = 1e-5


# ------------------------------------------------------------ storage decode

def decode_stored(a: np.ndarray, dtype: str) -> np.ndarray:
    """Stored values -> float64. bf16 values arrive as uint16 bit patterns: a bf16
    number is the upper half of the float32 with the same sign/exponent/mantissa."""
    if dtype == "bf16":
        u = np.asarray(a).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits), ties to
    even, returned as float64. Written from the format's definition with frexp."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                   # x = m * 2**e, 0.5 <= |m| < 1
    q = np.rint(m * 256.0) / 256.0       # keep 8 significant bits; rint is half-to-even
    return np.ldexp(q, e)


def round_to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_to_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    raise ValueError(dtype)


# ------------------------------------------------------------------ attention

def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Scaled dot-product attention for one sequence and one layer.

    q: [Hq, D]; K, V: [T, Hkv, D] (float64). Returns o: [Hq, D].
    o[h] = sum_j softmax_j(q[h] . K[j, g] / sqrt(D)) V[j, g], g = h // (Hq/Hkv).
    """
    Hq, D = q.shape
    T, Hkv, _ = K.shape
    group = Hq // Hkv
    o = np.empty((Hq, D), dtype=np.float64)
    for h in range(Hq):
        g = h // group
        z = K[:, g, :] @ q[h] / math.sqrt(D)
        p = np.exp(z - z.max())
        p /= p.sum()
        o[h] = p @ V[:, g, :]
    return o


def partial_softmax(q: np.ndarray, K: np.ndarray, V: np.ndarray):
    """Unnormalised attention over one chunk of keys for one head.

    q: [D]; K, V: [T, D]. Returns (m, l, acc): m = max score (-inf for an empty
    chunk), l = sum exp(z - m), acc = sum exp(z - m) V."""
    D = q.shape[0]
    if K.shape[0] == 0:
        return -np.inf, 0.0, np.zeros(V.shape[1])
    z = K @ q / math.sqrt(D)
    m = z.max()
    w = np.exp(z - m)
    return m, w.sum(), w @ V


def merge_partials(parts) -> np.ndarray:
    """Log-sum-exp merge of chunk results: o = sum_i acc_i e^(m_i - m) / sum_i l_i e^(m_i - m),
    m = max_i m_i; empty chunks (m = -inf) contribute nothing."""
    m = max(p[0] for p in parts)
    num = sum(p[2] * math.exp(p[0] - m) for p in parts if p[0] != -np.inf)
    den = sum(p[1] * math.exp(p[0] - m) for p in parts if p[0] != -np.inf)
    return num / den


# -------------------------------------------------------------------- LM head

def rms_scale(x: np.ndarray) -> np.ndarray:
    """Per-row 1 / sqrt(mean(x^2) + 1e-5) (unit-weight RMS normalisation)."""
    return 1.0 / np.sqrt(np.mean(np.square(x), axis=-1) + RMS_EPS)


def lm_head(x: np.ndarray, W: np.ndarray, norm: str = "rms") -> np.ndarray:
    """Full-vocabulary logits: s[i, v] = rho_i * sum_j x[i, j] W[v, j].

    x: [S, hidden] float64 (already at storage precision); W: [V, hidden] float64."""
    logits = x @ W.T
    if norm == "rms":
        logits = logits * rms_scale(x)[:, None]
    elif norm != "none":
        raise ValueError(norm)
    return logits


# ------------------------------------------------------------------ beta / JSD

def softmax(s: np.ndarray) -> np.ndarray:
    p = np.exp(s - s.max())
    return p / p.sum()


def jsd_bits(p: np.ndarray, q: np.ndarray) -> float:
    """Jensen-Shannon divergence in bits: 1/2 KL(p||m) + 1/2 KL(q||m), m = (p+q)/2,
    with 0 log 0 = 0."""
    m = 0.5 * (p + q)
    def kl(a):
        nz = a > 0
        return float(np.sum(a[nz] * np.log2(a[nz] / m[nz])))
    return 0.5 * kl(p) + 0.5 * kl(q)


def dynamic_beta(logits_query: np.ndarray, scalar: bool = False) -> np.ndarray:
    """beta_k = JSD(softmax s_k, softmax s_0) for k = 1..N (one query's rows, amateur first).
    ``scalar``: one beta for the query, the mean of those divergences (the paper's
    beta_0 read as a single number), repeated for every expert."""
    p0 = softmax(logits_query[0])
    b = np.array([jsd_bits(softmax(logits_query[k]), p0) for k in range(1, logits_query.shape[0])])
    return np.full_like(b, b.mean()) if scalar else b


# ----------------------------------------------------------------- Eq. 2 / 3

def clip_relevance(r: np.ndarray) -> np.ndarray:
    return np.clip(np.asarray(r, dtype=np.float64), RELEVANCE_EPS, 1.0 - RELEVANCE_EPS)


def prior_term(r: np.ndarray, gamma: float) -> np.ndarray:
    """gamma * ln(clip(r)), the retrieval prior of Eq. 2."""
    return gamma * np.log(clip_relevance(r))


@dataclasses.dataclass
class Selection:
    token: int
    winner: int        # expert index 1..N
    top1: float
    top2: float        # best fused score over all other tokens (-inf if V == 1)

    @property
    def gap(self) -> float:
        return self.top1 - self.top2


def contrastive_scores(logits_query: np.ndarray, beta: np.ndarray, prior: np.ndarray,
                       precision=np.float64) -> np.ndarray:
    """Eq. 2 for every expert k = 1..N and token v: [N, V].

    With ``precision=np.float32`` each operation of (1 + beta) s_k - beta s_0 + prior
    is rounded to float32 in the order the equation is written (no fused
    multiply-add), as a float32 implementation evaluates it."""
    if precision is np.float64:
        s = np.asarray(logits_query, dtype=np.float64)
        b = np.asarray(beta, dtype=np.float64)[:, None]
        return (1.0 + b) * s[1:] - b * s[0][None, :] + np.asarray(prior, dtype=np.float64)[:, None]
    f = np.float32
    s = np.asarray(logits_query, dtype=f)
    b = np.asarray(beta, dtype=f)[:, None]
    a = (f(1.0) + b).astype(f)
    t1 = (a * s[1:]).astype(f)
    t2 = (b * s[0][None, :]).astype(f)
    return ((t1 - t2).astype(f) + np.asarray(prior, dtype=f)[:, None]).astype(f)


def select(scores: np.ndarray) -> Selection:
    """Eq. 3 over calibrated scores [N, V]: y = argmax_v max_k s_hat_k(v); lowest
    token on ties, lowest expert among the maximisers at y."""
    best = scores.max(axis=0)                       # S(v) = max over experts
    top1 = best.max()
    token = int(np.flatnonzero(best == top1)[0])
    winner = int(np.flatnonzero(scores[:, token] == top1)[0]) + 1
    others = np.delete(best, token)
    top2 = float(others.max()) if others.size else -math.inf
    return Selection(token, winner, float(top1), top2)


# ------------------------------------------- aggregation rules (Appendix C.4)
# The ablation compares Max with a mixture (weighted sum) and a product
# (weighted product) of the experts' distributions, weights from the retrieval
# scores, without formulas. Reading used here: each expert's distribution is
# the softmax of its contrastive logits c_k = (1 + beta_k) s_k - beta_k s_0
# (Eq. 2 without the prior), and the weights are pi_k = r_k^gamma / sum_j r_j^gamma
# (so log pi_k is Eq. 2's prior gamma log r_k up to a constant). Scores are
# reported in log units:
#     MoE: log sum_k pi_k softmax(c_k)(v)        PoE: sum_k pi_k log softmax(c_k)(v)
# The token is the argmax (lowest token on ties); the reported expert is the one
# with the largest weighted probability pi_k softmax(c_k)(y) (lowest k on ties).

def expert_weights(relevance: np.ndarray, gamma: float) -> np.ndarray:
    """pi_k = r_k^gamma / sum_j r_j^gamma over one query's clipped relevance."""
    return softmax(prior_term(relevance, gamma))


def log_softmax(c: np.ndarray) -> np.ndarray:
    m = c.max(axis=-1, keepdims=True)
    return c - (m + np.log(np.sum(np.exp(c - m), axis=-1, keepdims=True)))


def aggregate_scores(logits_query: np.ndarray, relevance: np.ndarray, gamma: float, beta: np.ndarray,
                     rule: str):
    """MoE or PoE score of every token [V] and log(pi_k p_k(v)) [N, V] for one
    query (rows: amateur, experts)."""
    s = np.asarray(logits_query, dtype=np.float64)
    b = np.asarray(beta, dtype=np.float64)[:, None]
    c = (1.0 + b) * s[1:] - b * s[0][None, :]            # contrastive logits [N, V]
    logp = log_softmax(c)
    logw = np.log(expert_weights(relevance, gamma))[:, None]
    joint = logw + logp                                  # log(pi_k p_k(v))
    if rule == "moe":
        m = joint.max(axis=0)
        score = m + np.log(np.sum(np.exp(joint - m[None, :]), axis=0))
    elif rule == "poe":
        score = np.sum(np.exp(logw) * logp, axis=0)
    else:
        raise ValueError(rule)
    return score, joint


def aggregate_query(logits_query: np.ndarray, relevance: np.ndarray, gamma: float, beta: np.ndarray,
                    rule: str) -> Selection:
    """MoE or PoE aggregation and selection for one query (rows: amateur, experts)."""
    score, joint = aggregate_scores(logits_query, relevance, gamma, beta, rule)
    top1 = score.max()
    token = int(np.flatnonzero(score == top1)[0])
    col = joint[:, token]
    winner = int(np.flatnonzero(col == col.max())[0]) + 1
    others = np.delete(score, token)
    return Selection(token, winner, float(top1), float(others.max()) if others.size else -math.inf)


def fuse_query(logits_query: np.ndarray, relevance: np.ndarray, gamma: float,
               beta: np.ndarray, precision=np.float64, rule: str = "max") -> Selection:
    """Eq. 2 then Eq. 3 for one query (rows: amateur, expert 1..N); ``rule``
    "moe" / "poe" select by the aggregation variants instead."""
    if rule != "max":
        return aggregate_query(logits_query, relevance, gamma, beta, rule)
    prior = prior_term(relevance, gamma)
    if precision is np.float32:
        prior = prior.astype(np.float32)
    return select(contrastive_scores(logits_query, beta, prior, precision))


# ------------------------------------------------------------- decode steps

@dataclasses.dataclass
class StepResult:
    tokens: np.ndarray          # [B]
    winners: np.ndarray         # [B]
    top1: np.ndarray            # [B]
    top2: np.ndarray            # [B]
    beta: np.ndarray            # [sum N] beta used at this step
    logits: np.ndarray          # [S, V]
    hidden: np.ndarray          # [S, hidden] at storage precision
    attn: dict                  # {layer: [S, Hq, D]} for the layers computed

    @property
    def gaps(self) -> np.ndarray:
        return self.top1 - self.top2


class Oracle:
    """Stateful multi-step PCED decoding over contiguous caches.

    ``cache_k(s, l)`` / ``cache_v(s, l)`` return the preloaded cache of sequence s,
    layer l as stored values [T, Hkv, D]; they are called lazily so that a caller
    can restrict work to some layers. Rows appended by the shared history are
    kept separately and concatenated after the preloaded rows.
    """

    def __init__(self, *, n_layers, n_q_heads, n_kv_heads, head_dim, vocab, dtype,
                 n_experts: Sequence[int], cache_k: Callable, cache_v: Callable,
                 relevance, gamma: float = 2.5, beta=None, norm: str = "rms", aggregation: str = "max",
                 beta_scalar: bool = False):
        self.L, self.Hq, self.Hkv, self.D, self.V = n_layers, n_q_heads, n_kv_heads, head_dim, vocab
        self.dtype = dtype
        self.n_experts = list(n_experts)
        self.seq_off = np.concatenate([[0], np.cumsum([n + 1 for n in self.n_experts])]).astype(int)
        self.S = int(self.seq_off[-1])
        self.cache_k, self.cache_v = cache_k, cache_v
        self.relevance = np.asarray(relevance, dtype=np.float64)
        self.gamma = float(gamma)
        self.fixed_beta = None if beta is None else np.asarray(beta, dtype=np.float64)
        self.frozen_beta = None
        self.norm = norm
        self.aggregation = aggregation
        self.beta_scalar = bool(beta_scalar)
        self.appended_k = [[[] for _ in range(self.L)] for _ in range(self.S)]
        self.appended_v = [[[] for _ in range(self.L)] for _ in range(self.S)]
        self.t = 0

    def _full_cache(self, s, l):
        K = decode_stored(self.cache_k(s, l), self.dtype)
        V = decode_stored(self.cache_v(s, l), self.dtype)
        if self.appended_k[s][l]:
            K = np.concatenate([K, np.stack(self.appended_k[s][l])], axis=0)
            V = np.concatenate([V, np.stack(self.appended_v[s][l])], axis=0)
        return K, V

    def step(self, q, k_new, v_new, W, attn_layers: Optional[Sequence[int]] = None) -> StepResult:
        """One decode step.

        q: [S, L, Hq, D], k_new / v_new: [S, L, Hkv, D] (stored values);
        W: [V, hidden] stored values, or a float64 array already decoded.
        ``attn_layers`` limits which layers' attention is evaluated (the last
        layer is always evaluated: the logits depend on it alone)."""
        L = self.L
        layers = sorted(set(range(L)) if attn_layers is None else set(attn_layers) | {L - 1})
        qd = decode_stored(q, self.dtype)
        kd = decode_stored(k_new, self.dtype)
        vd = decode_stored(v_new, self.dtype)
        # 1. shared history: append this step's K/V row to every sequence, every layer
        for s in range(self.S):
            for l in range(L):
                self.appended_k[s][l].append(kd[s, l])
                self.appended_v[s][l].append(vd[s, l])
        # 2. attention
        attn = {}
        for l in layers:
            out = np.empty((self.S, self.Hq, self.D))
            for s in range(self.S):
                K, V = self._full_cache(s, l)
                out[s] = attention(qd[s, l], K, V)
            attn[l] = out
        # 3. hidden state at storage precision, 4. logits
        hidden = round_to_storage(attn[L - 1].reshape(self.S, self.Hq * self.D), self.dtype)
        Wd = W if W.dtype == np.float64 else decode_stored(W, self.dtype)
        logits = lm_head(hidden, Wd, self.norm)
        # 5. beta, 6. Eq. 2 / Eq. 3 per query
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
        self.t += 1
        return StepResult(
            tokens=np.array([x.token for x in sels]), winners=np.array([x.winner for x in sels]),
            top1=np.array([x.top1 for x in sels]), top2=np.array([x.top2 for x in sels]),
            beta=np.array(beta, copy=True), logits=logits, hidden=hidden, attn=attn)


# --------------------------------------------------------------------------
# Relevance scores from raw retrieval and reranker outputs (Section 3,
# "Retrieval and relevance scoring"; Appendix B). Every normalised score is
# clipped to [0, 1 - eps]; the harmonic mean carries eps in its denominator as
# Appendix B writes it (the Section 3 formula omits it).

def normalise_retrieval(s, mode: str) -> np.ndarray:
    """Appendix B: dense / ColBERT cosine scores in [-1, 1] are rescaled
    affinely, (s + 1) / 2; sparse scores (nonnegative, unbounded) go through
    (2 / pi) arctan(max(s, 0)). Both are clipped to [0, 1 - eps]."""
    s = np.asarray(s, dtype=np.float64)
    if mode in ("dense", "colbert"):
        r = (s + 1.0) / 2.0
    elif mode == "sparse":
        r = (2.0 / math.pi) * np.arctan(np.maximum(s, 0.0))
    else:
        raise ValueError(mode)
    return np.clip(r, 0.0, 1.0 - RELEVANCE_EPS)


def normalise_reranker(z) -> np.ndarray:
    """Appendix B: the reranker's logits through the logistic sigmoid, clipped
    to [0, 1 - eps]."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):  # exp(-z) = inf for very negative z gives sigma = 0
        return np.clip(1.0 / (1.0 + np.exp(-z)), 0.0, 1.0 - RELEVANCE_EPS)


def fuse_relevance(r_ret, r_rer) -> np.ndarray:
    """Appendix B: harmonic mean 2 r_ret r_rer / (r_ret + r_rer + eps)."""
    a = np.asarray(r_ret, dtype=np.float64)
    b = np.asarray(r_rer, dtype=np.float64)
    return 2.0 * a * b / (a + b + RELEVANCE_EPS)


def relevance(retrieval, mode: str, reranker_logits=None) -> np.ndarray:
    """r_k for Eq. 2 from raw scores; retrieval only when there is no reranker."""
    r = normalise_retrieval(retrieval, mode)
    return r if reranker_logits is None else fuse_relevance(r, normalise_reranker(reranker_logits))


def kv_bytes_per_token(n_layers: int, n_kv_heads: int, head_dim: int, bytes_per_value: int) -> int:
    """Bytes of K and V cached for one token across all layers."""
    return 2 * n_layers * n_kv_heads * head_dim * bytes_per_value
