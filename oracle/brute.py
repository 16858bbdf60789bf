"""Scalar-loop brute force of the PCED decode step for tiny inputs.

TEST INFRASTRUCTURE ONLY (see ``pced_oracle``). Pure Python floats and loops,
no NumPy linear algebra: an independent second reading of the same definitions
(Section 3, Eq. 2 and Eq. 3), used to cross-check the NumPy oracle. Inputs are
nested lists of Python floats that already hold the stored values.
"""
from __future__ import annotations

import math


def attention(q, K, V):
    """q[h][d]; K[t][g][d]; V[t][g][d] -> o[h][d]."""
    Hq, D, T, Hkv = len(q), len(q[0]), len(K), len(K[0])
    group = Hq // Hkv
    out = []
    for h in range(Hq):
        g = h // group
        z = []
        for t in range(T):
            acc = 0.0
            for d in range(D):
                acc += q[h][d] * K[t][g][d]
            z.append(acc / math.sqrt(D))
        zmax = max(z)
        w = [math.exp(x - zmax) for x in z]
        tot = sum(w)
        out.append([sum(w[t] * V[t][g][d] for t in range(T)) / tot for d in range(D)])
    return out


def logits(x, W, rms: bool):
    """x[j] (one sequence); W[v][j] -> s[v]."""
    n = len(x)
    rho = 1.0 / math.sqrt(sum(v * v for v in x) / n + 1e-5) if rms else 1.0
    return [rho * sum(x[j] * W[v][j] for j in range(n)) for v in range(len(W))]


def jsd_bits(sk, s0):
    def probs(s):
        m = max(s)
        e = [math.exp(x - m) for x in s]
        z = sum(e)
        return [x / z for x in e]
    p, q = probs(sk), probs(s0)
    tot = 0.0
    for a, b in zip(p, q):
        m = 0.5 * (a + b)
        if a > 0:
            tot += 0.5 * a * math.log2(a / m)
        if b > 0:
            tot += 0.5 * b * math.log2(b / m)
    return tot


def pick(rows, relevance, gamma, beta):
    """rows[0] = amateur logits, rows[1..N] = experts; returns (token, winner, top1, top2).

    Enumerates every (token, expert) pair."""
    N, V = len(rows) - 1, len(rows[0])
    best_v = []
    best_k = []
    for v in range(V):
        bv, bk = -math.inf, 0
        for k in range(1, N + 1):
            r = min(max(relevance[k - 1], 1e-8), 1 - 1e-8)
            val = (1 + beta[k - 1]) * rows[k][v] - beta[k - 1] * rows[0][v] + gamma * math.log(r)
            if val > bv:
                bv, bk = val, k
        best_v.append(bv)
        best_k.append(bk)
    tok = 0
    for v in range(1, V):
        if best_v[v] > best_v[tok]:
            tok = v
    top2 = -math.inf
    for v in range(V):
        if v != tok and best_v[v] > top2:
            top2 = best_v[v]
    return tok, best_k[tok], best_v[tok], top2


def aggregate_pick(rows, relevance, gamma, beta, rule):
    """The MoE / PoE aggregation variants with scalar loops (same reading as
    pced_oracle.aggregate_query): weights w_k proportional to clip(r_k)^gamma,
    distributions softmax((1 + beta_k) s_k - beta_k s_0); MoE score
    log sum_k w_k p_k(v), PoE score sum_k w_k log p_k(v).
    Returns (token, expert, best score, second-best score)."""
    s0 = rows[0]
    V, N = len(s0), len(rows) - 1
    raw = [min(max(r, 1e-8), 1.0 - 1e-8) ** gamma for r in relevance]
    w = [x / sum(raw) for x in raw]
    probs = []
    for k in range(1, N + 1):
        c = [(1.0 + beta[k - 1]) * rows[k][v] - beta[k - 1] * s0[v] for v in range(V)]
        m = max(c)
        e = [math.exp(x - m) for x in c]
        tot = sum(e)
        probs.append([x / tot for x in e])
    score = []
    for v in range(V):
        if rule == "moe":
            score.append(math.log(sum(w[k] * probs[k][v] for k in range(N))))
        else:
            score.append(sum(w[k] * math.log(probs[k][v]) for k in range(N)))
    best = max(score)
    token = score.index(best)
    contrib = [w[k] * probs[k][token] for k in range(N)]
    expert = contrib.index(max(contrib)) + 1
    second = max([score[v] for v in range(V) if v != token], default=-math.inf)
    return token, expert, best, second


# ------------------------------------------------------- decoder around the step

def bf16(x: float) -> float:
    """Round a Python float to bfloat16 (through float32, nearest-even)."""
    import struct
    u = struct.unpack("<I", struct.pack("<f", x))[0]
    # float64 -> float32 rounding happened in pack; now float32 -> bfloat16
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return struct.unpack("<f", struct.pack("<I", u))[0]


def decoder_layer(h, pos, W, cacheK, cacheV, Hq, Hkv, D, theta, eps=1e-5):
    """One decoder layer for one sequence, scalar loops.

    h[j]: residual stream; pos: the new token's position (cache length);
    W: dict of nested lists (attn_norm[j], wq[r][j], wk, wv, wo[j][r], mlp_norm,
    w_gate[f][j], w_up, w_down[j][f]); cacheK/cacheV: lists of [g][d] rows,
    extended in place. Returns (new h, attention output o[h][d])."""
    n = len(h)

    def rho_of(x):
        return 1.0 / math.sqrt(sum(v * v for v in x) / n + eps)

    def normed(x, g, M):
        a = [bf16(x[j] * g[j]) for j in range(n)]
        r = rho_of(x)
        return [r * sum(a[j] * row[j] for j in range(n)) for row in M]

    def rot(vec, p):
        out = list(vec)
        for i in range(D // 2):
            ang = p * theta ** (-2.0 * i / D)
            c, s = math.cos(ang), math.sin(ang)
            x0, x1 = vec[2 * i], vec[2 * i + 1]
            out[2 * i] = x0 * c - x1 * s
            out[2 * i + 1] = x0 * s + x1 * c
        return out

    q = normed(h, W["attn_norm"], W["wq"])
    k = normed(h, W["attn_norm"], W["wk"])
    v = normed(h, W["attn_norm"], W["wv"])
    qh = [[bf16(x) for x in rot(q[hh * D:(hh + 1) * D], pos)] for hh in range(Hq)]
    kh = [[bf16(x) for x in rot(k[g * D:(g + 1) * D], pos)] for g in range(Hkv)]
    vh = [[bf16(x) for x in v[g * D:(g + 1) * D]] for g in range(Hkv)]
    cacheK.append(kh)
    cacheV.append(vh)
    o = attention(qh, cacheK, cacheV)
    oflat = [bf16(x) for row in o for x in row]
    h2 = [h[j] + sum(oflat[r] * W["wo"][j][r] for r in range(len(oflat))) for j in range(n)]
    gate = normed(h2, W["mlp_norm"], W["w_gate"])
    up = normed(h2, W["mlp_norm"], W["w_up"])
    act = [bf16(gv / (1.0 + math.exp(-gv)) * uv) for gv, uv in zip(gate, up)]
    h3 = [h2[j] + sum(act[f] * W["w_down"][j][f] for f in range(len(act))) for j in range(n)]
    return h3, o


def model_logits(h, final_norm, lm_head, eps=1e-5):
    """RMSNorm(h) * g W^T for one sequence under the same rounding contract."""
    n = len(h)
    a = [bf16(h[j] * final_norm[j]) for j in range(n)]
    r = 1.0 / math.sqrt(sum(v * v for v in h) / n + eps)
    return [r * sum(a[j] * row[j] for j in range(n)) for row in lm_head]
