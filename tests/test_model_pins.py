"""Pins of the decoder-stack oracle (``oracle/model.py``) against closed forms,
invariants, a library routine and a scalar-loop brute force (CPU only)."""
import math

import numpy as np
import pytest
from scipy.special import expit

from oracle import brute as B
from oracle import model as M
from oracle.pced_oracle import attention, decode_stored, round_to_bf16
from pced_inputs import workloads as W
from pced_inputs.model import LAYER_TENSORS, ModelSpec, suffix_tokens


# ---------------------------------------------------------------- RoPE

def test_rope_position_zero_is_identity():
    x = np.random.default_rng(0).normal(size=(3, 8))
    np.testing.assert_array_equal(M.rope(x, 0, 10000.0), x)


def test_rope_first_pair_rotates_by_position_radians():
    # i = 0: theta^0 = 1, so the pair (1, 0) becomes (cos p, sin p), (0, 1) becomes (-sin p, cos p)
    for p in (1, 7, 1000):
        np.testing.assert_allclose(M.rope(np.array([1.0, 0.0]), p, 500000.0), [math.cos(p), math.sin(p)],
                                   atol=1e-12)
        np.testing.assert_allclose(M.rope(np.array([0.0, 1.0]), p, 500000.0), [-math.sin(p), math.cos(p)],
                                   atol=1e-12)


def test_rope_pair_frequencies():
    # D = 4, theta = 100: pair 1 turns by p * 100^(-2/4) = p / 10
    for p in (3, 25):
        out = M.rope(np.array([0.0, 0.0, 1.0, 0.0]), p, 100.0)
        np.testing.assert_allclose(out, [0, 0, math.cos(p / 10), math.sin(p / 10)], atol=1e-12)


def test_rope_preserves_pair_norms_and_depends_on_relative_position():
    rng = np.random.default_rng(1)
    q, k = rng.normal(size=16), rng.normal(size=16)
    for p in (0, 5, 123):
        r = M.rope(q, p, 500000.0)
        np.testing.assert_allclose(r[0::2] ** 2 + r[1::2] ** 2, q[0::2] ** 2 + q[1::2] ** 2, rtol=1e-12)
    # <rope(q, m), rope(k, n)> depends only on m - n
    d = [M.rope(q, m, 10000.0) @ M.rope(k, m - 4, 10000.0) for m in (4, 10, 300)]
    np.testing.assert_allclose(d, d[0], rtol=1e-10)


# ------------------------------------------------------- norm and SiLU

def test_normed_product_closed_form_constant_row():
    # h = c (constant), g = 1, W = I: rho = 1/sqrt(c^2 + eps), result = rho * bf16(c)
    for c in (0.5, -3.0, 1e-2):
        h = np.full((1, 8), c)
        out = M.normed_product(h, np.ones(8), np.eye(8))
        np.testing.assert_allclose(out, np.full((1, 8), float(round_to_bf16(np.array(c))) / math.sqrt(c * c + 1e-5)),
                                   rtol=1e-14)


def test_normed_product_is_scale_invariant_for_powers_of_two():
    rng = np.random.default_rng(2)
    h = rng.normal(size=(2, 64)) * 10
    g = 1 + 0.1 * rng.normal(size=64)
    Wm = rng.normal(size=(5, 64))
    a = M.normed_product(h, g, Wm, eps=0.0)
    b = M.normed_product(h * 8.0, g, Wm, eps=0.0)   # bf16 rounding commutes with x8
    np.testing.assert_allclose(a, b, rtol=1e-13)


def test_silu_is_x_times_logistic():
    x = np.linspace(-30, 30, 101)
    np.testing.assert_allclose(M.silu(x), x * expit(x), rtol=1e-13, atol=1e-300)
    assert M.silu(np.array([0.0]))[0] == 0.0


# ---------------------------------------------------------- model steps

def _tiny(seed=0, L=2, n_experts=(2, 1), lens=(3, 0, 2), am=(1, 2), V=11):
    geom = W.Geometry(L, 2, 1, 4, 8, V, "bf16")
    spec = ModelSpec(geom, ffn_dim=8, rope_theta=10000.0, seed=seed)
    rng = np.random.default_rng(seed)
    # per-sequence cache lengths: amateur first in each query
    clen, i = [], 0
    for b, n in enumerate(n_experts):
        clen.append(am[b])
        clen.extend(lens[i:i + n])
        i += n
    caches = {(s, l, kv): (rng.normal(size=(clen[s], 1, 4))) for s in range(len(clen)) for l in range(L)
              for kv in "kv"}
    caches = {k: W.counter.f32_to_bf16_bits(v.astype(np.float32)) for k, v in caches.items()}
    return geom, spec, clen, caches


def _oracle(geom, spec, clen, caches, n_experts, relevance, zero=(), beta=None):
    def weights(name, l):
        w = spec.host(name, l)
        return np.zeros_like(w) if name in zero else w
    return M.ModelOracle(
        n_layers=geom.n_layers, n_q_heads=geom.n_q_heads, n_kv_heads=geom.n_kv_heads, head_dim=geom.head_dim,
        vocab=geom.vocab, rope_theta=spec.rope_theta, n_experts=n_experts,
        cache_k=lambda s, l: caches[(s, l, "k")], cache_v=lambda s, l: caches[(s, l, "v")],
        weights=weights, embed=lambda rows: spec.host("embed", 0, rows), final_norm=spec.host("final_norm"),
        lm_head=W.host_values(W.counter.key(spec.seed, 99), 0, geom.vocab * geom.hidden, 0.02, "bf16")
        .reshape(geom.vocab, geom.hidden), relevance=relevance, beta=beta)


def test_model_step_matches_scalar_brute_force():
    n_exp = (2, 1)
    geom, spec, clen, caches = _tiny()
    orc = _oracle(geom, spec, clen, caches, n_exp, [0.3, 0.9, 0.5])
    toks = np.array([4, 9])
    res = orc.step(toks)
    dec = lambda a: decode_stored(a, "bf16").tolist()  # noqa: E731
    Wl = [{n: dec(spec.host(n, l)) for n in LAYER_TENSORS} for l in range(geom.n_layers)]
    lm = dec(W.host_values(W.counter.key(spec.seed, 99), 0, geom.vocab * geom.hidden, 0.02, "bf16")
             .reshape(geom.vocab, geom.hidden))
    seq_query = [0, 0, 0, 1, 1]
    for s in range(5):
        h = dec(spec.host("embed", 0, [toks[seq_query[s]]]))[0]
        for l in range(geom.n_layers):
            K = [list(r) for r in dec(caches[(s, l, "k")])]
            V = [list(r) for r in dec(caches[(s, l, "v")])]
            h, o = B.decoder_layer(h, clen[s], Wl[l], K, V, 2, 1, 4, spec.rope_theta)
            np.testing.assert_allclose(res.attn[l][s], o, rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(res.hidden[s], h, rtol=1e-9, atol=1e-12)
        lg = B.model_logits(h, dec(spec.host("final_norm")), lm)
        np.testing.assert_allclose(res.logits[s], lg, rtol=1e-9, atol=1e-12)


def test_layers_without_output_projections_leave_the_embedding():
    # wo = w_down = 0: every layer adds nothing, so the logits are the normed
    # product of each query's token embedding, whatever the caches hold
    n_exp = (2, 1)
    geom, spec, clen, caches = _tiny(seed=3)
    orc = _oracle(geom, spec, clen, caches, n_exp, [0.3, 0.9, 0.5], zero=("wo", "w_down"))
    toks = np.array([7, 2])
    res = orc.step(toks)
    emb = decode_stored(spec.host("embed", 0, [7, 7, 7, 2, 2]), "bf16")
    np.testing.assert_array_equal(res.hidden, emb)
    lm = decode_stored(W.host_values(W.counter.key(spec.seed, 99), 0, geom.vocab * geom.hidden, 0.02, "bf16")
                       .reshape(geom.vocab, geom.hidden), "bf16")
    np.testing.assert_allclose(res.logits, M.normed_product(emb, decode_stored(spec.host("final_norm"), "bf16"), lm),
                               rtol=1e-14)
    # every cache grew by one row per layer
    assert orc.lengths() == [c + 1 for c in clen]


def test_empty_cache_attends_only_to_the_new_token():
    # sequences with empty caches: each attention output is the sequence's own
    # (rounded) new value row, for every q-head of the group
    n_exp = (1,)
    geom, spec, clen, caches = _tiny(seed=4, L=1, n_experts=n_exp, lens=(0,), am=(0,))
    orc = _oracle(geom, spec, clen, caches, n_exp, [0.5])
    res = orc.step(np.array([5]))
    for s in range(2):
        v_row = orc.Vc[s][0][0]                           # the only row: the appended one
        np.testing.assert_array_equal(res.attn[0][s], np.repeat(v_row, 2, axis=0))


def test_prefill_one_token_at_a_time_equals_causal_block_form():
    # the sequential path against the matrix form of a multi-token prefill: all
    # suffix tokens' q/k/v at once (positions len .. len+n-1), causal block attention
    n_exp = (1,)
    geom, spec, clen, caches = _tiny(seed=5, L=2, n_experts=n_exp, lens=(3,), am=(2,))
    toks = suffix_tokens(5, 1, 4, geom.vocab)
    seq = _oracle(geom, spec, clen, caches, n_exp, [0.5])
    seq.prefill(toks)
    D, Hq, Hkv = geom.head_dim, geom.n_q_heads, geom.n_kv_heads
    wt = lambda n, l: decode_stored(spec.host(n, l), "bf16")  # noqa: E731
    for s in range(2):
        n = toks.shape[1]
        h = decode_stored(spec.host("embed", 0, toks[0]), "bf16")       # [n, hidden]
        for l in range(geom.n_layers):
            g = wt("attn_norm", l)
            q = M.normed_product(h, g, wt("wq", l)).reshape(n, Hq, D)
            k = M.normed_product(h, g, wt("wk", l)).reshape(n, Hkv, D)
            v = round_to_bf16(M.normed_product(h, g, wt("wv", l)).reshape(n, Hkv, D))
            q = np.stack([round_to_bf16(M.rope(q[i], clen[s] + i, spec.rope_theta)) for i in range(n)])
            k = np.stack([round_to_bf16(M.rope(k[i], clen[s] + i, spec.rope_theta)) for i in range(n)])
            K = np.concatenate([decode_stored(caches[(s, l, "k")], "bf16"), k])
            V = np.concatenate([decode_stored(caches[(s, l, "v")], "bf16"), v])
            np.testing.assert_allclose(seq.K[s][l], K, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(seq.Vc[s][l], V, rtol=1e-12, atol=1e-12)
            o = M.causal_block_attention(q, K, V, n)
            h = h + round_to_bf16(o.reshape(n, Hq * D)) @ wt("wo", l).T
            gm = wt("mlp_norm", l)
            act = round_to_bf16(M.silu(M.normed_product(h, gm, wt("w_gate", l))) *
                                M.normed_product(h, gm, wt("w_up", l)))
            h = h + act @ wt("w_down", l).T


def test_causal_block_attention_last_row_is_plain_attention():
    rng = np.random.default_rng(6)
    K, V = rng.normal(size=(9, 2, 8)), rng.normal(size=(9, 2, 8))
    Q = rng.normal(size=(3, 4, 8))
    out = M.causal_block_attention(Q, K, V, 3)
    for i in range(3):
        np.testing.assert_allclose(out[i], attention(Q[i], K[:7 + i], V[:7 + i]), rtol=1e-12)


@pytest.mark.parametrize("theta", [10000.0, 500000.0])
def test_per_sequence_positions_follow_cache_lengths(theta):
    # two sequences with the same token and identical caches except length:
    # their new K rows differ exactly by the RoPE of their positions
    n_exp = (1,)
    geom, spec, clen, caches = _tiny(seed=7, L=1, n_experts=n_exp, lens=(5,), am=(2,))
    spec = ModelSpec(geom, ffn_dim=8, rope_theta=theta, seed=7)
    orc = _oracle(geom, spec, clen, caches, n_exp, [0.5])
    orc.step(np.array([3]))
    k_am, k_ex = orc.K[0][0][-1], orc.K[1][0][-1]
    # both come from the same embedding row: undo each rotation and compare
    h = decode_stored(spec.host("embed", 0, [3]), "bf16")
    k = M.normed_product(h, decode_stored(spec.host("attn_norm", 0), "bf16"),
                         decode_stored(spec.host("wk", 0), "bf16")).reshape(1, 4)
    np.testing.assert_array_equal(k_am, round_to_bf16(M.rope(k, 2, theta)))
    np.testing.assert_array_equal(k_ex, round_to_bf16(M.rope(k, 5, theta)))
