"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test names the mistake it would catch. None of them re-types the oracle's
own formula: they use published values, hand-derived closed forms, special cases
that reduce to something simpler, invariants and a scalar brute force.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import brute
from oracle import pced_oracle as O
from oracle import synth as osynth
from pced_inputs import counter

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- generators

def test_splitmix64_published_vectors_inputs_module():
    g = golden("splitmix64.json")
    assert counter.splitmix64_sequence(1234567, 5) == [int(x) for x in g["seed_1234567"]]
    assert counter.splitmix64_sequence(0, 1)[0] == int(g["seed_0_first"])
    # counter form: output i of the stream seeded with k is mix(k + (i+1) G)
    h = counter.hashes_np(1234567, 0, 5)
    assert [int(x) for x in h] == [int(x) for x in g["seed_1234567"]]


def test_splitmix64_published_vectors_oracle_synth():
    g = golden("splitmix64.json")
    outs = [osynth._mix((1234567 + (i + 1) * osynth._G) & osynth._M) for i in range(5)]
    assert outs == [int(x) for x in g["seed_1234567"]]


def test_oracle_synth_and_input_generator_agree():
    # two implementations of the same published definition, bit for bit
    for dtype in ("bf16", "f32"):
        for fields in [(1, 2, 3), (0x51, 0, 7, 3, 999)]:
            k = counter.key(42, *fields)
            assert k == osynth.fold(42, *fields)
            a = counter.values_np(k, 0, 300, 1.0, dtype)
            b = osynth.stream_values(k, 300, dtype)
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_generator_torch_cpu_matches_numpy():
    torch = pytest.importorskip("torch")
    for dtype in ("bf16", "f32"):
        a = counter.values_np(12345, 77, 5000, 0.02, dtype)
        b = counter.values_torch(12345, 77, 5000, 0.02, dtype, "cpu").numpy()
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_generator_moments():
    v = counter.values_f32_np(counter.key(7, 1), 0, 400_000, 1.0)
    assert abs(v.mean()) < 0.01 and abs(v.std() - 1.0) < 0.01
    assert np.abs(v).max() <= 3.4642
    w = counter.values_f32_np(counter.key(7, 2), 0, 400_000, 0.02)
    assert abs(w.std() - 0.02) < 2e-4


# ---------------------------------------------------------------- bf16 rounding

@pytest.mark.parametrize("bits32,bits16", [
    (0x3F800000, 0x3F80),   # 1.0 exact
    (0x3EAAAAAB, 0x3EAB),   # 1/3 rounds up
    (0x3F808000, 0x3F80),   # halfway, even stays
    (0x3F818000, 0x3F82),   # halfway, odd rounds up to even
    (0x3F80FFFF, 0x3F81),   # just below halfway+1 ulp
    (0xBF808001, 0xBF81),   # negative, above halfway
    (0x00000000, 0x0000),
    (0x80000000, 0x8000),
])
def test_bf16_rne_known_patterns(bits32, bits16):
    x = np.array([bits32], dtype=np.uint32).view(np.float32)
    assert int(counter.f32_to_bf16_bits(x)[0]) == bits16
    # the oracle's independent rounding (frexp based) lands on the same value
    want = O.decode_stored(np.array([bits16], dtype=np.uint16), "bf16")[0]
    assert O.round_to_bf16(x.astype(np.float64))[0] == want


def test_bf16_two_roundings_agree_random():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(200_000) * np.exp(rng.uniform(-20, 20, 200_000))).astype(np.float32)
    a = O.decode_stored(counter.f32_to_bf16_bits(x), "bf16")
    b = O.round_to_bf16(x.astype(np.float64))
    assert np.array_equal(a, b)


# ------------------------------------------------------------------ attention

def _rand_qkv(rng, Hq=4, Hkv=2, T=9, D=8):
    return rng.standard_normal((Hq, D)), rng.standard_normal((T, Hkv, D)), rng.standard_normal((T, Hkv, D))


def test_attention_single_key_returns_value():
    # catches: a missing normalisation, a wrong kv-head index
    rng = np.random.default_rng(0)
    q, K, V = _rand_qkv(rng, T=1)
    o = O.attention(q, K, V)
    for h in range(4):
        assert np.allclose(o[h], V[0, h // 2], rtol=0, atol=1e-15)


def test_attention_equal_keys_returns_mean_value():
    rng = np.random.default_rng(1)
    q, K, V = _rand_qkv(rng, T=6)
    K[:] = K[0]
    o = O.attention(q, K, V)
    for h in range(4):
        assert np.allclose(o[h], V[:, h // 2].mean(axis=0), atol=1e-14)


def test_attention_two_keys_logistic_closed_form():
    # With two keys softmax reduces to a logistic of the score difference; the
    # 1/sqrt(D) scale and the sign of the score are pinned by this.
    rng = np.random.default_rng(2)
    D = 16
    q, K, V = _rand_qkv(rng, Hq=2, Hkv=1, T=2, D=D)
    o = O.attention(q, K, V)
    for h in range(2):
        dz = (q[h] @ K[0, 0] - q[h] @ K[1, 0]) / math.sqrt(D)
        w0 = 1.0 / (1.0 + math.exp(-dz))
        assert np.allclose(o[h], w0 * V[0, 0] + (1 - w0) * V[1, 0], atol=1e-14)


def test_attention_dominant_key():
    rng = np.random.default_rng(3)
    q, K, V = _rand_qkv(rng, Hq=1, Hkv=1, T=7, D=8)
    K[4, 0] = 80.0 * q[0] / np.linalg.norm(q[0])
    o = O.attention(q, K, V)
    assert np.allclose(o[0], V[4, 0], atol=1e-9)
    # scores far beyond exp's float64 range must still give the dominant value
    K[4, 0] = 1e4 * q[0] / np.linalg.norm(q[0])
    K[2, 0] = 0.98e4 * q[0] / np.linalg.norm(q[0])
    o = O.attention(q, K, V)
    assert np.all(np.isfinite(o)) and np.allclose(o[0], V[4, 0], atol=1e-9)


def test_attention_gqa_grouping():
    # q-heads 0..G-1 read kv-head 0 (h // G), not h % Hkv
    rng = np.random.default_rng(4)
    q, K, V = _rand_qkv(rng, Hq=8, Hkv=2, T=5, D=8)
    o1 = O.attention(q, K, V)
    K2, V2 = K.copy(), V.copy()
    K2[:, 1] += 3.0
    V2[:, 1] *= -2.0
    o2 = O.attention(q, K2, V2)
    assert np.array_equal(o1[:4], o2[:4])
    assert not np.allclose(o1[4:], o2[4:])


def test_attention_key_shift_along_orthogonal_direction_invariant():
    rng = np.random.default_rng(5)
    q, K, V = _rand_qkv(rng, Hq=1, Hkv=1, T=10, D=8)
    c = rng.standard_normal(8)
    c -= (c @ q[0]) / (q[0] @ q[0]) * q[0]          # orthogonal to q: scores unchanged
    assert np.allclose(O.attention(q, K + c, V), O.attention(q, K, V), atol=1e-14)
    u = rng.standard_normal(8)                      # value shift moves the output by u
    assert np.allclose(O.attention(q, K, V + u), O.attention(q, K, V) + u, atol=1e-13)


def test_split_cache_softmax_recombination():
    # attention over a cache split into chunks (including empty and 1-token ones)
    # and merged by log-sum-exp equals attention over the whole cache
    rng = np.random.default_rng(6)
    for trial in range(40):
        T = int(rng.integers(1, 300))
        D = 16
        q = rng.standard_normal(D) * 2
        K = rng.standard_normal((T, D)) * 2
        V = rng.standard_normal((T, D))
        cuts = np.sort(rng.integers(0, T + 1, size=int(rng.integers(0, 8))))
        bounds = [0, *cuts.tolist(), T]
        parts = [O.partial_softmax(q, K[a:b], V[a:b]) for a, b in zip(bounds[:-1], bounds[1:])]
        full = O.attention(q[None, :], K[:, None, :], V[:, None, :])[0]
        assert np.allclose(O.merge_partials(parts), full, rtol=0, atol=1e-12)


# -------------------------------------------------------------------- LM head

def test_lm_head_one_hot_hidden_closed_form():
    rng = np.random.default_rng(7)
    W = rng.standard_normal((11, 6))
    x = np.zeros((1, 6))
    x[0, 2] = 3.0
    rho = 1.0 / math.sqrt(9.0 / 6 + 1e-5)
    assert np.allclose(O.lm_head(x, W, "rms")[0], rho * 3.0 * W[:, 2], atol=1e-14)
    assert np.allclose(O.lm_head(x, W, "none")[0], 3.0 * W[:, 2], atol=1e-14)


def test_lm_head_rms_scale_invariance():
    rng = np.random.default_rng(8)
    W = rng.standard_normal((20, 64))
    x = rng.standard_normal((3, 64)) * 50
    a = O.lm_head(x, W, "rms")
    b = O.lm_head(x * 7.0, W, "rms")
    assert np.allclose(a, b, rtol=1e-7)   # eps = 1e-5 perturbs at ~1e-9 here


# ------------------------------------------------------------------ JSD / beta

def test_jsd_identity_symmetry_bounds():
    rng = np.random.default_rng(9)
    for _ in range(20):
        p = O.softmax(rng.standard_normal(50) * 3)
        q = O.softmax(rng.standard_normal(50) * 3)
        assert O.jsd_bits(p, p) == pytest.approx(0.0, abs=1e-15)
        assert O.jsd_bits(p, q) == pytest.approx(O.jsd_bits(q, p), abs=1e-14)
        assert 0.0 <= O.jsd_bits(p, q) <= 1.0


def test_jsd_disjoint_support_is_one_bit():
    assert O.jsd_bits(np.array([1.0, 0.0]), np.array([0.0, 1.0])) == pytest.approx(1.0, abs=1e-15)


def test_jsd_binary_entropy_closed_form():
    # JSD = H(m) - (H(p) + H(q)) / 2 with binary entropy in bits (a different formula)
    def H(a):
        return -sum(x * math.log2(x) for x in (a, 1 - a) if x > 0)
    for a, b in [(0.1, 0.7), (0.5, 0.5), (0.01, 0.99), (0.3, 0.0)]:
        want = H((a + b) / 2) - (H(a) + H(b)) / 2
        assert O.jsd_bits(np.array([a, 1 - a]), np.array([b, 1 - b])) == pytest.approx(want, abs=1e-14)


def test_dynamic_beta_shift_invariant():
    rng = np.random.default_rng(10)
    rows = rng.standard_normal((4, 40))
    b1 = O.dynamic_beta(rows)
    rows2 = rows + np.array([3.0, -1.0, 10.0, 0.5])[:, None]
    assert np.allclose(O.dynamic_beta(rows2), b1, atol=1e-13)
    assert b1.shape == (3,) and np.all((b1 >= 0) & (b1 <= 1))


# ---------------------------------------------------------------- Eq. 2 / Eq. 3

def test_eq2_eq3_hand_worked_example():
    g = golden("eq2_eq3_worked.json")
    sel = O.fuse_query(np.array(g["logits"]), np.array(g["relevance"]), g["gamma"], np.array(g["beta"]))
    assert (sel.token, sel.winner) == (g["token"], g["winner"])
    assert sel.top1 == pytest.approx(g["top1"], abs=1e-14)
    assert sel.top2 == pytest.approx(g["top2"], abs=1e-14)


def test_paper_constants():
    g = golden("paper_constants.json")
    assert O.RELEVANCE_EPS == g["relevance_eps"]["value"]
    # floor of the prior at the default gamma: gamma * ln(1e-8)
    assert O.prior_term(np.array([0.0]), g["gamma_default"]["value"])[0] == pytest.approx(
        2.5 * math.log(1e-8), rel=1e-15)
    # the fixed-beta grid lies inside the range of the bits-based dynamic beta
    assert all(0 <= b <= 1 for b in g["fixed_beta_grid"]["value"])


def test_single_expert_zero_beta_is_greedy():
    # N = 1, beta = 0: the prior is a constant shift, the amateur drops out
    rng = np.random.default_rng(11)
    for _ in range(20):
        rows = rng.standard_normal((2, 100))
        for gamma in (0.0, 2.5, 10.0):
            sel = O.fuse_query(rows, np.array([rng.random()]), gamma, np.array([0.0]))
            assert sel.token == int(np.argmax(rows[1])) and sel.winner == 1


def test_zero_beta_ignores_amateur():
    rng = np.random.default_rng(12)
    rows = rng.standard_normal((5, 64))
    r = rng.random(4)
    a = O.fuse_query(rows, r, 2.5, np.zeros(4))
    rows[0] = rng.standard_normal(64) * 100
    b = O.fuse_query(rows, r, 2.5, np.zeros(4))
    assert (a.token, a.winner, a.top1) == (b.token, b.winner, b.top1)


def test_zero_gamma_flat_prior():
    rng = np.random.default_rng(13)
    rows = rng.standard_normal((5, 64))
    beta = rng.random(4)
    a = O.fuse_query(rows, rng.random(4), 0.0, beta)
    b = O.fuse_query(rows, rng.random(4), 0.0, beta)
    assert (a.token, a.winner, a.top1) == (b.token, b.winner, b.top1)


def test_experts_equal_to_amateur_make_beta_irrelevant():
    rng = np.random.default_rng(14)
    base = rng.standard_normal(64)
    rows = np.stack([base] * 4)
    r = np.array([0.2, 0.9, 0.5])
    sels = [O.fuse_query(rows, r, 2.5, rng.random(3) * k) for k in range(4)]
    assert len({(s.token, s.winner) for s in sels}) == 1
    assert sels[0].token == int(np.argmax(base)) and sels[0].winner == 2  # highest r


def test_common_shift_of_all_rows():
    rng = np.random.default_rng(15)
    rows = rng.standard_normal((6, 80))
    r, beta = rng.random(5), rng.random(5)
    a = O.fuse_query(rows, r, 2.5, beta)
    b = O.fuse_query(rows + 4.25, r, 2.5, beta)
    assert (a.token, a.winner) == (b.token, b.winner)
    assert b.top1 - a.top1 == pytest.approx(4.25, abs=1e-12)


def test_expert_permutation_invariance():
    rng = np.random.default_rng(16)
    for _ in range(20):
        N = 7
        rows = rng.standard_normal((N + 1, 90))
        r, beta = rng.random(N), rng.random(N)
        a = O.fuse_query(rows, r, 2.5, beta)
        perm = rng.permutation(N)                      # new expert i is old expert perm[i]
        rows_p = np.concatenate([rows[:1], rows[1:][perm]])
        b = O.fuse_query(rows_p, r[perm], 2.5, beta[perm])
        assert a.token == b.token and a.top1 == pytest.approx(b.top1, abs=1e-12)
        assert perm[b.winner - 1] + 1 == a.winner


def test_duplicate_expert_changes_nothing():
    rng = np.random.default_rng(17)
    rows = rng.standard_normal((4, 50))
    r, beta = rng.random(3), rng.random(3)
    a = O.fuse_query(rows, r, 2.5, beta)
    rows_d = np.concatenate([rows, rows[2:3]])
    b = O.fuse_query(rows_d, np.append(r, r[1]), 2.5, np.append(beta, beta[1]))
    assert (a.token, a.winner, a.top1) == (b.token, b.winner, b.top1)


def test_relevance_floor_needs_46_nats_lead():
    gamma = 2.5
    floor = gamma * math.log(1e-8)                    # about -46.05
    rows = np.zeros((3, 4))
    rows[1, 0] = 1.0                                  # expert 1 (r = 1 - eps) likes token 0
    rows[2, 3] = -floor - 0.5                         # expert 2 (r = 0) lead just under the floor
    sel = O.fuse_query(rows, np.array([1.0, 0.0]), gamma, np.zeros(2))
    assert sel.token == 0 and sel.winner == 1
    rows[2, 3] = -floor + 1.5                         # lead above the floor: expert 2 wins
    sel = O.fuse_query(rows, np.array([1.0, 0.0]), gamma, np.zeros(2))
    assert sel.token == 3 and sel.winner == 2


def test_amateur_is_not_a_candidate():
    rows = np.zeros((2, 5))
    rows[0, 3] = 1000.0
    rows[1, 1] = 1.0
    sel = O.fuse_query(rows, np.array([0.5]), 2.5, np.array([0.0]))
    assert sel.token == 1


def test_tie_breaks_lowest_token_and_lowest_expert():
    rows = np.zeros((4, 6))
    rows[1, 4] = rows[1, 2] = 2.0
    rows[3, 2] = 2.0
    sel = O.fuse_query(rows, np.array([0.5, 0.5, 0.5]), 2.5, np.zeros(3))
    assert sel.token == 2 and sel.winner == 1 and sel.top2 == sel.top1


def test_float32_evaluation_close_to_float64():
    rng = np.random.default_rng(18)
    rows = (rng.standard_normal((9, 500)) * 1.3).astype(np.float32)
    r, beta = rng.random(8), rng.random(8).astype(np.float32)
    s64 = O.contrastive_scores(rows, beta, O.prior_term(r, 2.5))
    s32 = O.contrastive_scores(rows, beta, O.prior_term(r, 2.5).astype(np.float32), np.float32)
    assert s32.dtype == np.float32
    assert np.abs(s32 - s64).max() < 1e-5 * np.abs(s64).max()


# --------------------------------------------------------- brute force vs oracle

@pytest.mark.parametrize("N,T,V", [(1, 1, 7), (2, 2, 7), (5, 17, 64), (2, 17, 64)])
def test_brute_force_agrees(N, T, V):
    rng = np.random.default_rng(100 + N * T + V)
    Hq, Hkv, D = 4, 2, 8
    q, K, Vv = rng.standard_normal((Hq, D)), rng.standard_normal((T, Hkv, D)), rng.standard_normal((T, Hkv, D))
    assert np.allclose(O.attention(q, K, Vv), brute.attention(q.tolist(), K.tolist(), Vv.tolist()),
                       rtol=0, atol=1e-12)
    W = rng.standard_normal((V, 16))
    x = rng.standard_normal(16)
    assert np.allclose(O.lm_head(x[None], W, "rms")[0], brute.logits(x.tolist(), W.tolist(), True), atol=1e-12)
    rows = rng.standard_normal((N + 1, V))
    r, beta = rng.random(N), rng.random(N)
    sel = O.fuse_query(rows, r, 2.5, beta)
    tok, win, t1, t2 = brute.pick(rows.tolist(), r.tolist(), 2.5, beta.tolist())
    assert (sel.token, sel.winner) == (tok, win)
    assert sel.top1 == pytest.approx(t1, abs=1e-12)
    assert sel.top2 == pytest.approx(t2, abs=1e-12)
    for k in range(1, N + 1):
        assert O.jsd_bits(O.softmax(rows[k]), O.softmax(rows[0])) == pytest.approx(
            brute.jsd_bits(rows[k].tolist(), rows[0].tolist()), abs=1e-12)


def test_whole_step_brute_force_tiny():
    # two queries, ragged caches, fp32 storage, dynamic beta, two steps
    rng = np.random.default_rng(21)
    Hq, Hkv, D, V, L = 2, 1, 4, 9, 2
    n_exp = [2, 1]
    lens = [1, 3, 2, 2, 4]
    S = len(lens)
    ck = [rng.standard_normal((L, T, Hkv, D)).astype(np.float32) for T in lens]
    cv = [rng.standard_normal((L, T, Hkv, D)).astype(np.float32) for T in lens]
    W = (rng.standard_normal((V, Hq * D)) * 0.5).astype(np.float32)
    rel = rng.random(3).astype(np.float32)
    orc = O.Oracle(n_layers=L, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, vocab=V, dtype="f32",
                   n_experts=n_exp, cache_k=lambda s, l: ck[s][l], cache_v=lambda s, l: cv[s][l],
                   relevance=rel, gamma=2.5)
    hist_k = [[list(ck[s][l].astype(np.float64).tolist()) for l in range(L)] for s in range(S)]
    hist_v = [[list(cv[s][l].astype(np.float64).tolist()) for l in range(L)] for s in range(S)]
    beta = None
    for t in range(2):
        q = rng.standard_normal((S, L, Hq, D)).astype(np.float32)
        kn = rng.standard_normal((S, L, Hkv, D)).astype(np.float32)
        vn = rng.standard_normal((S, L, Hkv, D)).astype(np.float32)
        res = orc.step(q, kn, vn, W)
        logits = []
        for s in range(S):
            for l in range(L):
                hist_k[s][l].append(kn[s, l].astype(np.float64).tolist())
                hist_v[s][l].append(vn[s, l].astype(np.float64).tolist())
            o = brute.attention(q[s, L - 1].astype(np.float64).tolist(), hist_k[s][L - 1], hist_v[s][L - 1])
            x = [float(np.float32(v)) for row in o for v in row]
            logits.append(brute.logits(x, W.astype(np.float64).tolist(), True))
        assert np.allclose(res.logits, np.array(logits), atol=1e-12)
        if beta is None:
            beta = [brute.jsd_bits(logits[s], logits[0]) for s in (1, 2)] + [brute.jsd_bits(logits[4], logits[3])]
        assert np.allclose(res.beta, beta, atol=1e-12)
        for b, (s0, n, e0) in enumerate([(0, 2, 0), (3, 1, 2)]):
            tok, win, t1, t2 = brute.pick(logits[s0:s0 + n + 1], rel[e0:e0 + n].astype(np.float64).tolist(),
                                          2.5, beta[e0:e0 + n])
            assert (res.tokens[b], res.winners[b]) == (tok, win)
            assert res.top1[b] == pytest.approx(t1, abs=1e-12) and res.top2[b] == pytest.approx(t2, abs=1e-12)


def test_shared_history_append_reaches_every_expert():
    # the new token's K/V row is appended to every sequence before attending:
    # a new key aligned with the query dominates, so every output is ~ v_new
    rng = np.random.default_rng(22)
    Hq, Hkv, D, L = 2, 1, 8, 1
    lens = [3, 5, 4]
    ck = [rng.standard_normal((L, T, Hkv, D)) for T in lens]
    cv = [rng.standard_normal((L, T, Hkv, D)) for T in lens]
    orc = O.Oracle(n_layers=L, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, vocab=5, dtype="f32",
                   n_experts=[2], cache_k=lambda s, l: ck[s][l], cache_v=lambda s, l: cv[s][l],
                   relevance=[0.5, 0.5], beta=[0.0, 0.0])
    q = np.zeros((3, L, Hq, D), dtype=np.float32)
    q[..., 0] = 1.0
    kn = np.zeros((3, L, Hkv, D), dtype=np.float32)
    kn[..., 0] = 200.0
    vn = rng.standard_normal((3, L, Hkv, D)).astype(np.float32)
    res = orc.step(q, kn, vn, np.ones((5, Hq * D), dtype=np.float32))
    for s in range(3):
        assert np.allclose(res.attn[0][s], np.repeat(vn[s, 0], Hq, axis=0), atol=1e-12)


def test_dynamic_beta_frozen_after_first_step():
    rng = np.random.default_rng(23)
    Hq, Hkv, D, L, V = 2, 1, 4, 1, 30
    lens = [2, 6, 3]
    ck = [rng.standard_normal((L, T, Hkv, D)).astype(np.float32) for T in lens]
    cv = [rng.standard_normal((L, T, Hkv, D)).astype(np.float32) for T in lens]
    W = rng.standard_normal((V, Hq * D)).astype(np.float32)
    orc = O.Oracle(n_layers=L, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, vocab=V, dtype="f32",
                   n_experts=[2], cache_k=lambda s, l: ck[s][l], cache_v=lambda s, l: cv[s][l],
                   relevance=[0.3, 0.6])
    r0 = orc.step(*[rng.standard_normal(sh).astype(np.float32) for sh in
                    ((3, L, Hq, D), (3, L, Hkv, D), (3, L, Hkv, D))], W)
    r1 = orc.step(*[rng.standard_normal(sh).astype(np.float32) for sh in
                    ((3, L, Hq, D), (3, L, Hkv, D), (3, L, Hkv, D))], W)
    assert np.array_equal(r0.beta, r1.beta)
    assert np.allclose(r0.beta, O.dynamic_beta(r0.logits))
    assert not np.allclose(O.dynamic_beta(r1.logits), r0.beta)


# -------------------------------------------------------------- geometry (paper)

def test_kv_storage_figure_of_the_paper():
    g = golden("kv_storage_loft_hotpotqa.json")
    m = g["model_geometry"]
    per_token = O.kv_bytes_per_token(m["n_layers"], m["n_kv_heads"], m["head_dim"], m["bytes_per_value"])
    assert per_token == 128 * 1024
    total = g["passages"] * g["tokens_per_passage"] * per_token
    assert round(total / 2 ** 30, 2) == g["reported_gb"]


# ---------------------------------------------------------------- relevance
# Appendix B normalisation and fusion, pinned by closed forms and invariants.

def test_dense_and_colbert_rescaling_closed_forms():
    for mode in ("dense", "colbert"):
        r = O.normalise_retrieval([-1.0, 0.0, 0.5, -3.0, 1.0, 7.0], mode)
        assert r[0] == 0.0 and r[1] == 0.5 and r[2] == 0.75 and r[3] == 0.0
        assert r[4] == r[5] == 1.0 - 1e-8          # clipped below 1
    s = np.linspace(-1, 1, 101)
    assert np.all(np.diff(O.normalise_retrieval(s, "dense")) > 0)


def test_sparse_arctan_closed_forms():
    r = O.normalise_retrieval([0.0, 1.0, math.sqrt(3.0), 1.0 / math.sqrt(3.0), -5.0, 1e12], "sparse")
    assert r[0] == 0.0 and r[4] == 0.0                  # max(s, 0)
    assert abs(r[1] - 0.5) < 1e-15                      # atan(1) = pi/4
    assert abs(r[2] - 2.0 / 3.0) < 1e-15                # atan(sqrt 3) = pi/3
    assert abs(r[3] - 1.0 / 3.0) < 1e-15                # atan(1/sqrt 3) = pi/6
    assert r[5] == 1.0 - 1e-8
    assert np.all(np.diff(O.normalise_retrieval(np.linspace(0, 50, 200), "sparse")) > 0)


def test_reranker_sigmoid_closed_forms():
    r = O.normalise_reranker([0.0, math.log(3.0), -math.log(3.0), -800.0, 800.0])
    assert r[0] == 0.5
    assert abs(r[1] - 0.75) < 1e-15 and abs(r[2] - 0.25) < 1e-15
    assert r[3] == 0.0 and r[4] == 1.0 - 1e-8
    z = np.linspace(-6, 6, 25)
    assert np.allclose(O.normalise_reranker(z) + O.normalise_reranker(-z), 1.0, atol=1e-15)


def test_harmonic_mean_fusion():
    assert O.fuse_relevance(0.0, 0.7) == 0.0
    # harmonic mean of 1/3 and 1 is 1/2; eps only perturbs the 9th digit
    assert abs(O.fuse_relevance(1.0 / 3.0, 1.0) - 0.5) < 1e-8
    a, b = np.random.default_rng(0).random((2, 50))
    assert np.array_equal(O.fuse_relevance(a, b), O.fuse_relevance(b, a))
    h = O.fuse_relevance(a, b)
    assert np.all(h <= np.maximum(a, b)) and np.all(h >= np.minimum(a, b) - 1e-7)
    # equal inputs give (almost) that value; retrieval alone without a reranker
    assert np.allclose(O.fuse_relevance(a, a), a, atol=1e-7)
    assert np.array_equal(O.relevance([0.2, -0.4], "dense"), O.normalise_retrieval([0.2, -0.4], "dense"))


# ------------------------------------------------- aggregation variants (NEXT-2)
# MoE / PoE (Appendix C.4, read as in pced_oracle.aggregate_query), pinned by
# reductions to the Max rule and to single distributions, by invariants of
# mixtures and products of distributions, and by a scalar-loop brute force.

def _rand_query(rng, N, V, scale=3.0):
    rows = rng.normal(0, scale, (N + 1, V))
    return rows, rng.random(N), rng.random(N)


@pytest.mark.parametrize("rule", ["moe", "poe"])
def test_aggregation_with_one_expert_is_the_max_rule(rule):
    rng = np.random.default_rng(21)
    for _ in range(5):
        rows, rel, beta = _rand_query(rng, 1, 97)
        sel = O.aggregate_query(rows, rel, 2.5, beta, rule)
        ref = O.fuse_query(rows, rel, 2.5, beta)
        assert sel.token == ref.token and sel.winner == 1
        c = (1 + beta[0]) * rows[1] - beta[0] * rows[0]
        assert abs(sel.top1 - O.log_softmax(c)[sel.token]) < 1e-12


@pytest.mark.parametrize("rule", ["moe", "poe"])
def test_identical_experts_reduce_to_one_distribution(rule):
    rng = np.random.default_rng(22)
    rows, rel, _ = _rand_query(rng, 4, 80)
    rows[2:] = rows[1]
    beta = np.full(4, 0.4)
    sel = O.aggregate_query(rows, rel, 2.5, beta, rule)
    c = 1.4 * rows[1] - 0.4 * rows[0]
    assert sel.token == int(np.argmax(c))
    assert abs(sel.top1 - O.log_softmax(c).max()) < 1e-12


def test_mixture_is_a_distribution_and_product_is_below_it():
    rng = np.random.default_rng(23)
    rows, rel, beta = _rand_query(rng, 6, 50)
    s = rows
    c = (1 + beta[:, None]) * s[1:] - beta[:, None] * s[0][None, :]
    lp = O.log_softmax(c)
    w = O.expert_weights(rel, 2.5)
    assert abs(w.sum() - 1.0) < 1e-15
    moe = np.log(np.sum(w[:, None] * np.exp(lp), axis=0))
    poe = np.sum(w[:, None] * lp, axis=0)
    assert abs(np.exp(moe).sum() - 1.0) < 1e-12           # a mixture of distributions sums to 1
    assert np.all(poe <= moe + 1e-12)                        # weighted AM-GM
    assert O.aggregate_query(rows, rel, 2.5, beta, "moe").top1 == pytest.approx(moe.max(), abs=1e-12)
    assert O.aggregate_query(rows, rel, 2.5, beta, "poe").top1 == pytest.approx(poe.max(), abs=1e-12)


def test_weights_follow_the_prior_and_a_dominant_expert_decides():
    rel = np.array([0.2, 0.8, 0.4])
    w = O.expert_weights(rel, 2.0)
    assert np.allclose(w, rel ** 2 / np.sum(rel ** 2), rtol=1e-14)
    assert np.allclose(O.expert_weights(rel, 0.0), 1.0 / 3.0)
    rng = np.random.default_rng(24)
    rows, _, _ = _rand_query(rng, 3, 64)
    rel = np.array([0.01, 1.0, 0.01])
    for rule in ("moe", "poe"):
        sel = O.aggregate_query(rows, rel, 60.0, np.zeros(3), rule)
        assert sel.token == int(np.argmax(rows[2])) and sel.winner == 2


@pytest.mark.parametrize("rule", ["moe", "poe"])
def test_aggregation_permutation_invariant(rule):
    rng = np.random.default_rng(25)
    rows, rel, beta = _rand_query(rng, 5, 70)
    perm = rng.permutation(5)
    a = O.aggregate_query(rows, rel, 2.5, beta, rule)
    b = O.aggregate_query(np.concatenate([rows[:1], rows[1:][perm]]), rel[perm], 2.5, beta[perm], rule)
    assert a.token == b.token and perm[b.winner - 1] + 1 == a.winner
    assert abs(a.top1 - b.top1) < 1e-12


@pytest.mark.parametrize("rule", ["moe", "poe"])
@pytest.mark.parametrize("N,V", [(1, 5), (2, 7), (5, 13)])
def test_aggregation_brute_force_agrees(rule, N, V):
    rng = np.random.default_rng(26 + N)
    rows, rel, beta = _rand_query(rng, N, V)
    tok, exp_k, top1, top2 = brute.aggregate_pick(rows.tolist(), rel.tolist(), 1.7, beta.tolist(), rule)
    sel = O.aggregate_query(rows, rel, 1.7, beta, rule)
    assert (sel.token, sel.winner) == (tok, exp_k)
    assert abs(sel.top1 - top1) < 1e-12 and abs(sel.top2 - top2) < 1e-12


def test_scalar_beta_is_the_mean_of_the_divergences():
    rng = np.random.default_rng(27)
    rows, _, _ = _rand_query(rng, 4, 40, scale=1.0)
    per = O.dynamic_beta(rows)
    sc = O.dynamic_beta(rows, scalar=True)
    assert np.allclose(sc, per.mean()) and sc.shape == per.shape
    one = rows[:2]
    assert np.array_equal(O.dynamic_beta(one, scalar=True), O.dynamic_beta(one))
