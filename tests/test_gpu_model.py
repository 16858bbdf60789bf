"""GPU decoder stack around the step (pced_model_prefill / _step / _generate)
against the CPU decoder oracle (oracle/model.py), stage by stage, on the same
seeded weights, caches and tokens. Every GPU computation goes through the C ABI;
expected values come only from the oracle.

Stage-wise parity. Both sides round activations to bf16 at the same points, but
a value that the fp32 GPU path and the float64 oracle place on opposite sides of
a bf16 rounding boundary moves by one ulp; fed back into the next layer, such a
difference would be amplified by the softmax and compared against a different
input. So every stage of every layer is checked with the GPU's own inputs (the
step's per-layer traces): QKV + RoPE from the GPU's residual stream, attention
from the GPU's q over the GPU's cache (the oracle's cache is taught every row
the GPU appended), the O projection from the GPU's attention output, the MLP
activation and the down projection from the GPU's residual stream and
activation, the logits from the GPU's final residual stream. Each is held to the
bf16 contract of 2e-2 (per row: max abs error / max abs reference), and the
chosen token must equal the oracle's (given the GPU's final state) unless the
oracle's top-2 gap is below 1e-3.

The prefill has no per-layer trace: there the oracle runs the suffix tokens one
at a time with its own residual stream, its cache taught the GPU's K/V rows, and
the GPU's rows (read back from the pool) are held to 2e-2 against the oracle's
own rows at every layer and position."""
import numpy as np
import pytest

from oracle import model as OM
from oracle.pced_oracle import decode_stored
from pced_inputs import workloads as W
from pced_inputs.model import LAYER_TENSORS, ModelSpec, suffix_tokens
from tests.helpers import REL_TOL, beta_tol, check_tokens, rel_err_rows

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = REL_TOL["bf16"]


def _np(t):
    return t.detach().cpu().numpy()


def _bf16(t):
    """Decoded float64 values of a device tensor of bf16 bits (int16)."""
    return decode_stored(_np(t).view(np.uint16), "bf16")


def _setup(wl, spec, extra_tokens, max_attn_chunks=0):
    from paper_2601_08670_amd.session import session_for_workload
    sess = session_for_workload(wl, device=DEV, extra_tokens=extra_tokens, poison=True, ffn_dim=spec.ffn_dim,
                                rope_theta=int(spec.rope_theta), max_attn_chunks=max_attn_chunks)
    model = sess.pack_model(lambda l: [spec.device(n, l, DEV) for n in LAYER_TENSORS],
                            spec.device("embed", 0, DEV), spec.device("final_norm", 0, DEV))
    Wt = sess.pack_lm_head(wl.lm_head_device(DEV))
    torch.cuda.synchronize()
    return sess, model, Wt


def _oracle(wl, spec):
    g = wl.geom
    return OM.ModelOracle(
        n_layers=g.n_layers, n_q_heads=g.n_q_heads, n_kv_heads=g.n_kv_heads, head_dim=g.head_dim, vocab=g.vocab,
        rope_theta=spec.rope_theta, n_experts=wl.n_experts, cache_k=lambda s, l: wl.kcache_host(s, l),
        cache_v=lambda s, l: wl.vcache_host(s, l), weights=lambda n, l: spec.host(n, l),
        embed=lambda rows: spec.host("embed", 0, rows), final_norm=spec.host("final_norm"),
        lm_head=wl.lm_head_host(), relevance=wl.relevance, gamma=wl.gamma, beta=wl.beta)


def _err(got, ref, width):
    return rel_err_rows(np.asarray(got).reshape(-1, width), np.asarray(ref).reshape(-1, width))


WANT = ("attn_out", "logits", "winner", "top1", "top2", "beta_used", "hidden", "resid_trace", "qkv_trace",
        "act_trace")


def _check_step_stages(sess, wl, orc, out):
    """Stage-wise check of one decode step (see the module docstring); the
    oracle's caches learn the rows the GPU appended. Returns (oracle selection
    given the GPU's final state, number of exempted tokens)."""
    g = wl.geom
    L, S, Hq, Hkv, D = g.n_layers, wl.n_seqs, g.n_q_heads, g.n_kv_heads, g.head_dim
    qd, kd = Hq * D, Hkv * D
    resid = _np(out["resid_trace"]).astype(np.float64)      # [L][2][S][H]
    qkv = _bf16(out["qkv_trace"])                            # [L][S][qd + 2 kd]
    act = _bf16(out["act_trace"])                            # [L][S][F]
    attn = _np(out["attn_out"]).astype(np.float64)           # [S][L][Hq][D]
    h_final = _np(out["hidden"]).astype(np.float64)
    errs = []
    for l in range(L):
        pos = [orc.K[s][l].shape[0] for s in range(S)]
        q, k, v = orc.qkv(l, resid[l, 0], pos)
        gq = qkv[l][:, :qd].reshape(S, Hq, D)
        gk = qkv[l][:, qd:qd + kd].reshape(S, Hkv, D)
        gv = qkv[l][:, qd + kd:].reshape(S, Hkv, D)
        e_qkv = max(_err(gq, q, D), _err(gk, k, D), _err(gv, v, D))
        # the appended rows, read back from the pool, are the traced ones bit for bit
        for s in range(S):
            pk, pv = sess.read_cache(s, l, pos[s], 1)
            assert np.array_equal(_bf16(pk)[0], gk[s]) and np.array_equal(_bf16(pv)[0], gv[s]), (l, s)
        orc.append_rows(l, gk, gv)
        e_att = _err(attn[:, l], orc.attend(l, gq), D)
        e_o = _err(resid[l, 1], orc.o_residual(l, resid[l, 0], attn[:, l]), g.hidden)
        e_act = _err(act[l], orc.mlp_act(l, resid[l, 1]), act.shape[-1])
        h_next = resid[l + 1, 0] if l + 1 < L else h_final
        e_down = _err(h_next, orc.down_residual(l, resid[l, 1], act[l]), g.hidden)
        errs.append((l, e_qkv, e_att, e_o, e_act, e_down))
        for name, e in zip(("qkv", "attention", "o-proj", "mlp act", "down-proj"), errs[-1][1:]):
            assert e <= TOL, f"layer {l} {name}: rel err {e}"
    logits = orc.logits_of(h_final)
    lg = _np(out["logits"])
    e_lg = rel_err_rows(lg, logits)
    assert e_lg <= TOL, f"logits rel err {e_lg}"
    print("stage errors (layer, qkv, attn, o, act, down):", [tuple(round(x, 5) for x in e) for e in errs],
          "logits", round(e_lg, 6))
    ref = orc.select(logits)
    bt = beta_tol(lg, logits, wl)
    d_beta = np.abs(_np(out["beta_used"]).astype(np.float64) - ref.beta)
    assert (d_beta <= bt).all(), (d_beta, bt)
    exempt = check_tokens(_np(out["tokens"]), logits, wl, ref.beta, ref.tokens, ref.gaps)
    win = _np(out["winner"])
    for b in range(wl.n_queries):
        if int(out["tokens"][b]) == ref.tokens[b] and ref.gaps[b] > 1e-3:
            assert win[b] == ref.winners[b], b
    return ref, exempt


def _teach_prefill(sess, wl, orc, lens0, n_tok):
    """Oracle prefill with its cache taught the GPU's rows; the GPU's rows are
    held to 2e-2 against the oracle's own at every layer and position."""
    g = wl.geom
    S, L = wl.n_seqs, g.n_layers
    rows = {}
    for s in range(S):
        for l in range(L):
            k, v = sess.read_cache(s, l, lens0[s], n_tok)
            rows[(s, l)] = (_bf16(k), _bf16(v))
    torch.cuda.synchronize()

    def kv_rows(i, l):
        return (np.stack([rows[(s, l)][0][i] for s in range(S)]), np.stack([rows[(s, l)][1][i] for s in range(S)]))

    return kv_rows


def _run(wl, spec, steps, prefill=0, seed=1, max_attn_chunks=0):
    sess, model, Wt = _setup(wl, spec, extra_tokens=steps + prefill + 1, max_attn_chunks=max_attn_chunks)
    orc = _oracle(wl, spec)
    B, V = wl.n_queries, wl.geom.vocab
    lens0 = sess.lengths()
    if prefill:
        toks = suffix_tokens(seed, B, prefill, V)
        sess.ctx.pced_model_prefill(model, prefill, torch.from_numpy(toks).to(DEV))
        torch.cuda.synchronize()
        kv_rows = _teach_prefill(sess, wl, orc, lens0, prefill)
        own = orc.prefill(toks, kv_rows)
        worst = 0.0
        for (i, l), (_, k, v) in own.items():
            gk, gv = kv_rows(i, l)
            e = max(_err(gk, k, wl.geom.head_dim), _err(gv, v, wl.geom.head_dim))
            assert e <= TOL, f"prefill token {i} layer {l}: K/V rel err {e}"
            worst = max(worst, e)
        print(f"prefill K/V max rel err {worst:.5f}")
        assert sess.lengths() == [x + prefill for x in lens0] == orc.lengths()
    tok = suffix_tokens(seed + 1, B, 1, V)[:, 0].astype(np.int32)
    exempt = 0
    for t in range(steps):
        out = sess.model_step(model, Wt, torch.from_numpy(tok).to(DEV), want=WANT)
        torch.cuda.synchronize()
        _, ex = _check_step_stages(sess, wl, orc, out)
        exempt += ex
        tok = _np(out["tokens"]).astype(np.int32)   # both sides continue with the GPU's choice
    assert sess.lengths() == orc.lengths()
    return exempt


def test_model_steps_two_layers_two_queries():
    geom = W.Geometry(2, 8, 2, 64, 512, 3000, "bf16")
    wl = W.custom(geom, [3, 2], [40, 300, 17, 5, 129], amateur_len=16, steps=3, seed=21)
    spec = ModelSpec(geom, ffn_dim=1024, rope_theta=10000.0, seed=21)
    assert _run(wl, spec, steps=3) <= 1


def test_model_steps_two_row_tiles():
    # 2 queries of 10 and 8 documents: 20 rows, so the projections run with two
    # 16-row tiles in the matrix cores' N dimension (17..32 rows)
    geom = W.Geometry(2, 8, 2, 64, 512, 1200, "bf16")
    rng = np.random.default_rng(28)
    wl = W.custom(geom, [10, 8], rng.integers(5, 400, size=18).tolist(), amateur_len=12, steps=2, seed=28)
    spec = ModelSpec(geom, ffn_dim=1536, rope_theta=10000.0, seed=28)
    assert _run(wl, spec, steps=2, prefill=5) <= 1


@pytest.mark.parametrize("experts", [[15], [16], [15, 15], [23, 23]], ids=lambda e: f"{sum(e) + len(e)}-rows")
def test_model_steps_row_tile_edges(experts):
    # 16, 17, 32 and 48 rows: the edges of one, two and three 16-row tiles in the
    # projections' N dimension (48 is the most the split-K kernel takes)
    geom = W.Geometry(2, 4, 2, 64, 256, 800, "bf16")
    rng = np.random.default_rng(29 + sum(experts))
    wl = W.custom(geom, experts, rng.integers(3, 200, size=sum(experts)).tolist(), amateur_len=8, steps=1,
                  seed=29 + sum(experts))
    spec = ModelSpec(geom, ffn_dim=512, rope_theta=10000.0, seed=29)
    assert _run(wl, spec, steps=1) <= 1


def test_model_prefill_then_steps_shuffled_pages():
    geom = W.Geometry(1, 8, 2, 64, 512, 2000, "bf16")
    wl = W.custom(geom, [2], [20, 33], amateur_len=5, steps=2, seed=22, shuffle_pages=True)
    spec = ModelSpec(geom, ffn_dim=512, rope_theta=500000.0, seed=22)
    _run(wl, spec, steps=2, prefill=13)   # crosses page boundaries at 16 and 32


def test_model_many_rows_two_row_groups():
    # 57 sequences: more than 48 rows, so the decode steps' projections go to
    # the library GEMM too; the prefill runs as one chunk of 570 rows
    geom = W.Geometry(1, 4, 1, 64, 256, 700, "bf16")
    wl = W.custom(geom, [30, 25], list(range(3, 58)), amateur_len=7, steps=2, seed=23)
    spec = ModelSpec(geom, ffn_dim=256, rope_theta=10000.0, seed=23)
    _run(wl, spec, steps=2, prefill=10)


def test_model_prefill_in_two_chunks():
    # 101 sequences: a prefill chunk holds 2304 // 101 = 22 suffix tokens, so 30
    # tokens run as chunks of 22 and 8 (the second attends to the first's rows)
    geom = W.Geometry(1, 4, 1, 64, 256, 700, "bf16")
    wl = W.custom(geom, [50, 49], [3 + (7 * i) % 40 for i in range(99)], amateur_len=5, steps=1, seed=25)
    spec = ModelSpec(geom, ffn_dim=256, rope_theta=10000.0, seed=25)
    _run(wl, spec, steps=1, prefill=30)


def test_model_llama3_8b_layer_shapes():
    # Llama-3-8B decoder dimensions (hidden 4096, 32/8 heads of 128, MLP 14336),
    # two layers, 8 documents; a 4096-token vocabulary keeps the oracle's LM head small
    geom = W.Geometry(2, 32, 8, 128, 4096, 4096, "bf16")
    rng = np.random.default_rng(24)
    wl = W.custom(geom, [8], rng.integers(100, 700, size=8).tolist(), amateur_len=64, steps=2, seed=24)
    spec = ModelSpec(geom, ffn_dim=14336, rope_theta=500000.0, seed=24)
    _run(wl, spec, steps=2, prefill=20)


@pytest.mark.parametrize("case", [
    # (name, q-heads, kv-heads, hidden, attention chunk cap)
    ("4-per-kv-head-groups-of-4", 8, 2, 512, 0),
    ("2-per-kv-head-groups-of-8-padded-items", 8, 4, 512, 5),
    ("1-per-kv-head-groups-of-16-padded-items", 4, 4, 256, 6),
    ("16-per-kv-head-token-rows", 16, 1, 1024, 0),
    ("8-per-kv-head-groups-of-2-padded-items", 16, 2, 1024, 4),
], ids=lambda c: c[0])
def test_model_prefill_token_groups(case):
    """Two layers, so the second layer's K/V rows check the first layer's
    prefill attention: the prefill's attention items are groups of suffix
    tokens of one sequence (16 / (q-heads per kv-head) tokens; 21 tokens leave a
    ragged last group), each token with its own causal end. A small chunk cap
    pads the plan's short items to the chunk length and splits the long ones,
    so later splits hold columns without keys and pages past the items' own."""
    _, hq, hkv, hidden, cap = case
    geom = W.Geometry(2, hq, hkv, 64, hidden, 1000, "bf16")
    wl = W.custom(geom, [3, 2], [40, 300, 17, 5, 129], amateur_len=9, steps=1, seed=26)
    spec = ModelSpec(geom, ffn_dim=2 * hidden, rope_theta=10000.0, seed=26)
    _run(wl, spec, steps=1, prefill=21, max_attn_chunks=cap)


@pytest.mark.parametrize("n_tok", [1, 4, 16])
def test_model_prefill_short_suffixes(n_tok):
    """Two layers, 4 q-heads per kv-head: a one-token suffix (one token per
    group), one full group, and four full groups that fill a page."""
    geom = W.Geometry(2, 8, 2, 64, 512, 900, "bf16")
    wl = W.custom(geom, [3], [16, 47, 130], amateur_len=31, steps=1, seed=30 + n_tok)
    spec = ModelSpec(geom, ffn_dim=1024, rope_theta=10000.0, seed=30)
    _run(wl, spec, steps=1, prefill=n_tok)


def test_model_prefill_token_groups_long_caches():
    """Workload-3-like caches (32 documents of 512..2048 tokens and a 64-token
    amateur, 4 q-heads per kv-head) with a 32-token suffix: 264 groups of 4
    tokens, the amateur's short items padded to the chunk length in the plan,
    the documents' items split over 2..6 chunks; the second layer's K/V rows
    check the first layer's attention for every token."""
    geom = W.Geometry(2, 8, 2, 128, 1024, 1000, "bf16")
    rng = np.random.default_rng(27)
    wl = W.custom(geom, [32], rng.integers(512, 2049, size=32).tolist(), amateur_len=64, steps=1, seed=27)
    spec = ModelSpec(geom, ffn_dim=2048, rope_theta=500000.0, seed=27)
    _run(wl, spec, steps=1, prefill=32)


def test_model_generate_equals_checked_steps():
    """pced_model_generate (tokens fed back on the device) against a twin
    session stepping with pced_model_step on the tokens it chose itself, each
    step checked stage-wise: same tokens, same final logits bit for bit."""
    geom = W.Geometry(2, 8, 2, 64, 512, 1500, "bf16")
    wl = W.custom(geom, [2, 3], [30, 64, 8, 100, 45], amateur_len=9, steps=5, seed=25)
    spec = ModelSpec(geom, ffn_dim=512, rope_theta=10000.0, seed=25)
    n = 5
    sess, model, Wt = _setup(wl, spec, extra_tokens=n + 1)
    twin, model_b, Wt_b = _setup(wl, spec, extra_tokens=n + 1)
    first = suffix_tokens(3, wl.n_queries, 1, geom.vocab)[:, 0].astype(np.int32)
    toks = torch.empty((wl.n_queries, n), dtype=torch.int32, device=DEV)
    last = sess.out_buffers(("logits", "top1", "top2"))
    sess.ctx.pced_model_generate(model, Wt, n, torch.from_numpy(first).to(DEV), toks, last)
    torch.cuda.synchronize()
    orc = _oracle(wl, spec)
    tok = first
    for t in range(n):
        out = twin.model_step(model_b, Wt_b, torch.from_numpy(tok).to(DEV), want=WANT)
        torch.cuda.synchronize()
        _check_step_stages(twin, wl, orc, out)
        tok = _np(out["tokens"]).astype(np.int32)
        assert np.array_equal(tok, _np(toks[:, t])), t
    for k in ("logits", "top1", "top2"):
        assert np.array_equal(_np(last[k]).view(np.uint8), _np(out[k]).view(np.uint8)), k
    assert sess.lengths() == [x + n for x in wl.cache_len.tolist()]


def test_model_errors_before_any_launch():
    geom = W.Geometry(1, 4, 1, 64, 256, 300, "bf16")
    wl = W.custom(geom, [1], [20], amateur_len=3, steps=1, seed=26)
    spec = ModelSpec(geom, ffn_dim=256, seed=26)
    sess, model, Wt = _setup(wl, spec, extra_tokens=2)
    from paper_2601_08670_amd._lib import PcedError
    tok = torch.zeros(1, dtype=torch.int32, device=DEV)
    with pytest.raises(PcedError, match="CAPACITY"):
        sess.ctx.pced_model_prefill(model, 64, torch.zeros((1, 64), dtype=torch.int32, device=DEV))
    assert sess.lengths() == wl.cache_len.tolist()
    sess.model_step(model, Wt, tok)
    torch.cuda.synchronize()
    assert sess.lengths() == [x + 1 for x in wl.cache_len.tolist()]
