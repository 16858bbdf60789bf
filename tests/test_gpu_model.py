"""GPU decoder stack around the step (pced_model_prefill / _step / _generate)
against the CPU decoder oracle (oracle/model.py), element by element on the
same seeded weights, caches and tokens. Every GPU computation goes through the
C ABI; expected values come only from the oracle.

Token contract here: the decoder stack rounds activations to bf16 at the same
points on both sides, but a value that the fp32 GPU path and the float64
oracle place on different sides of a rounding boundary moves by one bf16 ulp,
so the logits agree to the measured error e (checked against the 2e-2 bound),
not to fp32 accumulation noise. A token that differs from the oracle's is
accepted only if its oracle score is within 2 (1 + 2 beta_max) e + 1e-3 of the
best: every fused score moves by at most (1 + 2 beta) e."""
import numpy as np
import pytest

from oracle import model as OM
from oracle import pced_oracle as O
from pced_inputs import workloads as W
from pced_inputs.model import LAYER_TENSORS, ModelSpec, suffix_tokens
from tests.helpers import REL_TOL, rel_err_rows

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = REL_TOL["bf16"]
# Past the first layer the inputs themselves differ: every layer re-rounds its
# activations (q, k, v, attention output, MLP activation, the next norm's input)
# to bf16, and a value the fp32 GPU path and the float64 oracle place on opposite
# sides of a rounding boundary moves by one ulp (2^-8 relative). Measured on the
# prefilled caches at Llama-3-8B shapes: layer-0 K/V rows exact or one ulp off,
# layer-1 rows one ulp off in a few elements (median 0.44%, max 0.97% per row);
# softmax turns that into up to 2.5% in layer 1's attention output. Bound for
# everything downstream of a re-rounded activation:
TOL_DEEP = 5e-2


def _np(t):
    return t.detach().cpu().numpy()


def _setup(wl, spec, extra_tokens):
    from paper_2601_08670_amd.session import session_for_workload
    sess = session_for_workload(wl, device=DEV, extra_tokens=extra_tokens, poison=True, ffn_dim=spec.ffn_dim,
                                rope_theta=int(spec.rope_theta))
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


def _check_tokens(wl, got, ref, logits_gpu):
    """Tokens under the contract in the module docstring; returns exemptions."""
    off = wl.seq_offsets
    exempt, e0 = 0, 0
    for b, n in enumerate(wl.n_experts):
        rows = ref.logits[off[b]:off[b + 1]]
        if int(got[b]) != int(ref.tokens[b]):
            err = float(np.abs(logits_gpu[off[b]:off[b + 1]] - rows).max())
            beta = ref.beta[e0:e0 + n]
            allow = 2.0 * (1.0 + 2.0 * float(beta.max())) * err + 1e-3
            S = O.contrastive_scores(rows, beta, O.prior_term(wl.relevance[e0:e0 + n], wl.gamma)).max(axis=0)
            assert S[int(got[b])] >= S.max() - allow, (b, int(got[b]), int(ref.tokens[b]), S.max(), allow)
            exempt += 1
        e0 += n
    return exempt


def _compare_step(wl, out, ref, beta_atol=1e-2):
    g = wl.geom
    D = g.head_dim
    a = _np(out["attn_out"])
    for l, ra in ref.attn.items():
        err = rel_err_rows(a[:, l].reshape(-1, D), ra.reshape(-1, D))
        assert err <= (TOL if l == 0 else TOL_DEEP), f"layer {l}: attention rel err {err}"
    err = rel_err_rows(_np(out["hidden"]), ref.hidden)
    assert err <= TOL_DEEP, f"residual stream rel err {err}"
    lg = _np(out["logits"])
    err = rel_err_rows(lg, ref.logits)
    assert err <= TOL_DEEP, f"logits rel err {err}"
    print(f"max rel err: attention {[round(rel_err_rows(a[:, l].reshape(-1, D), ra.reshape(-1, D)), 4) for l, ra in ref.attn.items()]}, logits {err:.4f}")
    np.testing.assert_allclose(_np(out["beta_used"]), ref.beta, rtol=0, atol=beta_atol)
    return _check_tokens(wl, _np(out["tokens"]), ref, lg)


WANT = ("attn_out", "logits", "winner", "top1", "top2", "beta_used", "hidden")


def _run(wl, spec, steps, prefill=0, seed=1):
    sess, model, Wt = _setup(wl, spec, extra_tokens=steps + prefill + 1)
    orc = _oracle(wl, spec)
    B, V = wl.n_queries, wl.geom.vocab
    lens0 = sess.lengths()
    if prefill:
        toks = suffix_tokens(seed, B, prefill, V)
        sess.ctx.pced_model_prefill(model, prefill, torch.from_numpy(toks).to(DEV))
        orc.prefill(toks)
        assert sess.lengths() == [x + prefill for x in lens0] == orc.lengths()
    tok = suffix_tokens(seed + 1, B, 1, V)[:, 0]
    exempt = 0
    for t in range(steps):
        out = sess.model_step(model, Wt, torch.from_numpy(tok.astype(np.int32)).to(DEV), want=WANT)
        torch.cuda.synchronize()
        ref = orc.step(tok)
        exempt += _compare_step(wl, out, ref)
        tok = ref.tokens.astype(np.int32)   # teacher forcing: both sides continue the oracle's history
    assert sess.lengths() == orc.lengths()
    return exempt


def test_model_steps_two_layers_two_queries():
    geom = W.Geometry(2, 8, 2, 64, 512, 3000, "bf16")
    wl = W.custom(geom, [3, 2], [40, 300, 17, 5, 129], amateur_len=16, steps=3, seed=21)
    spec = ModelSpec(geom, ffn_dim=1024, rope_theta=10000.0, seed=21)
    assert _run(wl, spec, steps=3) <= 1


def test_model_prefill_then_steps_shuffled_pages():
    geom = W.Geometry(1, 8, 2, 64, 512, 2000, "bf16")
    wl = W.custom(geom, [2], [20, 33], amateur_len=5, steps=2, seed=22, shuffle_pages=True)
    spec = ModelSpec(geom, ffn_dim=512, rope_theta=500000.0, seed=22)
    _run(wl, spec, steps=2, prefill=13)   # crosses page boundaries at 16 and 32


def test_model_many_rows_two_row_groups():
    # 57 sequences: the projections loop over two groups of 48 rows; the prefill
    # runs in chunks of 4 suffix tokens (228 rows: five row groups), then 2
    geom = W.Geometry(1, 4, 1, 64, 256, 700, "bf16")
    wl = W.custom(geom, [30, 25], list(range(3, 58)), amateur_len=7, steps=2, seed=23)
    spec = ModelSpec(geom, ffn_dim=256, rope_theta=10000.0, seed=23)
    _run(wl, spec, steps=2, prefill=10)


def test_model_llama3_8b_layer_shapes():
    # Llama-3-8B decoder dimensions (hidden 4096, 32/8 heads of 128, MLP 14336),
    # two layers, 8 documents; a 4096-token vocabulary keeps the oracle's LM head small
    geom = W.Geometry(2, 32, 8, 128, 4096, 4096, "bf16")
    rng = np.random.default_rng(24)
    wl = W.custom(geom, [8], rng.integers(100, 700, size=8).tolist(), amateur_len=64, steps=2, seed=24)
    spec = ModelSpec(geom, ffn_dim=14336, rope_theta=500000.0, seed=24)
    _run(wl, spec, steps=2, prefill=20)


def test_model_generate_follows_oracle_generation():
    geom = W.Geometry(2, 8, 2, 64, 512, 1500, "bf16")
    wl = W.custom(geom, [2, 3], [30, 64, 8, 100, 45], amateur_len=9, steps=5, seed=25)
    spec = ModelSpec(geom, ffn_dim=512, rope_theta=10000.0, seed=25)
    sess, model, Wt = _setup(wl, spec, extra_tokens=6)
    first = suffix_tokens(3, wl.n_queries, 1, geom.vocab)[:, 0].astype(np.int32)
    toks = torch.empty((wl.n_queries, 5), dtype=torch.int32, device=DEV)
    last = sess.out_buffers(("logits",))
    sess.ctx.pced_model_generate(model, Wt, 5, torch.from_numpy(first).to(DEV), toks, last)
    torch.cuda.synchronize()
    got = _np(toks)
    orc = _oracle(wl, spec)
    prev = first
    ref_tok, gaps = [], []
    for t in range(5):
        r = orc.step(prev)
        ref_tok.append(r.tokens.copy())
        gaps.append(r.gaps.copy())
        prev = r.tokens.astype(np.int32)
    ref_tok, gaps = np.array(ref_tok).T, np.array(gaps).T
    for b in range(wl.n_queries):
        for t in range(5):
            if got[b, t] != ref_tok[b, t]:
                # a near-tie may flip; the two histories differ from there on
                assert gaps[b, t] < 5e-2, (b, t, got[b], ref_tok[b], gaps[b])
                break
    if (got == ref_tok).all():   # same history: the last step's logits are comparable
        assert rel_err_rows(_np(last["logits"]), r.logits) <= TOL_DEEP
    assert sess.lengths() == [x + 5 for x in wl.cache_len.tolist()]


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
