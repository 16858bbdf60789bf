"""Split-state merge of the bf16 decode step: every layer but the last is merged
inside the next layer's attention launch, the last one by the merge kernel.

Both merges follow Section 3's attention (the log-sum-exp combination of the
partial states of a sequence cut into chunks), with the same operations in the
same order, so identical inputs in every layer must give bit-identical layer
outputs; the last layer's output is also checked against the oracle. All GPU
work goes through the C ABI; expected values come only from the oracle."""
import numpy as np
import pytest

from pced_inputs import workloads as W
from tests.helpers import REL_TOL, make_oracle, rel_err_rows

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"

CASES = [
    # (name, one-layer geometry, n_experts, expert lengths, amateur length, chunk cap)
    # a 5000-token expert cut into ~300 chunks: more than 16 splits (several merge groups)
    ("more-than-16-splits", W.Geometry(1, 4, 2, 64, 256, 300, "bf16"), [1], [5000], 8, 0),
    # two chunks for 7 sequences: 56 merge items on 4 waves (several items per wave)
    ("several-items-per-wave", W.Geometry(1, 8, 2, 128, 1024, 600, "bf16"), [6],
     [250, 9, 15, 17, 120, 48], 20, 2),
    # Llama-3-8B heads, 6 experts of 300-700 tokens plus the amateur
    ("llama-heads", W.Geometry(1, 32, 8, 128, 4096, 512, "bf16"), [6], [700, 300, 512, 650, 333, 480], 64, 0),
]


@pytest.mark.parametrize("name,geom,n_exp,lens,am,cap", CASES, ids=[c[0] for c in CASES])
def test_merge_in_next_launch_equals_merge_kernel(name, geom, n_exp, lens, am, cap):
    from paper_2601_08670_amd.session import PcedSession
    L, steps = 3, 2
    wl = W.custom(geom, n_exp, lens, am, steps=steps, seed=31)
    need = wl.pages_needed(steps)
    maxpps = int(need.max())
    sess = PcedSession(n_layers=L, n_q_heads=geom.n_q_heads, n_kv_heads=geom.n_kv_heads,
                       head_dim=geom.head_dim, vocab=geom.vocab, dtype=geom.dtype, max_queries=wl.n_queries,
                       max_seqs=wl.n_seqs, max_pages=int(need.sum()), max_pages_per_seq=maxpps,
                       device=DEV, poison=True, max_attn_chunks=cap)
    # the one-layer caches repeated in every layer
    src_k = [wl.kcache_device(s, DEV).expand(L, -1, -1, -1).contiguous() for s in range(wl.n_seqs)]
    src_v = [wl.vcache_device(s, DEV).expand(L, -1, -1, -1).contiguous() for s in range(wl.n_seqs)]
    sess.load(wl.n_experts, wl.cache_len.tolist(), src_k, src_v, wl.relevance.tolist(), gamma=wl.gamma,
              page_table=wl.page_table(steps, maxpps))
    Wt = sess.pack_lm_head(wl.lm_head_device(DEV))
    orc = make_oracle(wl)
    Wh = wl.lm_head_host()
    D = geom.head_dim
    for t in range(steps):
        q, kn, vn = (x.expand(-1, L, -1, -1).contiguous() for x in wl.step_inputs_device(t, DEV))
        out = sess.step(q, kn, vn, Wt, want=("attn_out", "logits"))
        torch.cuda.synchronize()
        a = out["attn_out"]
        assert torch.isfinite(a).all(), f"step {t}: non-finite layer output"
        for l in range(L - 1):  # merged in the next launch vs merged by the merge kernel
            assert torch.equal(a[:, l], a[:, L - 1]), f"step {t}: layer {l} differs from the last layer"
        ref = orc.step(*wl.step_inputs_host(t), Wh)
        err = rel_err_rows(a[:, L - 1].cpu().numpy().reshape(-1, D), ref.attn[0].reshape(-1, D))
        assert err <= REL_TOL["bf16"], f"step {t}: attention rel err {err}"
        err = rel_err_rows(out["logits"].cpu().numpy(), ref.logits)
        assert err <= REL_TOL["bf16"], f"step {t}: logits rel err {err}"
    assert sess.lengths() == [x + steps for x in wl.cache_len.tolist()]
