"""pced_lmhead_noalloc (no context, no workspace: its scratch is a
library-owned device array) against pced_lmhead on the same inputs, through the
C ABI: two calls in a row, the second with fewer rows, and the capacity limit."""
import numpy as np
import pytest

from pced_inputs import counter
from pced_inputs.workloads import device_values

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"

CASES = [
    # (dtype, vocab, q heads, head dim, rows of the two calls)
    ("bf16", 4103, 32, 128, (272, 33)),   # many-row kernel, then the 48-row kernel
    ("bf16", 5000, 8, 64, (100, 20)),
    ("f32", 1000, 4, 64, (9, 5)),
]


@pytest.mark.parametrize("dtype,vocab,hq,d,rows", CASES, ids=[f"{c[0]}-{c[1]}" for c in CASES])
def test_lmhead_noalloc_matches_lmhead(dtype, vocab, hq, d, rows):
    from paper_2601_08670_amd import _lib
    from paper_2601_08670_amd.session import PcedSession
    hidden = hq * d
    sess = PcedSession(n_layers=1, n_q_heads=hq, n_kv_heads=hq, head_dim=d, vocab=vocab, dtype=dtype,
                       max_queries=1, max_seqs=max(rows), max_pages=1, max_pages_per_seq=1, device=DEV)
    w = device_values(counter.key(7, 13), 0, vocab * hidden, 0.02, dtype, DEV).reshape(vocab, hidden)
    wp = sess.pack_lm_head(w)
    for i, n in enumerate(rows):
        x = device_values(counter.key(7, 40, i), 0, n * hidden, 1.0, dtype, DEV).reshape(n, hidden)
        ref = torch.empty((n, vocab), dtype=torch.float32, device=DEV)
        got = torch.full((n, vocab), float("nan"), dtype=torch.float32, device=DEV)
        sess.ctx.pced_lmhead(x, n, wp, ref)
        _lib.pced_lmhead_noalloc(sess.cfg, x, n, wp, got)
        torch.cuda.synchronize()
        assert np.array_equal(got.cpu().numpy().view(np.uint32), ref.cpu().numpy().view(np.uint32)), (i, n)


def test_lmhead_noalloc_capacity_limit():
    from paper_2601_08670_amd import _lib
    cfg = _lib.make_config(n_layers=1, n_q_heads=32, n_kv_heads=8, head_dim=128, vocab=4096, dtype="bf16",
                           max_queries=1, max_seqs=2, max_pages=1, max_pages_per_seq=1)
    x = torch.zeros((513, 4096), dtype=torch.int16, device=DEV)
    out = torch.empty((513, 4096), dtype=torch.float32, device=DEV)
    wp = torch.zeros(_lib.pced_lm_head_bytes(cfg), dtype=torch.uint8, device=DEV)
    with pytest.raises(_lib.PcedError, match="CAPACITY"):
        _lib.pced_lmhead_noalloc(cfg, x, 513, wp, out)    # 528 padded rows x 8 KiB > 4 MiB
    _lib.pced_lmhead_noalloc(cfg, x, 512, wp, out)        # exactly 4 MiB
    torch.cuda.synchronize()
    assert torch.count_nonzero(out[:512]).item() == 0
