"""pced_stream_read: the XOR of every 32-bit word it streams is the host's XOR
of the same seeded bytes, for empty, single-unit, ragged and large sizes and
for a source inside an allocation; a read past the end of the device
allocation (torch rounds its segments up, so a terabyte here) is rejected
before any launch."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _xor(words: np.ndarray) -> int:
    return int(np.bitwise_xor.reduce(words, initial=np.uint32(0)))


@pytest.mark.parametrize("n_words", [0, 4, 4 * 1000 + 4 * 37, 4 * (1 << 20) + 12, (64 << 20) // 4 + 4 * 5])
def test_stream_read_xor_matches_host(n_words):
    from paper_2601_08670_amd import _lib
    rng = np.random.default_rng(1234 + n_words)
    words = rng.integers(0, 2**32, size=n_words, dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(words.view(np.int32)).to(DEV)
    out = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    _lib.pced_stream_read(src, 4 * n_words, out)
    torch.cuda.synchronize()
    assert int(out.cpu().numpy().view(np.uint32)[0]) == _xor(words)


def test_stream_read_inside_an_allocation_and_bounds():
    from paper_2601_08670_amd import _lib
    rng = np.random.default_rng(7)
    words = rng.integers(0, 2**32, size=4096, dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(words.view(np.int32)).to(DEV)
    out = torch.zeros(1, dtype=torch.int32, device=DEV)
    _lib.pced_stream_read(src[8:], 4 * 1000, out)          # 32 bytes in, 4000 bytes
    torch.cuda.synchronize()
    assert int(out.cpu().numpy().view(np.uint32)[0]) == _xor(words[8:1008])
    with pytest.raises(_lib.PcedError, match="past the end"):
        _lib.pced_stream_read(src[8:], 1 << 40, out)           # far beyond any allocation
