"""PCED decode step on AMD Instinct MI355X (gfx950).

Parallel Context-of-Experts Decoding (arXiv 2601.08670): N document experts and
one no-context amateur decode in parallel over their own KV caches; their logits
are fused by a retrieval-aware contrastive rule into one token per step.

``_lib`` is the ctypes binding of the C ABI (include/pced.h); ``session`` sizes
and allocates the caller-owned device buffers with torch. The HIP library is
loaded on first use and its absence is an error.
"""
from . import _lib  # noqa: F401
from ._lib import PcedError, load_library  # noqa: F401
