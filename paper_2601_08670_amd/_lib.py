"""ctypes binding of libpced (include/pced.h), with the same entry-point names.

Argument marshalling only: torch supplies device memory and the current stream;
every step of the decode path runs in the library's HIP kernels. There is no
fallback: if the shared library is missing or fails to load, this module raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
# PCED_LIBRARY may name another build of the same library (e.g. a debug build)
LIB_PATH = os.environ.get("PCED_LIBRARY") or os.path.join(_HERE, "libpced.so")

PCED_F32, PCED_BF16 = 0, 1
PCED_NORM_NONE, PCED_NORM_RMS = 0, 1
STATUS = {0: "OK", 1: "INVALID_ARG", 2: "CAPACITY", 3: "HIP", 4: "UNSUPPORTED", 5: "STATE"}
PROF_CLASSES = ("append", "attn", "lmhead", "beta", "fuse", "synth", "combine", "embed", "qkv", "oproj",
                "gateup", "down", "fuse_merge")

EXPORTED = ("pced_pool_bytes", "pced_lm_head_bytes", "pced_pack_lm_head", "pced_workspace_bytes", "pced_create", "pced_destroy", "pced_last_error",
            "pced_load_caches", "pced_step", "pced_generate", "pced_lmhead", "pced_fuse",
            "pced_get_lengths", "pced_profile_enable", "pced_profile_read", "pced_relevance",
            "pced_model_bytes", "pced_pack_model_layer", "pced_pack_model_globals", "pced_model_prefill",
            "pced_model_step", "pced_model_generate", "pced_read_cache", "pced_lmhead_noalloc",
            "pced_stream_read")


class PcedError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class pced_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "n_q_heads", "n_kv_heads", "head_dim", "hidden", "vocab", "dtype", "page_size",
        "max_queries", "max_seqs", "max_pages", "max_pages_per_seq", "norm", "max_attn_chunks",
        "aggregation", "beta_scalar", "ffn_dim", "rope_theta")]


class pced_step_out(ctypes.Structure):
    _fields_ = [("attn_out", ctypes.c_void_p), ("logits", ctypes.c_void_p), ("winner", ctypes.c_void_p),
                ("top1", ctypes.c_void_p), ("top2", ctypes.c_void_p), ("beta_used", ctypes.c_void_p),
                ("hidden", ctypes.c_void_p), ("resid_trace", ctypes.c_void_p), ("qkv_trace", ctypes.c_void_p),
                ("act_trace", ctypes.c_void_p)]

STEP_OUT_FIELDS = tuple(n for n, _ in pced_step_out._fields_)


class pced_synth(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("first_token", ctypes.c_int32)]


class pced_profile(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64 * 13), ("total_ms", ctypes.c_double * 13),
                ("bytes", ctypes.c_double * 13), ("flops", ctypes.c_double * 13)]


_lib = None


def load_library() -> ctypes.CDLL:
    """Load libpced.so from the package directory (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() or "
                          "python paper_2601_08670_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    P, I, V = ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p
    sig = {
        "pced_pool_bytes": (ctypes.c_size_t, [ctypes.POINTER(pced_config)]),
        "pced_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(pced_config)]),
        "pced_lm_head_bytes": (ctypes.c_size_t, [ctypes.POINTER(pced_config)]),
        "pced_pack_lm_head": (I, [ctypes.POINTER(pced_config), P, P, V]),
        "pced_create": (I, [ctypes.POINTER(pced_config), P, ctypes.c_size_t, ctypes.POINTER(P)]),
        "pced_destroy": (None, [P]),
        "pced_last_error": (ctypes.c_char_p, []),
        "pced_load_caches": (I, [P, I, P, P, P, P, P, P, P, I, P, ctypes.c_float, P, V]),
        "pced_step": (I, [P, P, P, P, P, P, ctypes.POINTER(pced_step_out), V]),
        "pced_generate": (I, [P, I, ctypes.POINTER(pced_synth), P, P, ctypes.POINTER(pced_step_out), V]),
        "pced_lmhead": (I, [P, P, I, P, P, V]),
        "pced_fuse": (I, [P, P, I, P, ctypes.POINTER(pced_step_out), V]),
        "pced_get_lengths": (I, [P, P, I]),
        "pced_profile_enable": (I, [P, I]),
        "pced_profile_read": (I, [P, ctypes.POINTER(pced_profile)]),
        "pced_relevance": (I, [I, I, P, P, P]),
        "pced_model_bytes": (ctypes.c_size_t, [ctypes.POINTER(pced_config)]),
        "pced_pack_model_layer": (I, [ctypes.POINTER(pced_config), I, P, P, V]),
        "pced_pack_model_globals": (I, [ctypes.POINTER(pced_config), P, P, P, V]),
        "pced_model_prefill": (I, [P, P, I, P, V]),
        "pced_model_step": (I, [P, P, P, P, P, ctypes.POINTER(pced_step_out), V]),
        "pced_model_generate": (I, [P, P, P, I, P, P, ctypes.POINTER(pced_step_out), V]),
        "pced_read_cache": (I, [P, I, I, I, I, P, P, V]),
        "pced_lmhead_noalloc": (I, [ctypes.POINTER(pced_config), P, I, P, P, V]),
        "pced_stream_read": (I, [P, ctypes.c_size_t, P, V]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        raise PcedError(status, load_library().pced_last_error().decode())


def make_config(*, n_layers, n_q_heads, n_kv_heads, head_dim, vocab, dtype, max_queries, max_seqs,
                max_pages, max_pages_per_seq, norm="rms", hidden=None, max_attn_chunks=0, aggregation="max",
                beta_scalar=False, ffn_dim=0, rope_theta=500000) -> pced_config:
    return pced_config(
        n_layers=n_layers, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads, head_dim=head_dim,
        hidden=hidden if hidden is not None else n_q_heads * head_dim, vocab=vocab,
        dtype=PCED_BF16 if dtype == "bf16" else PCED_F32, page_size=16, max_queries=max_queries,
        max_seqs=max_seqs, max_pages=max_pages, max_pages_per_seq=max_pages_per_seq,
        norm=PCED_NORM_RMS if norm == "rms" else PCED_NORM_NONE, max_attn_chunks=max_attn_chunks,
        aggregation=AGGREGATIONS[aggregation], beta_scalar=int(bool(beta_scalar)), ffn_dim=ffn_dim,
        rope_theta=int(rope_theta))


def pced_pool_bytes(cfg: pced_config) -> int:
    return load_library().pced_pool_bytes(ctypes.byref(cfg))


def pced_workspace_bytes(cfg: pced_config) -> int:
    return load_library().pced_workspace_bytes(ctypes.byref(cfg))


def pced_lm_head_bytes(cfg: pced_config) -> int:
    return load_library().pced_lm_head_bytes(ctypes.byref(cfg))


def pced_pack_lm_head(cfg: pced_config, w, w_packed, stream=None):
    """Re-lay row-major [V][hidden] LM-head weights into the packed form the steps read."""
    _check(load_library().pced_pack_lm_head(ctypes.byref(cfg), w.data_ptr(), w_packed.data_ptr(), _stream(stream)))


def pced_lmhead_noalloc(cfg: pced_config, x, n_rows, lm_head, logits, stream=None):
    """Logits of n_rows hidden states with no context and no caller workspace."""
    _check(load_library().pced_lmhead_noalloc(ctypes.byref(cfg), x.data_ptr(), int(n_rows), lm_head.data_ptr(),
                                              logits.data_ptr(), _stream(stream)))


def pced_stream_read(src, nbytes, xor_out, stream=None):
    """XOR of the 32-bit words of nbytes of src (device), read with streaming loads."""
    _check(load_library().pced_stream_read(src.data_ptr(), int(nbytes), xor_out.data_ptr(), _stream(stream)))


def pced_model_bytes(cfg: pced_config) -> int:
    return load_library().pced_model_bytes(ctypes.byref(cfg))


def pced_pack_model_layer(cfg: pced_config, layer: int, tensors, model, stream=None):
    """Pack one decoder layer's 9 bf16 tensors (attn_norm, wq, wk, wv, wo,
    mlp_norm, w_gate, w_up, w_down; device, row-major [out][in]) into ``model``."""
    arr = (ctypes.c_void_p * 9)(*[t.data_ptr() for t in tensors])
    _check(load_library().pced_pack_model_layer(ctypes.byref(cfg), int(layer), arr, model.data_ptr(),
                                                _stream(stream)))


def pced_pack_model_globals(cfg: pced_config, embed, final_norm, model, stream=None):
    _check(load_library().pced_pack_model_globals(ctypes.byref(cfg), embed.data_ptr(), final_norm.data_ptr(),
                                                  model.data_ptr(), _stream(stream)))


SCORE_MODES = {"dense": 0, "colbert": 1, "sparse": 2}
AGGREGATIONS = {"max": 0, "moe": 1, "poe": 2}


def pced_relevance(mode: str, retrieval, reranker_logits=None):
    """Relevance scores r_k from raw retrieval scores (``mode`` dense, colbert or
    sparse) and optional reranker logits, by the library's host helper; returns a
    float32 NumPy array."""
    import numpy as np
    ret = np.ascontiguousarray(retrieval, dtype=np.float32)
    rer = None if reranker_logits is None else np.ascontiguousarray(reranker_logits, dtype=np.float32)
    if rer is not None and rer.shape != ret.shape:
        raise ValueError("retrieval and reranker_logits differ in shape")
    out = np.empty_like(ret)
    _check(load_library().pced_relevance(SCORE_MODES[mode], ret.size, ret.ctypes.data,
                                         None if rer is None else rer.ctypes.data, out.ctypes.data))
    return out


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _i32_array(values):
    arr = (ctypes.c_int32 * len(values))(*[int(v) for v in values])
    return arr


def _f32_array(values):
    return (ctypes.c_float * len(values))(*[float(v) for v in values])


def _step_out(extra: Optional[dict]):
    if not extra:
        return None
    so = pced_step_out()
    unknown = set(extra) - set(STEP_OUT_FIELDS)
    if unknown:
        raise ValueError(f"unknown step outputs {sorted(unknown)}")
    for name in STEP_OUT_FIELDS:
        t = extra.get(name)
        setattr(so, name, None if t is None else t.data_ptr())
    return ctypes.byref(so), so


class Context:
    """One PCED context: caller-owned (torch) workspace + the library's host state."""

    def __init__(self, cfg: pced_config, device="cuda"):
        import torch
        self.lib = load_library()
        self.cfg = cfg
        nbytes = pced_workspace_bytes(cfg)
        if nbytes == 0:
            raise PcedError(1, "invalid config")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        h = ctypes.c_void_p()
        _check(self.lib.pced_create(ctypes.byref(cfg), self.workspace.data_ptr(), nbytes, ctypes.byref(h)))
        self.handle = h
        self._keep = []

    def close(self):
        if getattr(self, "handle", None):
            self.lib.pced_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------- entry points
    def pced_load_caches(self, n_experts: Sequence[int], cache_len: Sequence[int], src_k, src_v,
                         k_pool, v_pool, relevance, gamma=2.5, beta=None, page_table=None,
                         reserve_tokens=0, stream=None):
        S = len(cache_len)
        ks = (ctypes.c_void_p * S)(*[t.data_ptr() for t in src_k])
        vs = (ctypes.c_void_p * S)(*[t.data_ptr() for t in src_v])
        pt = None
        if page_table is not None:
            import numpy as np
            flat = np.ascontiguousarray(page_table, dtype=np.int32).ravel()
            pt = flat.ctypes.data_as(ctypes.c_void_p)
        ne = _i32_array(n_experts)
        cl = _i32_array(cache_len)
        rel = _f32_array(relevance)
        bt = None if beta is None else _f32_array(beta)
        _check(self.lib.pced_load_caches(self.handle, len(n_experts), ne, cl, ks, vs, k_pool.data_ptr(),
                                         v_pool.data_ptr(), pt, int(reserve_tokens), rel,
                                         ctypes.c_float(gamma), bt, _stream(stream)))
        # the sources are read by the load kernel: keep them alive with the context
        self._keep = [list(src_k), list(src_v), k_pool, v_pool]

    def pced_step(self, q, k_new, v_new, lm_head, tokens_out, extra: Optional[dict] = None, stream=None):
        so = _step_out(extra)
        _check(self.lib.pced_step(self.handle, q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(),
                                  lm_head.data_ptr(), tokens_out.data_ptr(), so[0] if so else None,
                                  _stream(stream)))

    def pced_generate(self, n_steps, seed, first_token, lm_head, tokens_out, last_extra=None, stream=None):
        syn = pced_synth(seed=seed, first_token=first_token)
        so = _step_out(last_extra)
        _check(self.lib.pced_generate(self.handle, int(n_steps), ctypes.byref(syn), lm_head.data_ptr(),
                                      tokens_out.data_ptr(), so[0] if so else None, _stream(stream)))

    def pced_lmhead(self, x, n_rows, lm_head, logits, stream=None):
        _check(self.lib.pced_lmhead(self.handle, x.data_ptr(), int(n_rows), lm_head.data_ptr(),
                                    logits.data_ptr(), _stream(stream)))

    def pced_fuse(self, logits, refresh_beta, tokens_out, extra: Optional[dict] = None, stream=None):
        so = _step_out(extra)
        _check(self.lib.pced_fuse(self.handle, logits.data_ptr(), int(refresh_beta), tokens_out.data_ptr(),
                                  so[0] if so else None, _stream(stream)))

    def pced_model_prefill(self, model, n_tokens, tokens, stream=None):
        _check(self.lib.pced_model_prefill(self.handle, model.data_ptr(), int(n_tokens), tokens.data_ptr(),
                                           _stream(stream)))

    def pced_model_step(self, model, lm_head, in_tokens, tokens_out, extra: Optional[dict] = None, stream=None):
        so = _step_out(extra)
        _check(self.lib.pced_model_step(self.handle, model.data_ptr(), lm_head.data_ptr(), in_tokens.data_ptr(),
                                        tokens_out.data_ptr(), so[0] if so else None, _stream(stream)))

    def pced_model_generate(self, model, lm_head, n_steps, first_tokens, tokens_out, last_extra=None,
                            stream=None):
        so = _step_out(last_extra)
        _check(self.lib.pced_model_generate(self.handle, model.data_ptr(), lm_head.data_ptr(), int(n_steps),
                                            first_tokens.data_ptr(), tokens_out.data_ptr(), so[0] if so else None,
                                            _stream(stream)))

    def pced_read_cache(self, seq, layer, start, count, k_out, v_out, stream=None):
        _check(self.lib.pced_read_cache(self.handle, int(seq), int(layer), int(start), int(count), k_out.data_ptr(),
                                        v_out.data_ptr(), _stream(stream)))

    def pced_get_lengths(self, n_seqs):
        out = (ctypes.c_int32 * n_seqs)()
        _check(self.lib.pced_get_lengths(self.handle, out, n_seqs))
        return list(out)

    def pced_profile_enable(self, on: bool):
        _check(self.lib.pced_profile_enable(self.handle, int(bool(on))))

    def pced_profile_read(self) -> dict:
        p = pced_profile()
        _check(self.lib.pced_profile_read(self.handle, ctypes.byref(p)))
        return {name: {"launches": p.launches[i], "ms": p.total_ms[i], "bytes": p.bytes[i], "flops": p.flops[i]}
                for i, name in enumerate(PROF_CLASSES)}
