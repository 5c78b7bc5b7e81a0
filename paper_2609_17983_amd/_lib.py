"""ctypes binding of libkvr.so (include/kvr.h): the same calls, argument
marshalling only.  Every step of prefill and repair runs in the library's HIP
kernels; nothing here computes.

Device buffers are passed as integer addresses (e.g. ``tensor.data_ptr()``)
and streams as integer handles (e.g. ``torch.cuda.current_stream().cuda_stream``).
Non-OK statuses raise KvrError.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int, c_int32, c_int64, c_size_t, c_uint64, c_void_p
from typing import Optional, Sequence

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvr.so")

KVR_OK, KVR_E_ARG, KVR_E_RANGE, KVR_E_UNSUPPORTED, KVR_E_NOMEM, KVR_E_HIP = range(6)
KVR_F32, KVR_BF16 = 0, 1
KVR_EDIT_LOCAL, KVR_RANDOM = 0, 1

STATUS_NAMES = {0: "KVR_OK", 1: "KVR_E_ARG", 2: "KVR_E_RANGE", 3: "KVR_E_UNSUPPORTED", 4: "KVR_E_NOMEM",
                5: "KVR_E_HIP"}

EXPORTED = ("kvr_create", "kvr_destroy", "kvr_cache_bytes", "kvr_workspace_bytes", "kvr_prefill", "kvr_repair",
            "kvr_select", "kvr_select_to_boundary", "kvr_transplant", "kvr_score", "kvr_generate", "kvr_select_cacheblend",
            "kvr_select_attention", "kvr_select_attention_noalloc", "kvr_answer_logprob", "kvr_margin_recovery", "kvr_flipped",
            "kvr_profile_enable", "kvr_profile_read", "kvr_last_error")


class KvrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class kvr_dims(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_heads", c_int32), ("n_kv_heads", c_int32),
                ("head_dim", c_int32), ("d_ffn", c_int32), ("vocab", c_int32), ("qkv_bias", c_int32),
                ("rms_eps", c_float), ("rope_theta", c_double), ("max_ctx", c_int32), ("max_rows", c_int32),
                ("dtype", c_int)]


class kvr_layer_weights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "bq", "bk", "bv", "wo",
                                        "mlp_norm", "w_gate", "w_up", "w_down")]


class kvr_weights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p), ("layers", POINTER(kvr_layer_weights)),
                ("lm_head", c_void_p)]


class kvr_doc(ctypes.Structure):
    _fields_ = [("d_cache", c_void_p), ("n", c_int32), ("n_cap", c_int32), ("d_tokens_new", c_void_p),
                ("edit_start", c_int32), ("edit_end", c_int32), ("h_positions", POINTER(c_int32)),
                ("n_positions", c_int32), ("d_hidden_out", c_void_p)]


_lib = None


def load() -> ctypes.CDLL:
    """Load libkvr.so from the package directory; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_17983_amd.build`")
    try:  # share torch's HIP runtime when torch is present (same SONAME)
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    lib.kvr_create.argtypes = [POINTER(kvr_dims), POINTER(kvr_weights), POINTER(c_void_p)]
    lib.kvr_create.restype = c_int
    lib.kvr_destroy.argtypes = [c_void_p]
    lib.kvr_destroy.restype = None
    lib.kvr_cache_bytes.argtypes = [POINTER(kvr_dims), c_int32]
    lib.kvr_cache_bytes.restype = c_size_t
    lib.kvr_workspace_bytes.argtypes = [c_void_p]
    lib.kvr_workspace_bytes.restype = c_size_t
    lib.kvr_prefill.argtypes = [c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_void_p, c_void_p]
    lib.kvr_prefill.restype = c_int
    lib.kvr_repair.argtypes = [c_void_p, POINTER(kvr_doc), c_int32, c_void_p]
    lib.kvr_repair.restype = c_int
    lib.kvr_select.argtypes = [c_int, c_int32, c_int32, c_int32, c_int32, c_uint64, POINTER(c_int32), POINTER(c_int32)]
    lib.kvr_select.restype = c_int
    lib.kvr_select_to_boundary.argtypes = [c_int32, c_int32, c_int32, c_int32, c_int32, POINTER(c_int32),
                                           POINTER(c_int32)]
    lib.kvr_select_to_boundary.restype = c_int
    lib.kvr_transplant.argtypes = [c_void_p, c_void_p, c_int32, c_void_p, c_int32, POINTER(c_int32), c_int32,
                                   c_void_p]
    lib.kvr_transplant.restype = c_int
    lib.kvr_score.argtypes = [c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_int32, c_void_p, c_void_p, c_void_p]
    lib.kvr_score.restype = c_int
    lib.kvr_generate.argtypes = [c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_int32, c_int32, c_void_p]
    lib.kvr_generate.restype = c_int
    lib.kvr_select_cacheblend.argtypes = [c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_int32, c_int32, c_int32,
                                          c_int32, c_void_p, c_void_p, POINTER(c_int32), c_void_p]
    lib.kvr_select_cacheblend.restype = c_int
    lib.kvr_select_attention.argtypes = [c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_int32, c_int32, c_int32,
                                         c_int32, c_void_p, c_void_p, POINTER(c_int32), c_void_p]
    lib.kvr_select_attention.restype = c_int
    lib.kvr_select_attention_noalloc.argtypes = lib.kvr_select_attention.argtypes
    lib.kvr_select_attention_noalloc.restype = c_int
    lib.kvr_answer_logprob.argtypes = [POINTER(c_float), c_int32, c_int32, c_int32, POINTER(c_double)]
    lib.kvr_answer_logprob.restype = c_int
    lib.kvr_margin_recovery.argtypes = [c_double, c_double, c_double, POINTER(c_double), POINTER(c_int32)]
    lib.kvr_margin_recovery.restype = c_int
    lib.kvr_flipped.argtypes = [POINTER(c_int32), c_int32, POINTER(c_int32), c_int32, POINTER(c_int32), c_int32,
                                POINTER(c_int32)]
    lib.kvr_flipped.restype = c_int
    lib.kvr_profile_enable.argtypes = [c_void_p, c_int32]
    lib.kvr_profile_enable.restype = c_int
    lib.kvr_profile_read.argtypes = [c_void_p, c_int32, POINTER(c_char_p), POINTER(c_double), POINTER(c_int64),
                                     POINTER(c_int32)]
    lib.kvr_profile_read.restype = c_int
    lib.kvr_last_error.argtypes = [c_void_p]
    lib.kvr_last_error.restype = c_char_p
    _lib = lib
    return lib


def _check(status: int, ctx: Optional[int] = None) -> None:
    if status != KVR_OK:
        raise KvrError(status, kvr_last_error(ctx))


def kvr_last_error(ctx: Optional[int] = None) -> str:
    msg = load().kvr_last_error(ctx)
    return msg.decode() if msg else ""


def kvr_create(dims: kvr_dims, weights: kvr_weights) -> int:
    out = c_void_p()
    _check(load().kvr_create(ctypes.byref(dims), ctypes.byref(weights), ctypes.byref(out)))
    return out.value


def kvr_destroy(ctx: Optional[int]) -> None:
    load().kvr_destroy(ctx)


def kvr_cache_bytes(dims: kvr_dims, n_cap: int) -> int:
    return load().kvr_cache_bytes(ctypes.byref(dims), n_cap)


def kvr_workspace_bytes(ctx: int) -> int:
    return load().kvr_workspace_bytes(ctx)


def kvr_prefill(ctx: int, d_tokens: int, n: int, n_cap: int, d_cache: int, d_hidden_out: Optional[int] = None,
                stream: Optional[int] = None) -> None:
    _check(load().kvr_prefill(ctx, d_tokens, n, n_cap, d_cache, d_hidden_out, stream), ctx)


def make_doc(d_cache: int, n: int, n_cap: int, d_tokens_new: int, edit_start: int, edit_end: int,
             positions: Sequence[int], d_hidden_out: Optional[int] = None) -> kvr_doc:
    """A kvr_doc; the position array is kept alive on the returned object."""
    arr = (c_int32 * max(1, len(positions)))(*positions)
    doc = kvr_doc(d_cache, n, n_cap, d_tokens_new, edit_start, edit_end,
                  ctypes.cast(arr, POINTER(c_int32)), len(positions), d_hidden_out)
    doc._positions = arr  # keep alive
    return doc


def kvr_repair(ctx: int, docs: Sequence[kvr_doc], stream: Optional[int] = None) -> None:
    arr = (kvr_doc * max(1, len(docs)))(*docs)
    _check(load().kvr_repair(ctx, arr, len(docs), stream), ctx)


def kvr_profile_enable(ctx: int, enable: bool = True) -> None:
    _check(load().kvr_profile_enable(ctx, 1 if enable else 0), ctx)


def kvr_profile_read(ctx: int) -> dict:
    """{step name: (total ms, launches)} accumulated since the previous read."""
    cap = 32
    names = (c_char_p * cap)()
    ms = (c_double * cap)()
    cnt = (c_int64 * cap)()
    n = c_int32(0)
    _check(load().kvr_profile_read(ctx, cap, names, ms, cnt, ctypes.byref(n)), ctx)
    return {names[i].decode(): (ms[i], cnt[i]) for i in range(min(n.value, cap))}


def kvr_select(policy: int, n: int, edit_start: int, edit_end: int, K: int, seed: int = 0) -> list:
    out = (c_int32 * max(1, K))()
    cnt = c_int32(0)
    _check(load().kvr_select(policy, n, edit_start, edit_end, K, seed & ((1 << 64) - 1), out, ctypes.byref(cnt)))
    return list(out[:cnt.value])


def kvr_select_to_boundary(n: int, edit_start: int, edit_end: int, boundary: int, capacity: Optional[int] = None) -> list:
    cap = max(0, n) if capacity is None else capacity
    out = (c_int32 * max(1, cap))()
    cnt = c_int32(0)
    _check(load().kvr_select_to_boundary(n, edit_start, edit_end, boundary, cap, out, ctypes.byref(cnt)))
    return list(out[:cnt.value])


def kvr_transplant(ctx: int, d_src: int, src_n_cap: int, d_dst: int, dst_n_cap: int, positions: Sequence[int],
                   stream: Optional[int] = None) -> None:
    arr = (c_int32 * max(1, len(positions)))(*positions)
    _check(load().kvr_transplant(ctx, d_src, src_n_cap, d_dst, dst_n_cap, arr, len(positions), stream), ctx)


def kvr_score(ctx: int, d_cache: int, n: int, n_cap: int, d_tokens: int, m: int, d_logprob: Optional[int],
              d_argmax: Optional[int] = None, stream: Optional[int] = None) -> None:
    _check(load().kvr_score(ctx, d_cache, n, n_cap, d_tokens, m, d_logprob, d_argmax, stream), ctx)


def kvr_generate(ctx: int, d_cache: int, n: int, n_cap: int, d_tokens: int, q: int, max_new: int,
                 stream: Optional[int] = None) -> None:
    _check(load().kvr_generate(ctx, d_cache, n, n_cap, d_tokens, q, max_new, stream), ctx)


def kvr_select_cacheblend(ctx: int, d_cache: int, n: int, n_cap: int, d_tokens_new: int, edit_start: int,
                          edit_end: int, K: int, layer: int, d_out: Optional[int], d_dev_out: Optional[int] = None,
                          stream: Optional[int] = None) -> int:
    """Enqueues the selection; returns the number of positions written to d_out."""
    cnt = c_int32(0)
    _check(load().kvr_select_cacheblend(ctx, d_cache, n, n_cap, d_tokens_new, edit_start, edit_end, K, layer, d_out,
                                        d_dev_out, ctypes.byref(cnt), stream), ctx)
    return cnt.value


def kvr_select_attention(ctx: int, d_cache: int, n: int, n_cap: int, d_tokens: int, q: int, edit_start: int,
                         edit_end: int, K: int, d_out: Optional[int], d_mass_out: Optional[int] = None,
                         stream: Optional[int] = None) -> int:
    """Enqueues the selection; returns the number of positions written to d_out."""
    cnt = c_int32(0)
    _check(load().kvr_select_attention(ctx, d_cache, n, n_cap, d_tokens, q, edit_start, edit_end, K, d_out,
                                       d_mass_out, ctypes.byref(cnt), stream), ctx)
    return cnt.value


def kvr_select_attention_noalloc(ctx: int, d_cache: int, n: int, n_cap: int, d_tokens: int, q: int,
                                 edit_start: int, edit_end: int, K: int, d_out: Optional[int],
                                 d_mass_out: Optional[int] = None, stream: Optional[int] = None) -> int:
    """kvr_select_attention with its scratch in the library's fixed device array
    (allocates nothing); returns the number of positions written to d_out."""
    cnt = c_int32(0)
    _check(load().kvr_select_attention_noalloc(ctx, d_cache, n, n_cap, d_tokens, q, edit_start, edit_end, K, d_out,
                                               d_mass_out, ctypes.byref(cnt), stream), ctx)
    return cnt.value


def kvr_answer_logprob(logprob: Sequence[float], query_len: int, answer_len: int) -> float:
    """Mean log p of the answer tokens of a block scored as query + answer
    (logprob: kvr_score's output copied to the host)."""
    arr = (c_float * max(1, len(logprob)))(*logprob)
    out = c_double(0.0)
    _check(load().kvr_answer_logprob(arr, len(logprob), query_len, answer_len, ctypes.byref(out)))
    return out.value


def kvr_margin_recovery(m_repaired: float, m_stale: float, m_oracle: float) -> Optional[float]:
    """Eq. 2 (unclipped); None when the stale-to-oracle gap is zero."""
    out = c_double(0.0)
    defined = c_int32(0)
    _check(load().kvr_margin_recovery(m_repaired, m_stale, m_oracle, ctypes.byref(out), ctypes.byref(defined)))
    return out.value if defined.value else None


def kvr_flipped(continuation: Sequence[int], a_new: Sequence[int], a_old: Sequence[int]) -> bool:
    """Eq. 3 for one item: a_new occurs in the greedy continuation and a_old does not."""
    arrs = [(c_int32 * max(1, len(x)))(*x) for x in (continuation, a_new, a_old)]
    out = c_int32(0)
    _check(load().kvr_flipped(arrs[0], len(continuation), arrs[1], len(a_new), arrs[2], len(a_old),
                              ctypes.byref(out)))
    return bool(out.value)
