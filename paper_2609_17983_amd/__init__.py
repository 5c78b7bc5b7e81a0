"""Budgeted in-place KV-cache repair on MI355X (gfx950).

The HIP library libkvr.so (include/kvr.h) holds every kernel; this package is
its ctypes binding (same call names) plus struct-marshalling helpers.
"""
from ._lib import (KVR_BF16, KVR_E_ARG, KVR_E_HIP, KVR_E_NOMEM, KVR_E_RANGE, KVR_E_UNSUPPORTED, KVR_EDIT_LOCAL,
                   KVR_F32, KVR_OK, KVR_RANDOM, EXPORTED, LIB_PATH, KvrError, kvr_cache_bytes, kvr_create, kvr_destroy,
                   kvr_dims, kvr_doc, kvr_last_error, kvr_layer_weights, kvr_prefill, kvr_profile_enable,
                   kvr_profile_read, kvr_repair, kvr_select, kvr_select_to_boundary, kvr_transplant,
                   kvr_score, kvr_generate, kvr_select_cacheblend, kvr_select_attention, kvr_select_attention_noalloc,
                   kvr_answer_logprob, kvr_margin_recovery, kvr_flipped,
                   kvr_weights, kvr_workspace_bytes, load, make_doc)
from .marshal import dims_for, weights_struct

__all__ = [
    "KVR_BF16", "KVR_E_ARG", "KVR_E_HIP", "KVR_E_NOMEM", "KVR_E_RANGE", "KVR_E_UNSUPPORTED", "KVR_EDIT_LOCAL",
    "KVR_F32", "KVR_OK", "KVR_RANDOM", "EXPORTED", "LIB_PATH", "KvrError", "kvr_cache_bytes", "kvr_create",
    "kvr_destroy", "kvr_dims", "kvr_doc", "kvr_last_error", "kvr_layer_weights", "kvr_prefill",
    "kvr_profile_enable", "kvr_profile_read", "kvr_repair", "kvr_select", "kvr_select_to_boundary",
    "kvr_transplant", "kvr_score", "kvr_generate", "kvr_select_cacheblend", "kvr_select_attention", "kvr_select_attention_noalloc",
    "kvr_answer_logprob",
    "kvr_margin_recovery", "kvr_flipped", "kvr_weights", "kvr_workspace_bytes", "load", "make_doc", "dims_for", "weights_struct",
]
