"""Marshalling helpers: build the C structs of include/kvr.h from a model
shape and device tensors (torch is used only for memory).  No compute."""
from __future__ import annotations

import ctypes
from typing import Dict, List

from . import _lib

_LAYER_FIELDS = ("attn_norm", "wq", "wk", "wv", "bq", "bk", "bv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


def dims_for(shape, dtype: int, max_ctx: int, max_rows: int) -> _lib.kvr_dims:
    """kvr_dims from any object with the decoder fields (n_layers, d_model, ...)."""
    return _lib.kvr_dims(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                         shape.d_ffn, shape.vocab, int(bool(shape.qkv_bias)), float(shape.rms_eps),
                         float(shape.rope_theta), int(max_ctx), int(max_rows), int(dtype))


def weights_struct(weights: Dict[str, object]) -> _lib.kvr_weights:
    """kvr_weights from {'embed', 'final_norm', 'layers': [dict of tensors],
    optionally 'lm_head'} on the device.

    The returned struct keeps its layer array alive; the tensors must outlive
    the context created from it.
    """
    layers: List[Dict[str, object]] = weights["layers"]
    arr = (_lib.kvr_layer_weights * len(layers))()
    for i, lw in enumerate(layers):
        for f in _LAYER_FIELDS:
            t = lw.get(f)
            setattr(arr[i], f, None if t is None else t.data_ptr())
    lm = weights.get("lm_head")
    ws = _lib.kvr_weights(weights["embed"].data_ptr(), weights["final_norm"].data_ptr(),
                          ctypes.cast(arr, ctypes.POINTER(_lib.kvr_layer_weights)),
                          None if lm is None else lm.data_ptr())
    ws._layers = arr
    return ws
