"""Forward-based selection policies of Table 1 (oracle side).

TEST INFRASTRUCTURE ONLY; float64; shares no code with the library.

Attention (Table 1: the K pool positions that the query attends to most over
the stale cache; Section 3, "Cost accounting": it costs one scoring pass over
the stale cache).  Readings (the paper's
appendix with the aggregation rule is not available):
* the query tokens are appended after the n stale positions and run through
  the decoder as in the scoring forward (they attend over the stale cache and
  causally over each other; their keys/values occupy scratch slots);
* the score of a stale position p is the softmax attention probability that
  the query assigns to p, summed over every layer, query head and query
  token;
* top-K over the pool D by decreasing score, ties to the lower position,
  ascending.

CacheBlend (Table 1: the K pool positions whose keys/values of the second
layer moved most; Section 3, "Cost accounting": its extra cost is about one
prefill layer).  Readings:
* the second layer counts from one, i.e. layer index 1: its keys/values need the
  full first layer over the changed suffix plus one projection, which is the
  stated cost of about one prefill layer (index 2 would cost two);
* the fresh keys/values of the positions from the edit start to the end are
  computed from C' layer by layer over the stale cache (positions before the
  edit are unchanged by it, so their stale states are also their fresh ones),
  written into a scratch copy, never into the stale cache;
* deviation of position p: ||K_fresh[p] - K_stale[p]||_2 +
  ||V_fresh[p] - V_stale[p]||_2, each norm over all kv heads and dimensions
  of that layer;
* top-K over the pool D = [s_end, n - 1) by decreasing deviation, ties to the
  lower position, returned in ascending order.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

from . import decoder as od
from .select import check_span, pool


def fresh_kv(shape, weights, cache: np.ndarray, tokens_new: np.ndarray, edit_start: int,
             layer: int) -> Tuple[np.ndarray, np.ndarray]:
    """Keys and values of layer ``layer`` for positions [edit_start, n) of C',
    computed over a scratch copy of the stale cache: [H_kv, n - edit_start, hd] each."""
    tokens_new = np.asarray(tokens_new, dtype=np.int64)
    n = tokens_new.shape[0]
    P = np.arange(edit_start, n, dtype=np.int64)
    scratch = np.array(cache[:layer + 1], dtype=np.float64)
    h = weights.embed_rows(tokens_new[P])
    for l in range(layer):
        h = od.layer_forward(shape, weights.layer(l), h, P, scratch[l, 0], scratch[l, 1])
    w = weights.layer(layer)
    x = od.rms_norm(h, w["attn_norm"], shape.rms_eps)
    k = x @ w["wk"].T
    v = x @ w["wv"].T
    if w.get("bk") is not None:
        k = k + w["bk"]
        v = v + w["bv"]
    R, Hkv, hd = P.shape[0], shape.n_kv_heads, shape.head_dim
    k = od.rope(k.reshape(R, Hkv, hd), P, shape.rope_theta).transpose(1, 0, 2)
    v = v.reshape(R, Hkv, hd).transpose(1, 0, 2)
    return k, v


def cacheblend_deviation(shape, weights, cache: np.ndarray, tokens_new: np.ndarray, edit_start: int,
                         edit_end: int, layer: int = 1) -> np.ndarray:
    """Deviation of every pool position [edit_end, n - 1) at ``layer``."""
    n = len(tokens_new)
    k, v = fresh_kv(shape, weights, cache, tokens_new, edit_start, layer)
    D = np.asarray(pool(n, edit_end), dtype=np.int64)
    j = D - edit_start
    dk = k[:, j, :] - np.asarray(cache[layer, 0][:, D, :], dtype=np.float64)
    dv = v[:, j, :] - np.asarray(cache[layer, 1][:, D, :], dtype=np.float64)
    return np.sqrt((dk ** 2).sum(axis=(0, 2))) + np.sqrt((dv ** 2).sum(axis=(0, 2)))


def top_k_positions(dev: np.ndarray, first: int, k: int) -> List[int]:
    """Positions first + i of the k largest dev[i], ties to the lower position, ascending."""
    order = sorted(range(len(dev)), key=lambda i: (-float(dev[i]), i))
    return sorted(first + i for i in order[:min(k, len(dev))])


def select_cacheblend(shape, weights, cache: np.ndarray, tokens_new: np.ndarray, edit_start: int,
                      edit_end: int, k: int, layer: int = 1) -> List[int]:
    check_span(len(tokens_new), edit_start, edit_end, k)
    dev = cacheblend_deviation(shape, weights, cache, tokens_new, edit_start, edit_end, layer)
    return top_k_positions(dev, edit_end, k)


def attention_mass(shape, weights, cache: np.ndarray, tokens: np.ndarray, n: int, q: int) -> np.ndarray:
    """Summed attention probability on each stale position [0, n) from the q
    query tokens tokens[n:n+q] over all layers and query heads."""
    tokens = np.asarray(tokens, dtype=np.int64)
    P = np.arange(n, n + q, dtype=np.int64)
    scratch = np.array(cache, dtype=np.float64)
    Hq, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    G = Hq // Hkv
    mass = np.zeros(n, dtype=np.float64)
    h = weights.embed_rows(tokens[P])
    for l in range(shape.n_layers):
        w = weights.layer(l)
        x = od.rms_norm(h, w["attn_norm"], shape.rms_eps)
        qx, kx, vx = x @ w["wq"].T, x @ w["wk"].T, x @ w["wv"].T
        if w.get("bq") is not None:
            qx, kx, vx = qx + w["bq"], kx + w["bk"], vx + w["bv"]
        qr = od.rope(qx.reshape(q, Hq, hd), P, shape.rope_theta)
        kr = od.rope(kx.reshape(q, Hkv, hd), P, shape.rope_theta)
        scratch[l, 0][:, P, :] = kr.transpose(1, 0, 2)
        scratch[l, 1][:, P, :] = vx.reshape(q, Hkv, hd).transpose(1, 0, 2)
        for r in range(q):
            keys = scratch[l, 0][:, :P[r] + 1, :]
            for j in range(Hq):
                sc = keys[j // G] @ qr[r, j] / np.sqrt(hd)
                pr = np.exp(sc - sc.max())
                pr /= pr.sum()
                mass += pr[:n]
        h = od.layer_forward(shape, w, h, P, scratch[l, 0], scratch[l, 1])
    return mass


def select_attention(shape, weights, cache: np.ndarray, tokens: np.ndarray, n: int, q: int, edit_start: int,
                     edit_end: int, k: int) -> List[int]:
    check_span(n, edit_start, edit_end, k)
    mass = attention_mass(shape, weights, cache, tokens, n, q)
    D = pool(n, edit_end)
    return top_k_positions(mass[D[0]:D[-1] + 1] if D else np.zeros(0), edit_end, k)
