"""fp64 CPU oracle for the decoder, full prefill and in-place cache repair.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this module:
only the tests, the package's smoke check and the benchmark's CPU-baseline
leg call it.  It shares no code with the HIP library.

What it computes (paper, Section 3 "Cache Repair as Budgeted Recomputation"):

* The model is a Llama-style pre-norm decoder (RMSNorm, Q/K/V projections
  with optional bias, rotary embedding at each token's absolute position,
  causal grouped-query attention with 1/sqrt(head_dim) scale, output
  projection, SwiGLU MLP, residual connections, final RMSNorm).  The paper
  runs Llama/Qwen/Mistral checkpoints of exactly this family (Section 4,
  "Models and decoding").
* ``prefill`` is the full forward over all n positions of a context, writing
  the key/value states of every position: the cache K(C), and for the edited
  context K(C') the paper's repair target (Section 3, "Question Setting").
* ``repair`` is the operator R(K(C), C', P) of Section 3 ("The repair
  interface"): the positions of P are recomputed from C' layer by layer over
  the stale cache, every other cache entry is left unchanged.  Within a layer
  the fresh keys/values of all of P are written first, then every p in P
  attends over cache slots t <= p, fresh where t is in P and stale elsewhere.
  This order is the reading under which the endpoint identity (Eq. 1) holds.

Everything is float64; weights and caches given in bf16 are exactly
representable in float64, so they are passed in upcast.  Rotary angles are
computed in float64.

Inputs
* ``shape``: any object with the fields n_layers, d_model, n_heads,
  n_kv_heads, head_dim, d_ffn, rms_eps, rope_theta.
* ``weights``: an object with ``embed_rows(token_ids) -> [R, d]``,
  ``layer(l) -> dict`` (keys attn_norm, wq, wk, wv, bq, bk, bv, wo, mlp_norm,
  w_gate, w_up, w_down; biases may be None; matrices are [out][in]) and
  ``final_norm -> [d]``, all float64 numpy arrays.  ``DenseWeights`` wraps a
  dict of arrays.
* ``cache``: float64 array [L][2][H_kv][n_cap][head_dim] (index 0 = keys,
  1 = values), modified in place.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np


class DenseWeights:
    """Weights held fully in memory as float64 numpy arrays."""

    def __init__(self, embed: np.ndarray, layers: Sequence[Dict[str, Optional[np.ndarray]]],
                 final_norm: np.ndarray):
        self.embed = np.asarray(embed, dtype=np.float64)
        self.layers = [{k: (None if v is None else np.asarray(v, dtype=np.float64))
                        for k, v in lw.items()} for lw in layers]
        self.final_norm = np.asarray(final_norm, dtype=np.float64)

    def embed_rows(self, token_ids: np.ndarray) -> np.ndarray:
        return self.embed[np.asarray(token_ids, dtype=np.int64)]

    def layer(self, l: int) -> Dict[str, Optional[np.ndarray]]:
        return self.layers[l]


def rms_norm(h: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps) * gain


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing (i, i + head_dim/2).

    x: [R, H, head_dim]; row r is rotated by angles positions[r] * theta^(-2i/head_dim).
    The positions are the tokens' absolute document positions, which an in-place,
    length-preserving edit leaves unchanged (Section 3, "Question Setting").
    """
    hd = x.shape[-1]
    half = hd // 2
    i = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def attend(q: np.ndarray, positions: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray) -> np.ndarray:
    """Causal grouped-query attention of R query rows over one layer's cache.

    q: [R, H_q, hd]; k_cache, v_cache: [H_kv, n_cap, hd].  Query head j reads
    kv head j // (H_q / H_kv).  Row r attends over slots 0..positions[r].
    """
    R, Hq, hd = q.shape
    Hkv = k_cache.shape[0]
    G = Hq // Hkv
    scale = 1.0 / np.sqrt(hd)
    out = np.empty_like(q)
    for r in range(R):
        p = int(positions[r])
        for g in range(Hkv):
            keys = k_cache[g, :p + 1]
            vals = v_cache[g, :p + 1]
            s = (q[r, g * G:(g + 1) * G] @ keys.T) * scale
            s = s - s.max(axis=1, keepdims=True)
            w = np.exp(s)
            w = w / w.sum(axis=1, keepdims=True)
            out[r, g * G:(g + 1) * G] = w @ vals
    return out


def layer_forward(shape, w: Dict[str, Optional[np.ndarray]], h: np.ndarray, positions: np.ndarray,
                  k_cache: np.ndarray, v_cache: np.ndarray) -> np.ndarray:
    """One decoder layer for the rows ``positions`` with residual input h [R, d].

    Writes the rows' fresh keys/values into k_cache/v_cache at ``positions``
    first, then attends (each row over slots <= its own position).
    Returns the layer's residual output [R, d].
    """
    R = h.shape[0]
    Hq, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    x = rms_norm(h, w["attn_norm"], shape.rms_eps)
    q = x @ w["wq"].T
    k = x @ w["wk"].T
    v = x @ w["wv"].T
    if w.get("bq") is not None:
        q = q + w["bq"]
        k = k + w["bk"]
        v = v + w["bv"]
    q = rope(q.reshape(R, Hq, hd), positions, shape.rope_theta)
    k = rope(k.reshape(R, Hkv, hd), positions, shape.rope_theta)
    v = v.reshape(R, Hkv, hd)
    pos = np.asarray(positions, dtype=np.int64)
    k_cache[:, pos, :] = k.transpose(1, 0, 2)
    v_cache[:, pos, :] = v.transpose(1, 0, 2)
    o = attend(q, pos, k_cache, v_cache).reshape(R, Hq * hd)
    h = h + o @ w["wo"].T
    x = rms_norm(h, w["mlp_norm"], shape.rms_eps)
    a = silu(x @ w["w_gate"].T) * (x @ w["w_up"].T)
    return h + a @ w["w_down"].T


def empty_cache(shape, n_cap: int) -> np.ndarray:
    return np.zeros((shape.n_layers, 2, shape.n_kv_heads, n_cap, shape.head_dim), dtype=np.float64)


def prefill(shape, weights, tokens: np.ndarray, n_cap: Optional[int] = None):
    """Full causal forward over all positions of ``tokens``.

    Returns (cache [L][2][H_kv][n_cap][hd], y [n, d]) where y is the
    final-RMSNorm output of every position.
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    n = tokens.shape[0]
    cache = empty_cache(shape, n if n_cap is None else n_cap)
    pos = np.arange(n)
    h = weights.embed_rows(tokens)
    for l in range(shape.n_layers):
        h = layer_forward(shape, weights.layer(l), h, pos, cache[l, 0], cache[l, 1])
    return cache, rms_norm(h, weights.final_norm, shape.rms_eps)


def repaired_set(edit_start: int, edit_end: int, positions: Sequence[int]) -> np.ndarray:
    """P = S u A, ascending (S = [edit_start, edit_end))."""
    return np.array(sorted(set(range(edit_start, edit_end)) | {int(p) for p in positions}),
                    dtype=np.int64)


def repair(shape, weights, cache: np.ndarray, tokens_new: np.ndarray, edit_start: int,
           edit_end: int, positions: Sequence[int], n_layers: Optional[int] = None) -> np.ndarray:
    """R(K(C), C', P): recompute P = S u A from C' layer by layer, in place.

    ``cache`` holds the stale K(C) and is updated in place: at every layer the
    slots of P receive their recomputed keys/values, all other slots are never
    written.  Returns the final-RMSNorm output of the rows of P [|P|, d], in
    ascending position order.  ``n_layers`` < L stops after that many layers and
    returns the residual stream instead (used only to time a bounded sample).
    """
    P = repaired_set(edit_start, edit_end, positions)
    if P.size == 0:
        return np.zeros((0, shape.d_model), dtype=np.float64)
    tokens_new = np.asarray(tokens_new, dtype=np.int64)
    h = weights.embed_rows(tokens_new[P])
    L = shape.n_layers if n_layers is None else n_layers
    for l in range(L):
        h = layer_forward(shape, weights.layer(l), h, P, cache[l, 0], cache[l, 1])
    if L < shape.n_layers:
        return h
    return rms_norm(h, weights.final_norm, shape.rms_eps)


def transplant(cache: np.ndarray, oracle_cache: np.ndarray, positions: Sequence[int]) -> None:
    """Copy the K/V states of ``positions`` from the oracle cache K(C') (Section 3,
    "Transplant is not recomputation").  A diagnostic, not a repair method."""
    pos = np.asarray(positions, dtype=np.int64)
    cache[:, :, :, pos, :] = oracle_cache[:, :, :, pos, :]
