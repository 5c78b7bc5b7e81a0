"""Pins for the oracle's CacheBlend selector (no GPU).

Table 1 (the K pool positions whose second-layer keys/values moved most) and
Section 3: the fresh
keys/values of one early layer are compared with the stale cache's.  Pinned
by: the fresh states equal the full prefill of C' at that layer (the edit
cannot change earlier positions), the deviation equals its definition taken
from two full prefills, a null edit deviates nowhere, and the top-K rule
matches an exhaustive search on small inputs.
"""
import itertools

import numpy as np
import pytest
import torch

import synth
from oracle import decoder as od
from oracle import selectors as osl
from oracle import select as osel
from tests.test_oracle import MICRO_BIAS, SMALL, dense, relmax


def _case(shape, n=24, s0=7, span=3, seed=31):
    W, _ = dense(shape, seed=seed, std=0.2)
    toks = synth.make_tokens(n, shape.vocab, seed=seed).numpy()
    new = synth.apply_edit(torch.from_numpy(toks), s0, span, shape.vocab, seed=seed).numpy()
    return W, toks, new


@pytest.mark.parametrize("shape,layer", [(SMALL, 1), (MICRO_BIAS, 0), (MICRO_BIAS, 1)])
def test_fresh_kv_equals_prefill_of_edited_context(shape, layer):
    W, toks, new = _case(shape)
    stale, _ = od.prefill(shape, W, toks)
    k, v = osl.fresh_kv(shape, W, stale, new, 7, layer)
    ref, _ = od.prefill(shape, W, new)
    assert relmax(k, ref[layer, 0][:, 7:]) < 1e-12
    assert relmax(v, ref[layer, 1][:, 7:]) < 1e-12


def test_deviation_is_the_distance_between_the_two_prefills():
    shape = SMALL
    W, toks, new = _case(shape)
    stale, _ = od.prefill(shape, W, toks)
    ref, _ = od.prefill(shape, W, new)
    dev = osl.cacheblend_deviation(shape, W, stale, new, 7, 10, layer=1)
    D = np.arange(10, 23)
    want = (np.sqrt(((ref[1, 0][:, D] - stale[1, 0][:, D]) ** 2).sum(axis=(0, 2)))
            + np.sqrt(((ref[1, 1][:, D] - stale[1, 1][:, D]) ** 2).sum(axis=(0, 2))))
    assert relmax(dev, want) < 1e-12
    assert np.all(dev > 0)


def test_null_edit_deviates_nowhere():
    shape = SMALL
    W, toks, _ = _case(shape)
    stale, _ = od.prefill(shape, W, toks)
    dev = osl.cacheblend_deviation(shape, W, stale, toks, 7, 10, layer=1)
    assert np.max(np.abs(dev)) < 1e-12 * max(1.0, float(np.max(np.abs(stale))))
    # exact ties (all zero) break to the lowest positions, i.e. EditLocal's window
    assert osl.top_k_positions(np.zeros(13), 10, 5) == osel.select_edit_local(24, 7, 10, 5)


def test_top_k_rule_against_exhaustive_search():
    rng = np.random.default_rng(5)
    for _ in range(200):
        m = int(rng.integers(1, 8))
        dev = rng.integers(0, 4, size=m).astype(np.float64)  # many ties
        k = int(rng.integers(0, m + 1))
        best = max(itertools.combinations(range(m), k),
                   key=lambda c: (sum(dev[list(c)]), [-i for i in sorted(c)]))
        assert osl.top_k_positions(dev, 100, k) == sorted(100 + i for i in best)


def test_attention_mass_matches_causal_lm_attentions():
    """The summed attention on each stale position equals the sum of a float64
    transformers causal LM's attention probabilities (output_attentions) over
    layers, heads and query rows, when the stale cache is K(C)."""
    from tests.test_oracle_scoring import _causal_lm
    shape = SMALL
    n, q = 22, 5
    W, _ = dense(shape, seed=41, std=0.2)
    lm = synth.make_lm_head(shape, dtype=torch.float32, seed=41).to(torch.float64).numpy()
    toks = synth.make_tokens(n + q, shape.vocab, seed=42).numpy().astype(np.int64)
    cache, _ = od.prefill(shape, W, toks[:n], n_cap=n + q)
    mass = osl.attention_mass(shape, W, cache, toks, n, q)
    model = _causal_lm(shape, W, lm)
    with torch.no_grad():
        att = model(input_ids=torch.from_numpy(toks)[None], output_attentions=True).attentions
    ref = sum(a[0, :, n:n + q, :n].sum(dim=(0, 1)).numpy() for a in att)
    assert relmax(mass, ref) < 1e-5
    # each (layer, head, query row) distributes mass 1 over [0, its position]
    assert np.sum(mass) <= shape.n_layers * shape.n_heads * q + 1e-9


def test_select_attention_takes_top_mass():
    shape = MICRO_BIAS
    n, q = 18, 3
    W, _ = dense(shape, seed=43, std=0.3)
    toks = synth.make_tokens(n + q, shape.vocab, seed=44).numpy().astype(np.int64)
    cache, _ = od.prefill(shape, W, toks[:n], n_cap=n + q)
    mass = osl.attention_mass(shape, W, cache.copy(), toks, n, q)
    sel = osl.select_attention(shape, W, cache.copy(), toks, n, q, 4, 6, 5)
    assert len(sel) == 5 and all(6 <= p < n - 1 for p in sel)
    rest = [p for p in range(6, n - 1) if p not in sel]
    assert min(mass[sel]) >= max(mass[rest])
