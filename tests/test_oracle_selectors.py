"""Pins for the oracle's CacheBlend selector (no GPU).

Table 1 ("top-K by layer-2 key/value deviation") and Section 3: the fresh
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
