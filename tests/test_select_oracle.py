"""Pins for the oracle's position selection (no GPU).

Paper Table 1 and Section 3 ("The repair interface"): policies pick K
positions from D = [s_end, n - 1); EditLocal takes the K positions right after
the span, Random draws uniformly.  The generator is this build's reading
(SplitMix64), pinned to its published test vectors.
"""
import json
import os

import pytest

from oracle import select as osel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_splitmix64_published_vectors():
    g = _golden("splitmix64.json")
    for vec in g["vectors"]:
        rng = osel.SplitMix64(vec["seed"])
        if "outputs_hex" in vec:
            assert [f"{rng.next():016x}" for _ in vec["outputs_hex"]] == vec["outputs_hex"]
        else:
            assert [rng.next() for _ in vec["outputs"]] == vec["outputs"]


def test_edit_local_worked_window():
    g = _golden("editlocal_tiny.json")
    sel = osel.select_edit_local(g["n"], g["edit_start"], g["edit_end"], g["K"])
    assert sel == list(range(g["positions_first"], g["positions_last"] + 1))


def test_edit_local_pool_end_and_clipping():
    # the pool excludes position n-1
    assert osel.select_edit_local(10, 2, 4, 100) == [4, 5, 6, 7, 8]
    assert osel.select_edit_local(10, 2, 9, 5) == []
    assert osel.select_edit_local(10, 2, 10, 5) == []
    assert osel.select_edit_local(10, 3, 3, 0) == []
    with pytest.raises(ValueError):
        osel.select_edit_local(10, 5, 4, 1)
    with pytest.raises(ValueError):
        osel.select_edit_local(10, 2, 11, 1)


@pytest.mark.parametrize("seed", range(5))
def test_random_properties(seed):
    n, s0, s1, K = 5000, 1200, 1216, 32
    a = osel.select_random(n, s0, s1, K, seed)
    assert len(a) == K and len(set(a)) == K and a == sorted(a)
    assert all(s1 <= p < n - 1 for p in a)
    assert a == osel.select_random(n, s0, s1, K, seed)  # replay determinism
    if seed:
        assert a != osel.select_random(n, s0, s1, K, seed - 1)


def test_random_is_uniform_over_pool():
    # every pool position is drawn with probability K/|D|
    n, s0, s1, K = 40, 5, 10, 6
    counts = {p: 0 for p in range(s1, n - 1)}
    T = 6000
    for seed in range(T):
        for p in osel.select_random(n, s0, s1, K, seed):
            counts[p] += 1
    expect = T * K / len(counts)
    assert all(abs(c - expect) < 5 * (expect ** 0.5) for c in counts.values())


def test_random_full_pool_and_empty():
    assert osel.select_random(20, 3, 5, 1000, 1) == list(range(5, 19))
    assert osel.select_random(20, 3, 19, 4, 1) == []
    assert osel.select_random(1, 0, 0, 4, 1) == []


def test_random_first_draw_by_hand():
    # D = [2, 3, 4, 5, 6] (n = 8, span [1, 2)); K = 1 picks D[next() mod 5]
    first = osel.SplitMix64(7).next()
    assert osel.select_random(8, 1, 2, 1, 7) == [2 + first % 5]


def test_to_boundary_is_edit_local_up_to_the_boundary():
    """EditLocal@boundary (Section 5.2) recomputes from the edit end to the next
    document boundary: it equals EditLocal with K = boundary - s_end while the
    boundary lies inside the pool, and the pool end n-1 clips it otherwise."""
    for n, s0, s1 in ((5000, 1500, 1516), (64, 10, 14), (20, 0, 0)):
        for k in range(0, 40):
            b = s1 + k
            assert osel.select_to_boundary(n, s0, s1, b) == osel.select_edit_local(n, s0, s1, k)
    assert osel.select_to_boundary(64, 10, 14, 14) == []
    assert osel.select_to_boundary(64, 10, 14, 10 ** 6) == list(range(14, 63))
    with pytest.raises(ValueError):
        osel.select_to_boundary(64, 10, 14, 13)
