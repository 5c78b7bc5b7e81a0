"""Position selection for the repair budget (oracle side).

TEST INFRASTRUCTURE ONLY; shares no code with the library's host selector.

Paper, Section 3 ("The repair interface") and Table 1:
* the downstream pool is D = [s_end, n - 1) (it excludes the last position);
* a policy picks A, a subset of D with |A| = K (K counts only downstream
  positions; the edit span is always recomputed and is not counted);
* EditLocal: the K positions immediately after the span;
* Random: K positions uniform from the pool (the paper uses 5 seeds and does
  not name a generator).

Readings where the paper is silent:
* K > |D| selects all of D (the count returned is min(K, |D|)).
* Random draws with SplitMix64 (Steele, Lea and Flood, "Fast splittable
  pseudorandom number generators", OOPSLA 2014) seeded with ``seed``: the
  state advances by the golden-gamma constant and each output is the state
  passed through the variant-13 finaliser.  A partial Fisher-Yates shuffle
  over D in ascending order takes j = i + (next() mod (m - i)) for
  i = 0..K-1, swapping D[i] and D[j]; the first K entries, sorted ascending,
  are A.
"""
from __future__ import annotations

from typing import List

_MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15


class SplitMix64:
    """SplitMix64 as published: state += gamma; z = mix(state)."""

    def __init__(self, seed: int):
        self.state = seed & _MASK64

    def next(self) -> int:
        self.state = (self.state + GOLDEN_GAMMA) & _MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
        return z ^ (z >> 31)


def check_span(n: int, edit_start: int, edit_end: int, k: int) -> None:
    if n < 1 or not (0 <= edit_start <= edit_end <= n) or k < 0:
        raise ValueError(f"bad selection arguments n={n} span=[{edit_start},{edit_end}) K={k}")


def pool(n: int, edit_end: int) -> List[int]:
    """D = [s_end, n - 1)."""
    return list(range(edit_end, n - 1))


def select_edit_local(n: int, edit_start: int, edit_end: int, k: int) -> List[int]:
    check_span(n, edit_start, edit_end, k)
    d = pool(n, edit_end)
    return d[:min(k, len(d))]


def select_random(n: int, edit_start: int, edit_end: int, k: int, seed: int) -> List[int]:
    check_span(n, edit_start, edit_end, k)
    d = pool(n, edit_end)
    m = len(d)
    kk = min(k, m)
    rng = SplitMix64(seed)
    for i in range(kk):
        j = i + rng.next() % (m - i)
        d[i], d[j] = d[j], d[i]
    return sorted(d[:kk])


def select_to_boundary(n: int, edit_start: int, edit_end: int, boundary: int) -> List[int]:
    """EditLocal@boundary (Section 5.2, "How Far the Window Should Extend"):
    every pool position from the end of the edit up to the next document
    boundary, i.e. [s_end, min(boundary, n - 1)) -- the pool D ends at n - 1."""
    check_span(n, edit_start, edit_end, 0)
    if boundary < edit_end:
        raise ValueError("boundary before the end of the edit")
    return list(range(edit_end, min(boundary, n - 1)))
