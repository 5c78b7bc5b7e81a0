"""Repair metrics of the paper from kvr_score / kvr_generate outputs (host
arithmetic on a handful of scalars; every forward runs in the library).

Section 3, "What counts as repaired": for a cache state x, m_x is the
difference between the length-averaged teacher-forced log-probabilities of the
post-edit answer a_new and the pre-edit answer a_old.  Eq. 2 (margin
recovery) compares the repaired margin with the stale and oracle ones; Eq. 3
(flip) asks whether the greedy continuation contains a_new and not a_old.
"""
from __future__ import annotations

from typing import Optional, Sequence


def answer_logprob(logprob: Sequence[float], query_len: int, answer_len: int) -> float:
    """Mean log p of the answer tokens of a block scored as query + answer:
    entry j of kvr_score's output predicts appended token j+1, so the answer's
    tokens are predicted by entries query_len-1 .. query_len+answer_len-2."""
    vals = [float(v) for v in logprob[query_len - 1:query_len - 1 + answer_len]]
    if len(vals) != answer_len or answer_len < 1:
        raise ValueError("the scored block does not hold the whole answer")
    return sum(vals) / answer_len


def margin(lp_new: float, lp_old: float) -> float:
    """m_x = mean log p(a_new) - mean log p(a_old)."""
    return lp_new - lp_old


def margin_recovery(m_repaired: float, m_stale: float, m_oracle: float) -> Optional[float]:
    """Eq. 2, unclipped; None when the stale-to-oracle gap is zero (such items
    are excluded)."""
    gap = m_oracle - m_stale
    return None if gap == 0 else (m_repaired - m_stale) / gap


def _occurs(seq: Sequence[int], sub: Sequence[int]) -> bool:
    n, k = len(seq), len(sub)
    return k == 0 or any(list(seq[i:i + k]) == list(sub) for i in range(n - k + 1))


def flipped(continuation: Sequence[int], a_new: Sequence[int], a_old: Sequence[int]) -> bool:
    """One item of Eq. 3: a_new appears in the greedy continuation (as a
    contiguous token run) and a_old does not."""
    return _occurs(continuation, a_new) and not _occurs(continuation, a_old)


def flip_rate(items) -> float:
    """Eq. 3: mean of flipped(y, a_new, a_old) over the retained items."""
    items = list(items)
    return sum(flipped(*it) for it in items) / len(items) if items else 0.0
