"""Fresh-query forward, teacher-forced scoring and the repair metrics (oracle).

TEST INFRASTRUCTURE ONLY; float64; shares no code with the library.

Paper Section 3, "What counts as repaired":
* the query (and a candidate answer) are appended after the cached context and
  read the cache; for a cache state x, m_x is the difference between the
  length-averaged teacher-forced log-probabilities of the post-edit answer
  a_new and the pre-edit answer a_old;
* margin recovery (Eq. 2) MR = (m_repaired - m_stale) / (m_oracle - m_stale),
  unclipped, undefined (None) for a zero gap;
* flip (Eq. 3) for one item: a_new occurs in the greedy continuation y of at
  most 16 tokens and a_old does not; the flip rate is its mean over items.

Readings: the appended tokens are processed exactly like repaired rows (they
attend over the cache and causally over each other, and their keys/values
occupy the cache slots after the context); "a in y" is contiguous
token-subsequence containment; the greedy argmax takes the lowest token id
among equal maxima.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import decoder as od


def log_softmax(z: np.ndarray) -> np.ndarray:
    """Row-wise log-softmax, max-shifted."""
    z = np.asarray(z, dtype=np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    return z - m - np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True))


def score(shape, weights, lm_head: np.ndarray, cache: np.ndarray, tokens: np.ndarray, n: int,
          m: int) -> Tuple[np.ndarray, np.ndarray]:
    """Append tokens[n:n+m] after the n cached positions (cache updated in
    slots [n, n+m)).  Returns (lp [m-1], argmax [m]): lp[j] = log p(tokens[n+j+1]
    | tokens[:n+j+1]) and argmax[j] the most probable token after position n+j."""
    tokens = np.asarray(tokens, dtype=np.int64)
    y = od.repair(shape, weights, cache, tokens, n, n + m, [])
    logits = y @ np.asarray(lm_head, dtype=np.float64).T
    lsm = log_softmax(logits)
    lp = np.array([lsm[j, tokens[n + j + 1]] for j in range(m - 1)], dtype=np.float64)
    return lp, np.argmax(logits, axis=-1)


def generate(shape, weights, lm_head: np.ndarray, cache: np.ndarray, tokens: Sequence[int], n: int, q: int,
             max_new: int) -> List[int]:
    """Greedy continuation of tokens[:n+q] (first n already in the cache):
    max_new tokens, each the argmax after the previous one."""
    toks = [int(t) for t in tokens[:n + q]]
    _, am = score(shape, weights, lm_head, cache, np.array(toks), n, q)
    out = [int(am[-1])]
    for i in range(1, max_new):
        toks.append(out[-1])
        _, am = score(shape, weights, lm_head, cache, np.array(toks), n + q + i - 1, 1)
        out.append(int(am[-1]))
    return out


def mean_answer_logprob(lp: np.ndarray, q: int, k: int) -> float:
    """Length-averaged teacher-forced log-probability of the k answer tokens
    that follow a q-token query in a scored block of q + k tokens."""
    return float(np.mean(np.asarray(lp)[q - 1:q - 1 + k]))


def margin(mean_lp_new: float, mean_lp_old: float) -> float:
    """m_x: post-edit answer minus pre-edit answer."""
    return float(mean_lp_new - mean_lp_old)


def margin_recovery(m_repaired: float, m_stale: float, m_oracle: float) -> Optional[float]:
    """Eq. 2, unclipped; None for a zero stale-to-oracle gap (excluded items)."""
    gap = m_oracle - m_stale
    if gap == 0.0:
        return None
    return (m_repaired - m_stale) / gap


def contains(seq: Sequence[int], sub: Sequence[int]) -> bool:
    sub = list(sub)
    if not sub:
        return True
    seq = list(seq)
    return any(seq[i:i + len(sub)] == sub for i in range(len(seq) - len(sub) + 1))


def flip(y: Sequence[int], a_new: Sequence[int], a_old: Sequence[int]) -> bool:
    """One item of Eq. 3."""
    return contains(y, a_new) and not contains(y, a_old)


def flip_rate(items: Sequence[Tuple[Sequence[int], Sequence[int], Sequence[int]]]) -> float:
    """Eq. 3 over retained items (y, a_new, a_old)."""
    return float(np.mean([flip(y, a, b) for y, a, b in items])) if items else 0.0
