"""Oracle: importance score, high-precision budget and top-k selection.

Test infrastructure only.

Importance (H2O policy, cited in Sections 3.1 and 4.1; Fig. 3 right): the
paper adopts heavy-hitter accumulated attention without restating it.
Reading: each decode step adds the step's post-softmax probability of every
token to that token's score; no decay; a new token starts at 0; under
grouped-query attention the probabilities of the query heads sharing a KV
head are summed, left to right in query-head order, in fp32, and that sum is
added to the score with one fp32 add.

Selection (Fig. 3 right; Sections 2.1 and 3.1): tokens local to the current
position (the recent window) and the top tokens by importance form the
importance (high-precision) cache, every other token the retained
(low-precision) cache.  Readings:
  * the window is the last W positions and is always high precision;
  * eligible tokens are those currently high precision and outside the window
    (at the first selection after prefill: every token outside the window);
  * the k_heavy eligible tokens with the largest key (score, position) are
    kept -- a tie in score goes to the newer token -- and the other eligible
    tokens are demoted;
  * demotion is one way: a retained token is never promoted again (its
    high-precision data no longer exists).
"""
from __future__ import annotations

import numpy as np


def heavy_budget(length: int, ratio_num: int, ratio_den: int, window: int, window_in_ratio: bool) -> int:
    """Number of non-window tokens kept at high precision for a cache of
    ``length`` tokens: floor(ratio * length), minus the window when the window
    counts towards the ratio, and never below zero."""
    k = (ratio_num * length) // ratio_den
    if window_in_ratio:
        k -= window
    return max(0, k)


def accumulate(acc, probs) -> np.ndarray:
    """acc fp32 [L]; probs fp32 [G, L] -> acc + ((p_0 + p_1) + ...) in fp32."""
    probs = np.asarray(probs, dtype=np.float32)
    s = probs[0].copy()
    for i in range(1, probs.shape[0]):
        s = s + probs[i]
    return np.asarray(acc, dtype=np.float32) + s


def select(acc, is_hi, length: int, k_heavy: int, window: int, initial: bool) -> np.ndarray:
    """Return the new high-precision mask [length] (bool).

    acc fp32 [length]; is_hi bool [length] (ignored when ``initial``).
    """
    acc = np.asarray(acc, dtype=np.float32)[:length]
    pos = np.arange(length)
    in_window = pos >= length - window
    if initial:
        eligible = ~in_window
    else:
        eligible = np.asarray(is_hi, dtype=bool)[:length] & ~in_window
    idx = pos[eligible]
    # Sort by score descending, then position descending.
    order = np.lexsort((-idx, -acc[idx]))
    keep = idx[order[:k_heavy]]
    new_hi = in_window.copy()
    new_hi[keep] = True
    return new_hi


def heavy_list(acc, is_hi, length: int, window: int) -> np.ndarray:
    """The heavy hitters after a selection, most important first: the
    high-precision positions outside the window, ordered by score
    descending, an exact score tie to the newer position (the selection's
    own order).  Returns int64 positions."""
    acc = np.asarray(acc, dtype=np.float32)[:length]
    pos = np.arange(length)
    idx = pos[np.asarray(is_hi, dtype=bool)[:length] & (pos < length - window)]
    return idx[np.lexsort((-idx, -acc[idx]))]


def prefill_importance(q16, k16, scale: float) -> np.ndarray:
    """H2O importance of the prompt tokens at the end of prefill.

    q16 fp16 [G, T, D] (the query heads sharing one KV head); k16 fp16 [T, D].
    Every prompt query i attends causally to keys 0..i; token j's score is
    the sum, over the G query heads and every query i >= j, of its softmax
    probability.  Computed in fp64 from the fp16 inputs; returned as fp32 [T].
    """
    q = np.asarray(q16, dtype=np.float16).astype(np.float64)
    k = np.asarray(k16, dtype=np.float16).astype(np.float64)
    G, T, _ = q.shape
    causal = np.tril(np.ones((T, T), dtype=bool))          # [query i, key j]: j <= i
    total = np.zeros(T, dtype=np.float64)
    for g in range(G):
        s = (q[g] @ k.T) * float(scale)
        s = np.where(causal, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        e = np.where(causal, np.exp(s), 0.0)
        p = e / e.sum(axis=1, keepdims=True)
        total += p.sum(axis=0)
    return total.astype(np.float32)
