"""Exhaustive selection for tiny caches (TEST INFRASTRUCTURE ONLY).

Checks the oracle's greedy eviction against the objective it claims to
solve.  Eq. 1 keeps at most B tokens, forces the pinned set in and maximises
the kept sum of retention scores; at page granularity (Sec. III-D) the kept
sum is the sum of |p| * S_p over kept pages, and the paper states that the
greedy ascending-S_p rule is optimal there because pages have equal size.

``best_eviction`` enumerates every subset of non-pinned pages, keeps the
feasible ones, and returns the subset with the largest kept sum, breaking
ties by fewer evicted pages, then by fewer evicted tokens.  Pure Python,
exponential: for at most ~16 candidate pages.
"""
from __future__ import annotations

from itertools import combinations
from typing import Optional, Sequence, Tuple


def best_eviction(page_score: Sequence[float], sizes: Sequence[int],
                  pinned: Sequence[bool], budget: int) -> Optional[Tuple[int, ...]]:
    """Indices of the pages to evict, or None when no subset meets the budget."""
    m = len(page_score)
    n = sum(sizes)
    cand = [i for i in range(m) if not pinned[i]]
    best = None
    best_key = None
    for k in range(len(cand) + 1):
        for ev in combinations(cand, k):
            removed = sum(sizes[i] for i in ev)
            if n - removed > budget:
                continue
            kept = sum(sizes[i] * page_score[i] for i in cand if i not in ev)
            key = (-kept, len(ev), removed)
            if best_key is None or key < best_key:
                best_key, best = key, tuple(sorted(ev))
    return best


def best_tokens(scores: Sequence[float], pinned: Sequence[bool], budget: int) -> Tuple[int, ...]:
    """Token-level optimum of Eq. 1 by enumeration: indices of the kept tokens
    (pinned forced in), largest kept sum, ties by more kept tokens."""
    n = len(scores)
    forced = [i for i in range(n) if pinned[i]]
    free = [i for i in range(n) if not pinned[i]]
    room = budget - len(forced)
    best, best_key = None, None
    for k in range(0, max(0, min(room, len(free))) + 1):
        for keep in combinations(free, k):
            key = (-sum(scores[i] for i in keep), -k)
            if best_key is None or key < best_key:
                best_key, best = key, tuple(sorted(forced + list(keep)))
    if best is None:
        best = tuple(forced)
    return best
