"""Pure-Python brute force used to pin the NumPy oracle on tiny inputs.

Test infrastructure only.  Sums use ``math.fsum`` (correctly rounded), every
candidate is scored, and prefetch sets are found by enumerating all subsets.
"""
from __future__ import annotations

import itertools
import math
from typing import List, Sequence, Tuple


def cosine_fsum(u: Sequence[float], v: Sequence[float]) -> float:
    """u.v / (|u| |v|) with correctly rounded sums; 0 when a norm is 0."""
    dot = math.fsum(a * b for a, b in zip(u, v))
    nu = math.sqrt(math.fsum(a * a for a in u))
    nv = math.sqrt(math.fsum(b * b for b in v))
    if nu == 0.0 or nv == 0.0:
        return 0.0
    return dot / (nu * nv)


def best_matches(scores: Sequence[float], k: int) -> List[int]:
    """Indices of the k highest scores; ties go to the lower index, NaN last."""
    def key(y):
        s = scores[y]
        return (1, 0.0, y) if math.isnan(s) else (0, -s, y)
    order = sorted(range(len(scores)), key=key)
    return order[:k] + [-1] * max(0, k - len(scores))


def min_cardinality(p: Sequence[float], tau: float) -> int:
    """Smallest |S| over all subsets S of experts with fsum(p[S]) >= tau
    (len(p) if no subset reaches tau), by enumeration."""
    E = len(p)
    for size in range(E + 1):
        for S in itertools.combinations(range(E), size):
            if math.fsum(p[j] for j in S) >= tau:
                return size
    return E


def max_sum_of_size(p: Sequence[float], size: int) -> float:
    """Largest correctly rounded sum over subsets of the given size."""
    return max(math.fsum(p[j] for j in S) for S in itertools.combinations(range(len(p)), size))


def prefetch_set(p: Sequence[float], tau: float, k_min: int, k_max: int) -> Tuple[int, frozenset]:
    """Eq. 6-8 by enumeration: the minimum cardinality k* reaching tau, clamped
    to [k_min, k_max]; among sets of that size, the one with the largest sum,
    ties broken towards lexicographically smaller sorted-by-rank sets."""
    E = len(p)
    kstar = min_cardinality(p, tau)
    kk = min(max(kstar, k_min), k_max)
    rank = sorted(range(E), key=lambda j: (-p[j], j))
    best = None
    best_key = None
    for S in itertools.combinations(range(E), kk):
        s = math.fsum(p[j] for j in S)
        key = (-s, sorted(rank.index(j) for j in S))
        if best_key is None or key < best_key:
            best, best_key = S, key
    return kk, frozenset(best if best is not None else ())
