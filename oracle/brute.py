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


def redundancy_fsum(old_map: Sequence[Sequence[float]], old_emb, new_map: Sequence[Sequence[float]], new_emb,
                    d: int) -> float:
    """RDY of one (new, stored) pair (Section 4.4) from correctly rounded
    cosines: (d/L) * cos(embeddings) + ((L-d)/L) * cos(whole maps flattened),
    a zero-weight term left out."""
    L = len(old_map)
    r = 0.0
    if d > 0:
        r += (d / L) * cosine_fsum(list(new_emb), list(old_emb))
    if d < L:
        flat_new = [v for row in new_map for v in row]
        flat_old = [v for row in old_map for v in row]
        r += ((L - d) / L) * cosine_fsum(flat_new, flat_old)
    return r


def dedup_by_enumeration(rdy: Sequence[Sequence[float]], size: int, cap: int) -> List[int]:
    """Slots of a batch by exhaustive search (Section 4.4, no NaN in rdy).

    The first cap - size new iterations are appended.  Over every injective
    assignment of the remaining ones (in batch order) to stored iterations
    (as many as can be assigned, the rest -1), take the one whose sequence of
    (RDY, -index) pairs is lexicographically largest: the first replacing
    iteration gets its most redundant entry, the next the most redundant of
    the rest, and so on."""
    m = len(rdy)
    free = max(0, cap - size)
    head = [size + x for x in range(min(m, free))]
    rest = list(range(min(m, free), m))
    r = min(len(rest), size)
    best, best_key = None, None
    for perm in itertools.permutations(range(size), r):
        key = []
        for x, y in zip(rest, perm):
            key += [rdy[x][y], -y]
        if best_key is None or key > best_key:
            best, best_key = perm, key
    tail = list(best) if best is not None else []
    return head + tail + [-1] * (len(rest) - len(tail))


def priority_list(p_rows: Sequence[Sequence[float]], bits: Sequence[int], pri_of) -> List[Tuple[float, int]]:
    """Section 4.5 ordering by exhaustive comparison: every candidate (l, j)
    with bit j of bits[l] set gets pri_of(l, j, p) with p its guiding
    probability (a Python float rounded as the caller defines); a candidate
    is placed after exactly
    the candidates that beat it (larger priority, or equal and lower
    l * E + j; NaN below every number)."""
    E = len(p_rows[0])
    cand = [(pri_of(l, j, float(p_rows[l][j])), l * E + j)
            for l in range(len(bits)) for j in range(E) if (bits[l] >> j) & 1]

    def beats(a, b):
        an, bn = math.isnan(a[0]), math.isnan(b[0])
        if an or bn:
            return (not an and bn) or (an and bn and a[1] < b[1])
        return a[0] > b[0] or (a[0] == b[0] and a[1] < b[1])

    out = [None] * len(cand)
    for c in cand:
        out[sum(1 for d in cand if d is not c and beats(d, c))] = c
    return out


def misses_by_enumeration(p: Sequence[float], K: int, chosen: int) -> int:
    """Activated experts outside the set ``chosen`` (a bit mask), with the
    activated set found as the K-subset of largest fsum (ties: the subset
    whose sorted indices come first), by enumeration (no NaN in p)."""
    E = len(p)
    best, best_key = None, None
    for S in itertools.combinations(range(E), min(K, E)):
        key = (-math.fsum(p[j] for j in S), sorted(S))
        if best_key is None or key < best_key:
            best, best_key = S, key
    return sum(1 for j in best if not (chosen >> j) & 1)


def blend_fsum(rows: Sequence[Sequence[float]], scores: Sequence[float]) -> List[float]:
    """Similarity-weighted mean of the given rows with correctly rounded sums:
    weight max(score, 0), a NaN score weighing 0, and equal weights when every
    weight is 0 (the blend extension used with several matches)."""
    w = [0.0 if math.isnan(s) or s <= 0.0 else float(s) for s in scores]
    if math.fsum(w) == 0.0:
        w = [1.0] * len(w)
    den = math.fsum(w)
    E = len(rows[0])
    return [math.fsum(w[i] * rows[i][j] for i in range(len(rows))) / den for j in range(E)]


def guide_fsum(maps, idx_row: Sequence[int], score_row: Sequence[float], blend: bool, l: int) -> List[float]:
    """Guiding probabilities of layer l for one query, from a list of stored
    maps (maps[y][l][j] as Python floats): the best match's row, or with
    ``blend`` the weighted mean over the matches whose index is not -1."""
    if not blend:
        return [float(v) for v in maps[idx_row[0]][l]]
    keep = [i for i, y in enumerate(idx_row) if y >= 0]
    return blend_fsum([[float(v) for v in maps[idx_row[i]][l]] for i in keep], [score_row[i] for i in keep])
