"""NumPy float64 oracle of FineMoE's expert-map search and prefetch selection.

Test infrastructure only (see the package docstring).  Inputs are the arrays
the synthetic generator draws: float32 arrays, or bf16 values carried as
uint16 bit patterns.  Both widen to float64 exactly, and every sum below is
taken in float64.

Conventions where the paper leaves a choice open (each is listed, with its
reason, in the design notes of the repository):

* equal scores: the lower store index ranks first; NaN scores rank last;
* a zero-norm vector has cosine 0 with everything;
* equal probabilities: the lower expert index is picked first;
* the threshold test is ``>=`` (Eq. 7); if no prefix reaches it, all experts
  are taken before the cap;
* a store with fewer than k entries fills the rest with index -1 and score
  -inf, and a query whose best index is -1 selects nothing.
"""
from __future__ import annotations

import math
from typing import Tuple

import numpy as np

TAU_FIXED = 0
TAU_DYNAMIC = 1
BLEND_NONE = 0
BLEND_SCORE = 1

_CHUNK = 16384


# ---------------------------------------------------------------- inputs

def widen(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of a float32 array or of bf16 bit patterns."""
    if dtype == "bf16":
        a = np.ascontiguousarray(arr, dtype=np.uint16)
        return np.left_shift(a, 16, dtype=np.uint32).view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(arr, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


# ---------------------------------------------------------------- cosine (Eq. 4, Eq. 5)

def cosine(u: np.ndarray, v: np.ndarray) -> float:
    """Cosine similarity u.v / (|u| |v|) in float64; 0 if either norm is 0."""
    u = np.asarray(u, dtype=np.float64).ravel()
    v = np.asarray(v, dtype=np.float64).ravel()
    nu = math.sqrt(float(np.dot(u, u)))
    nv = math.sqrt(float(np.dot(v, v)))
    dot = float(np.dot(u, v))
    if math.isnan(dot) or math.isnan(nu) or math.isnan(nv):
        return math.nan
    if nu == 0.0 or nv == 0.0:
        return 0.0
    return dot / (nu * nv)


def _cosine_many(V: np.ndarray, u: np.ndarray) -> np.ndarray:
    """Cosine of every row of V with u (float64), same conventions as cosine()."""
    dots = V @ u
    nv = np.sqrt(np.einsum("ij,ij->i", V, V))
    nu = math.sqrt(float(np.dot(u, u)))
    with np.errstate(invalid="ignore", divide="ignore"):
        s = dots / (nv * nu)
    zero = (nv == 0.0) | (nu == 0.0)
    s[zero & ~np.isnan(dots) & ~np.isnan(nv)] = 0.0
    if math.isnan(nu):
        s[:] = np.nan
    return s


def _cosine_cols(V: np.ndarray, U: np.ndarray) -> np.ndarray:
    """Cosine of every row of V [n][m] with every column of U [m][c] (float64),
    as a [n][c] array, with the conventions of cosine()."""
    dots = V @ U
    nv = np.sqrt(np.einsum("ij,ij->i", V, V))[:, None]
    nu = np.sqrt(np.einsum("ij,ij->j", U, U))[None, :]
    with np.errstate(invalid="ignore", divide="ignore"):
        s = dots / (nv * nu)
    zero = (nv == 0.0) | (nu == 0.0)
    s[zero & ~np.isnan(dots) & ~np.isnan(nv) & ~np.isnan(nu)] = 0.0
    s[:, np.isnan(nu[0])] = np.nan
    return s


def trajectory_scores(maps64: np.ndarray, q64: np.ndarray, p: int) -> np.ndarray:
    """Eq. 5: cosine between the observed trajectory of the first ``p`` layers of
    query ``q64`` [L][E] and the same ``p`` layers of every stored map
    ``maps64`` [n][L][E], both flattened over (layer, expert)."""
    n, L, E = maps64.shape
    V = maps64[:, :p, :].reshape(n, p * E)
    u = q64[:p, :].reshape(p * E)
    return _cosine_many(V, u)


def trajectory_scores_many(maps64: np.ndarray, Q64: np.ndarray, p: int) -> np.ndarray:
    """Eq. 5 for several queries observed to the same depth ``p``: [n][c] cosines
    between the first ``p`` layers of every stored map (maps64 [n][L][E]) and of
    every query (Q64 [c][L][E]), flattened over (layer, expert).  In a map
    flattened layer by layer, its first p layers are its first p * E values."""
    n, L, E = maps64.shape
    V = np.ascontiguousarray(maps64).reshape(n, L * E)[:, :p * E]
    U = np.ascontiguousarray(Q64).reshape(Q64.shape[0], L * E)[:, :p * E].T
    return _cosine_cols(V, U)


def semantic_scores(embs64: np.ndarray, qs64: np.ndarray) -> np.ndarray:
    """Eq. 4: cosine between a query embedding [d] and every stored embedding [n][d]."""
    return _cosine_many(embs64, qs64)


# ---------------------------------------------------------------- ranking

def rank(scores: np.ndarray, k: int, idx: np.ndarray = None) -> Tuple[np.ndarray, np.ndarray]:
    """The k best entries by (score descending, index ascending), NaN last.

    ``idx`` gives the store index of each score (default 0..n-1).  Missing
    entries (fewer than k scores) are returned as index -1, score -inf.
    """
    s = np.asarray(scores, dtype=np.float64)
    if idx is None:
        idx = np.arange(s.shape[0], dtype=np.int64)
    idx = np.asarray(idx, dtype=np.int64)
    nan = np.isnan(s)
    order = np.lexsort((idx, -np.where(nan, 0.0, s), nan))
    top = order[:k]
    out_i = np.full(k, -1, dtype=np.int64)
    out_s = np.full(k, -np.inf, dtype=np.float64)
    out_i[:top.size] = idx[top]
    out_s[:top.size] = s[top]
    return out_i, out_s


def _merge(best_i, best_s, new_i, new_s, k):
    keep = best_i >= 0
    return rank(np.concatenate([best_s[keep], new_s]), k, np.concatenate([best_i[keep], new_i]))


def match_trajectory(maps: np.ndarray, dtype: str, Q: np.ndarray, depth: np.ndarray, k: int,
                     n: int = None) -> Tuple[np.ndarray, np.ndarray]:
    """Trajectory search (Section 4.2.2): for each query b, the k stored maps with
    the highest Eq. 5 score over the first depth[b] layers (clamped to [1, L]).

    maps [n][L][E], Q [B][L][E] (dtype "f32" or "bf16"), depth [B].
    Returns idx [B][k] (int64, -1 if missing) and score [B][k] (float64).
    """
    n = maps.shape[0] if n is None else n
    B, L, E = Q.shape
    depth = np.clip(np.asarray(depth, dtype=np.int64), 1, L)
    Q64 = widen(Q, dtype)
    out_i = np.full((B, k), -1, dtype=np.int64)
    out_s = np.full((B, k), -np.inf, dtype=np.float64)
    for a in range(0, n, _CHUNK):
        b = min(a + _CHUNK, n)
        M = widen(maps[a:b], dtype)
        ids = np.arange(a, b, dtype=np.int64)
        S = np.empty((b - a, B), dtype=np.float64)
        for p in np.unique(depth):
            qs = np.flatnonzero(depth == p)
            S[:, qs] = trajectory_scores_many(M, Q64[qs], int(p))
        for q in range(B):
            out_i[q], out_s[q] = _merge(out_i[q], out_s[q], ids, S[:, q], k)
    return out_i, out_s


def match_semantic(embs: np.ndarray, Qs: np.ndarray, k: int, n: int = None) -> Tuple[np.ndarray, np.ndarray]:
    """Semantic search (Section 4.2.1): for each query embedding, the k stored
    embeddings with the highest Eq. 4 score.  embs [n][d], Qs [B][d], bf16 bits."""
    n = embs.shape[0] if n is None else n
    B = Qs.shape[0]
    Q64 = widen(Qs, "bf16")
    out_i = np.full((B, k), -1, dtype=np.int64)
    out_s = np.full((B, k), -np.inf, dtype=np.float64)
    for a in range(0, n, _CHUNK):
        b = min(a + _CHUNK, n)
        X = widen(embs[a:b], "bf16")
        ids = np.arange(a, b, dtype=np.int64)
        S = _cosine_cols(X, Q64.T)
        for q in range(B):
            out_i[q], out_s[q] = _merge(out_i[q], out_s[q], ids, S[:, q], k)
    return out_i, out_s


def research_schedule(maps: np.ndarray, dtype: str, Q: np.ndarray, k: int, d: int):
    """The per-layer trajectory re-search of one pass (Section 4.2.2): the
    prediction for target layer l in [d+1, L] (1-based) uses the trajectory
    of layers 1 .. l-d, i.e. a search of prefix depth p = l - d for every
    query.  Returns {l: (idx [B][k], score [B][k])} for l = d+1 .. L, each a
    plain ``match_trajectory`` at that depth."""
    n, L, E = maps.shape
    if not 0 <= d < L:
        raise ValueError(f"prefetch distance {d} outside [0, {L})")
    B = Q.shape[0]
    out = {}
    for l in range(d + 1, L + 1):
        p = l - d
        out[l] = match_trajectory(maps, dtype, Q, np.full(B, p, dtype=np.int64), k)
    return out


# ---------------------------------------------------------------- store deduplication (Section 4.4)

def redundancy(old_maps: np.ndarray, old_embs, new_maps: np.ndarray, new_embs, dtype: str,
               d: int) -> np.ndarray:
    """Pairwise redundancy RDY[x][y] of Section 4.4 between new iterations x
    (rows) and stored iterations y (columns):

        RDY[x][y] = (d / L) * score_sem[x][y] + ((L - d) / L) * score_traj[x][y]

    with score_sem the Eq. 4 cosine of the embeddings and score_traj the Eq. 5
    cosine over all L layers (a finished iteration has its whole map), d the
    prefetch distance (0 <= d <= L).  A term whose weight is 0 is left out, so
    a store without embeddings is deduplicated with d = 0 and a NaN in an
    unused score does not reach RDY.  The weighted terms are added in that
    order, in float64.

    old_maps [s][L][E], new_maps [m][L][E] of ``dtype``; old_embs [s][d_emb]
    and new_embs [m][d_emb] bf16 bits (may be None when d == 0).
    Returns float64 [m][s].
    """
    s, L, E = old_maps.shape
    m = new_maps.shape[0]
    if not 0 <= d <= L:
        raise ValueError(f"prefetch distance {d} outside [0, {L}]")
    w_sem = d / L
    w_traj = (L - d) / L
    out = np.zeros((m, s), dtype=np.float64)
    for a in range(0, s, _CHUNK):
        b = min(a + _CHUNK, s)
        M = widen(old_maps[a:b], dtype) if w_traj > 0.0 else None
        X = widen(old_embs[a:b], "bf16") if w_sem > 0.0 else None
        for x in range(m):
            r = np.zeros(b - a, dtype=np.float64)
            if w_sem > 0.0:
                r = r + w_sem * semantic_scores(X, widen(new_embs[x], "bf16"))
            if w_traj > 0.0:
                r = r + w_traj * trajectory_scores(M, widen(new_maps[x], dtype), L)
            out[x, a:b] = r
    return out


def dedup_slots(rdy: np.ndarray, size: int, cap: int) -> np.ndarray:
    """Where each new iteration x = 0..m-1 of a batch is written (Section 4.4).

    While the store has room, new iterations are appended in batch order
    (slots size, size + 1, ...).  Once it is full, each remaining x, in batch
    order, replaces the stored iteration it is most redundant with: the
    highest RDY[x][y] (lower y first on equal values, NaN last) among the
    iterations stored before this batch that no earlier x has replaced.  An x
    left without such a candidate is dropped (slot -1).

    rdy [m][size] float64 (rows of appended x are not read).
    Returns slots [m] int64.
    """
    rdy = np.asarray(rdy, dtype=np.float64)
    m = rdy.shape[0]
    free = max(0, cap - size)
    slots = np.full(m, -1, dtype=np.int64)
    taken = np.zeros(size, dtype=bool)
    for x in range(m):
        if x < free:
            slots[x] = size + x
            continue
        cand = np.flatnonzero(~taken)
        if cand.size == 0:
            continue
        best, _ = rank(rdy[x, cand], 1, cand)
        slots[x] = best[0]
        taken[best[0]] = True
    return slots


def insert_dedup(old_maps: np.ndarray, old_embs, cap: int, new_maps: np.ndarray, new_embs,
                 dtype: str, d: int) -> np.ndarray:
    """Slots of a batch of new iterations inserted into a store holding
    ``old_*`` (size = len(old_maps)) of capacity ``cap``: RDY is computed for
    the new iterations that find the store full, then ``dedup_slots``."""
    size = old_maps.shape[0]
    m = new_maps.shape[0]
    free = max(0, cap - size)
    rdy = np.zeros((m, size), dtype=np.float64)
    if m > free and size > 0:
        rdy[free:] = redundancy(old_maps, old_embs, new_maps[free:],
                                None if new_embs is None else new_embs[free:], dtype, d)
    return dedup_slots(rdy, size, cap)


# ---------------------------------------------------------------- threshold and selection (Section 4.3)

def threshold(mode: int, tau: float, score: float) -> float:
    """The probability mass a prefetch set must reach.

    FIXED: the given tau (a float32 parameter, widened exactly).
    DYNAMIC: delta = Clip(1 - score, 0, 1) of Section 4.3; a NaN score gives 1.
    """
    if mode == TAU_FIXED:
        return float(np.float32(tau))
    if mode == TAU_DYNAMIC:
        s = float(score)
        if math.isnan(s):
            return 1.0
        return max(0.0, min(1.0 - s, 1.0))
    raise ValueError(mode)


def select_row(p: np.ndarray, tau: float, k_min: int, k_max: int) -> Tuple[int, int, np.ndarray]:
    """Eq. 6-8 on one layer's probabilities ``p`` [E] (float64 values).

    Experts are taken in order of probability (highest first, lower index
    first on equal values, NaN last); k* is the smallest k whose running sum of
    the first k taken reaches tau (k* = E if none does); the set is the first
    min(max(k*, k_min), k_max) of that order.
    Returns (mask with bit j = expert j, count, order).
    """
    p = np.asarray(p, dtype=np.float64)
    E = p.shape[0]
    nan = np.isnan(p)
    order = np.lexsort((np.arange(E), -np.where(nan, 0.0, p), nan))
    kstar = E
    c = 0.0
    for k in range(E + 1):
        if c >= tau:
            kstar = k
            break
        if k < E:
            c = c + float(p[order[k]])
    kk = min(max(kstar, k_min), k_max)
    mask = 0
    for i in range(kk):
        mask |= 1 << int(order[i])
    return mask, kk, order


def blend_rows(rows: np.ndarray, scores: np.ndarray) -> np.ndarray:
    """Similarity-weighted mean of k rows: sum_i w_i row_i / sum_i w_i with
    w_i = max(score_i, 0) (a NaN score weighs 0), summed in order
    i = 0..k-1; if every weight is 0 the plain mean is used."""
    rows = np.asarray(rows, dtype=np.float64)
    w = [float(s) if float(s) > 0.0 else 0.0 for s in scores]
    if sum(w) == 0.0:
        w = [1.0] * len(w)
    num = np.zeros(rows.shape[1], dtype=np.float64)
    den = 0.0
    for i in range(rows.shape[0]):
        num = num + w[i] * rows[i]
        den = den + w[i]
    return num / den


def select_prefetch(maps: np.ndarray, dtype: str, idx: np.ndarray, score: np.ndarray,
                    lb: np.ndarray, le: np.ndarray, mode: int, tau: float, k_min: int, k_max: int,
                    blend: int) -> Tuple[np.ndarray, np.ndarray]:
    """Prefetch sets for each query b and layer l in [lb[b], le[b]).

    The guiding row is layer l of the best match idx[b][0] (BLEND_NONE), or
    the similarity-weighted mean of layer l over the valid matches in idx[b]
    (BLEND_SCORE).  The threshold comes from ``threshold`` with the best
    match's score.  Layers outside the range, and queries without a match,
    get an empty set.  Returns mask [B][L] uint64 and count [B][L] uint8.
    """
    n, L, E = maps.shape
    idx = np.asarray(idx, dtype=np.int64)
    score = np.asarray(score, dtype=np.float64)
    B = idx.shape[0]
    mask = np.zeros((B, L), dtype=np.uint64)
    count = np.zeros((B, L), dtype=np.uint8)
    for b in range(B):
        if idx[b, 0] < 0:
            continue
        t = threshold(mode, tau, score[b, 0])
        lo = max(0, int(lb[b]))
        hi = min(L, int(le[b]))
        for l in range(lo, hi):
            p = guide_row(maps, dtype, idx[b], score[b], blend, l)
            m, c, _ = select_row(p, t, k_min, k_max)
            mask[b, l] = np.uint64(m)
            count[b, l] = c
    return mask, count


def guide_row(maps: np.ndarray, dtype: str, idx_row: np.ndarray, score_row: np.ndarray, blend: int,
              l: int) -> np.ndarray:
    """The guiding probabilities of layer l for one query [E] (float64):
    layer l of the best match idx_row[0] (BLEND_NONE), or the
    similarity-weighted mean of layer l over the valid matches (BLEND_SCORE,
    ``blend_rows``)."""
    if blend == BLEND_SCORE:
        valid = [i for i in range(len(idx_row)) if idx_row[i] >= 0]
        rows = np.stack([widen(maps[idx_row[i], l], dtype) for i in valid])
        return blend_rows(rows, [score_row[i] for i in valid])
    return widen(maps[idx_row[0], l], dtype)


# ---------------------------------------------------------------- misses (Section 3, problem formulation)

def activated(p: np.ndarray, K: int) -> int:
    """The K experts a gate with probabilities p [E] activates: the K
    highest (lower index first on equal values, NaN last), as a bit mask."""
    p = np.asarray(p, dtype=np.float64)
    E = p.shape[0]
    nan = np.isnan(p)
    order = np.lexsort((np.arange(E), -np.where(nan, 0.0, p), nan))
    m = 0
    for j in order[:K]:
        m |= 1 << int(j)
    return m


def miss_counts(Q: np.ndarray, dtype: str, masks: np.ndarray, K: int, lb: np.ndarray, le: np.ndarray) -> np.ndarray:
    """Misses of the prefetch sets (Section 3): R_{l,j} = 1 iff expert j of
    layer l is activated and not in the set; summed over j for every query b
    and layer l in [lb[b], le[b]) (clamped to [0, L]), 0 elsewhere.  The
    activated experts are the top-K of the query's own gate probabilities
    Q [B][L][E] at that layer (``activated``); masks [B][L] are the sets.
    Returns [B][L] uint8."""
    Q64 = widen(Q, dtype)
    B, L, E = Q64.shape
    out = np.zeros((B, L), dtype=np.uint8)
    for b in range(B):
        for l in range(max(0, int(lb[b])), min(L, int(le[b]))):
            act = activated(Q64[b, l], K)
            out[b, l] = bin(act & ~int(masks[b, l])).count("1")
    return out


# ---------------------------------------------------------------- prefetch and eviction priorities (Section 4.5)

PRI_PREFETCH = 0
PRI_EVICT = 1


def priority_order(maps: np.ndarray, dtype: str, idx: np.ndarray, score: np.ndarray, blend: int, kind: int,
                   masks: np.ndarray, l_now=None, freq=None, cap: int = None):
    """Experts of each query in the order of the Section 4.5 priorities.

    PRI_PREFETCH: the candidates are the experts j of the query's prefetch
    set masks[b][l] (bit j) in the layers after the current one, l > l_now[b];
    PRI = p_{l,j} / (l - l_now[b]).
    PRI_EVICT: the candidates are the cached experts (masks[l], one mask per
    layer for the cache); PRI = 1 / (p_{l,j} * freq[l][j]) with freq the
    cache's visit counts.
    p_{l,j} is the query's guiding probability (``guide_row``, as for the
    selection).  PRI is computed in float64 and rounded to float32; the
    candidates are ordered by PRI descending, lower l * E + j first on equal
    values, NaN last.  A query without a match has no candidates.

    Returns order [B][cap] int64 (l * E + j, -1 past the candidates), pri
    [B][cap] float32 (-inf past the candidates) and count [B] (all candidates,
    before the first ``cap`` are kept; cap defaults to L * E).
    """
    n, L, E = maps.shape
    idx = np.asarray(idx, dtype=np.int64)
    score = np.asarray(score, dtype=np.float64)
    B = idx.shape[0]
    cap = L * E if cap is None else cap
    order = np.full((B, cap), -1, dtype=np.int64)
    pri = np.full((B, cap), -np.inf, dtype=np.float32)
    count = np.zeros(B, dtype=np.int64)
    for b in range(B):
        if idx[b, 0] < 0:
            continue
        cand = []
        for l in range(L):
            if kind == PRI_PREFETCH:
                if l <= int(l_now[b]):
                    continue
                bits = int(masks[b, l])
            else:
                bits = int(masks[l])
            if bits == 0:
                continue
            p = guide_row(maps, dtype, idx[b], score[b], blend, l)
            for j in range(E):
                if not (bits >> j) & 1:
                    continue
                with np.errstate(divide="ignore", invalid="ignore"):
                    if kind == PRI_PREFETCH:
                        v = np.float64(p[j]) / np.float64(l - int(l_now[b]))
                    else:
                        v = np.float64(1.0) / (np.float64(p[j]) * np.float64(np.float32(freq[l, j])))
                cand.append((np.float32(v), l * E + j))
        key = lambda c: (1, 0.0, c[1]) if np.isnan(c[0]) else (0, -float(c[0]), c[1])
        cand.sort(key=key)
        count[b] = len(cand)
        for i, (v, e) in enumerate(cand[:cap]):
            order[b, i] = e
            pri[b, i] = v
    return order, pri, count
