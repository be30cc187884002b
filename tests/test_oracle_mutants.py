"""Planted mistakes in the oracle (on the CPU only): each plausible slip — a
dropped term, a wrong sign or index, a transposed operand, a reversed tie
rule — must make at least one pin of oracle_checks fail."""
import math

import numpy as np
import pytest

import oracle.finemoe as F
import oracle_checks as C

_orig_select_row = F.select_row
_orig_traj = F.trajectory_scores
_orig_cos_many = F._cosine_many
_orig_rank = F.rank
_orig_threshold = F.threshold


def strict_threshold_select(p, tau, k_min, k_max):
    p = np.asarray(p, dtype=np.float64)
    E = p.shape[0]
    order = np.lexsort((np.arange(E), -p))
    kstar, c = E, 0.0
    for k in range(E + 1):
        if c > tau:                       # ">" instead of ">="
            kstar = k
            break
        if k < E:
            c += p[order[k]]
    kk = min(max(kstar, k_min), k_max)
    return sum(1 << int(order[i]) for i in range(kk)), kk, order


def high_index_first_select(p, tau, k_min, k_max):
    p = np.asarray(p, dtype=np.float64)
    E = p.shape[0]
    order = np.lexsort((-np.arange(E), -p))   # ties: higher expert index first
    kstar, c = E, 0.0
    for k in range(E + 1):
        if c >= tau:
            kstar = k
            break
        if k < E:
            c += p[order[k]]
    kk = min(max(kstar, k_min), k_max)
    return sum(1 << int(order[i]) for i in range(kk)), kk, order


def sum_before_test_select(p, tau, k_min, k_max):
    p = np.asarray(p, dtype=np.float64)
    E = p.shape[0]
    order = np.lexsort((np.arange(E), -p))
    kstar, c = E, 0.0
    for k in range(E):
        c += p[order[k]]                  # adds expert k before testing c_k
        if c >= tau:
            kstar = k
            break
    kk = min(max(kstar, k_min), k_max)
    return sum(1 << int(order[i]) for i in range(kk)), kk, order


def no_cap_select(p, tau, k_min, k_max):
    m, c, order = _orig_select_row(p, tau, k_min, len(p))
    c = max(c, k_min)
    return sum(1 << int(order[i]) for i in range(c)), c, order


def ascending_select(p, tau, k_min, k_max):
    return _orig_select_row(-np.asarray(p, dtype=np.float64), -tau, k_min, k_max)


def prefix_off_by_one(maps64, q64, p):
    return _orig_traj(maps64, q64, min(p + 1, maps64.shape[1]))


def prefix_over_experts(maps64, q64, p):
    n, L, E = maps64.shape
    V = maps64[:, :, :min(p, E)].reshape(n, -1)
    u = q64[:, :min(p, E)].reshape(-1)
    return F._cosine_many(V, u)


def missing_sqrt(V, u):
    dots = V @ u
    nv = np.einsum("ij,ij->i", V, V)      # squared norm used as the norm
    nu = math.sqrt(float(np.dot(u, u)))
    with np.errstate(invalid="ignore", divide="ignore"):
        s = dots / (nv * nu)
    s[(nv == 0) | (nu == 0)] = 0.0
    return s


def no_query_norm(V, u):
    dots = V @ u
    nv = np.sqrt(np.einsum("ij,ij->i", V, V))
    with np.errstate(invalid="ignore", divide="ignore"):
        s = dots / nv
    s[nv == 0] = 0.0
    return s


def rank_high_index_first(scores, k, idx=None):
    s = np.asarray(scores, dtype=np.float64)
    if idx is None:
        idx = np.arange(s.shape[0])
    return _orig_rank(s, k, idx) if s.size == 0 else _rank_rev(s, k, np.asarray(idx))


def _rank_rev(s, k, idx):
    nan = np.isnan(s)
    order = np.lexsort((-idx, -np.where(nan, 0.0, s), nan))[:k]
    oi = np.full(k, -1, dtype=np.int64)
    os_ = np.full(k, -np.inf)
    oi[:order.size] = idx[order]
    os_[:order.size] = s[order]
    return oi, os_


def rank_ascending(scores, k, idx=None):
    s = np.asarray(scores, dtype=np.float64)
    i, _ = _orig_rank(-s, k, idx)
    full_idx = np.arange(s.shape[0]) if idx is None else np.asarray(idx)
    pos = {int(v): j for j, v in enumerate(full_idx)}
    return i, np.array([s[pos[int(v)]] if v >= 0 else -np.inf for v in i])


def unnormalised_blend(rows, scores):
    rows = np.asarray(rows, dtype=np.float64)
    w = [max(float(s), 0.0) for s in scores]
    return sum(w[i] * rows[i] for i in range(rows.shape[0]))


def softmax_weight_blend(rows, scores):
    rows = np.asarray(rows, dtype=np.float64)
    w = np.exp(np.asarray(scores, dtype=np.float64))
    return (w[:, None] * rows).sum(0) / w.sum()


def unclipped_delta(mode, tau, score):
    if mode == F.TAU_DYNAMIC:
        return 1.0 - float(score)
    return _orig_threshold(mode, tau, score)


def score_as_delta(mode, tau, score):
    if mode == F.TAU_DYNAMIC:
        return max(0.0, min(float(score), 1.0))
    return _orig_threshold(mode, tau, score)


_orig_redundancy = F.redundancy
_orig_dedup_slots = F.dedup_slots


def redundancy_swapped_weights(old_maps, old_embs, new_maps, new_embs, dtype, d):
    L = old_maps.shape[1]
    return _orig_redundancy(old_maps, old_embs, new_maps, new_embs, dtype, L - d)


def redundancy_partial_depth(old_maps, old_embs, new_maps, new_embs, dtype, d):
    L = old_maps.shape[1]
    out = np.zeros((new_maps.shape[0], old_maps.shape[0]))
    for x in range(new_maps.shape[0]):
        r = 0.0
        if d > 0:
            r = r + (d / L) * F.semantic_scores(F.widen(old_embs, "bf16"), F.widen(new_embs[x], "bf16"))
        if d < L:
            r = r + ((L - d) / L) * F.trajectory_scores(F.widen(old_maps, dtype), F.widen(new_maps[x], dtype), L - 1)
        out[x] = r
    return out


def dedup_reuses_victims(rdy, size, cap):
    rdy = np.asarray(rdy, dtype=np.float64)
    free = max(0, cap - size)
    out = np.full(rdy.shape[0], -1, dtype=np.int64)
    for x in range(rdy.shape[0]):
        if x < free:
            out[x] = size + x
        elif size > 0:
            out[x] = F.rank(rdy[x], 1)[0][0]
    return out


def dedup_least_redundant(rdy, size, cap):
    return _orig_dedup_slots(-np.asarray(rdy, dtype=np.float64), size, cap)


def dedup_never_appends(rdy, size, cap):
    return _orig_dedup_slots(rdy, size, min(cap, size) if size > 0 else cap)


_orig_research = F.research_schedule


def research_one_layer_late(maps, dtype, Q, k, d):
    return {l: F.match_trajectory(maps, dtype, Q, np.full(Q.shape[0], min(l - d + 1, maps.shape[1])), k)
            for l in range(d + 1, maps.shape[1] + 1)}


def research_all_layers(maps, dtype, Q, k, d):
    return {l: F.match_trajectory(maps, dtype, Q, np.full(Q.shape[0], l), k)
            for l in range(d + 1, maps.shape[1] + 1)}


_orig_priority = F.priority_order


def priority_distance_off_by_one(maps, dtype, idx, score, blend, kind, masks, l_now=None, freq=None, cap=None):
    if kind == F.PRI_PREFETCH:
        return _orig_priority(maps, dtype, idx, score, blend, kind, masks, l_now=[x - 1 for x in l_now], freq=freq,
                              cap=cap)
    return _orig_priority(maps, dtype, idx, score, blend, kind, masks, l_now=l_now, freq=freq, cap=cap)


def priority_ascending(maps, dtype, idx, score, blend, kind, masks, l_now=None, freq=None, cap=None):
    order, pri, cnt = _orig_priority(maps, dtype, idx, score, blend, kind, masks, l_now=l_now, freq=freq, cap=cap)
    for b in range(order.shape[0]):
        order[b, :cnt[b]] = order[b, :cnt[b]][::-1]
        pri[b, :cnt[b]] = pri[b, :cnt[b]][::-1]
    return order, pri, cnt


def evict_by_ratio(maps, dtype, idx, score, blend, kind, masks, l_now=None, freq=None, cap=None):
    if kind == F.PRI_EVICT:
        freq = np.where(freq == 0, 0, 1.0 / np.where(freq == 0, 1, freq)).astype(np.float32)
    return _orig_priority(maps, dtype, idx, score, blend, kind, masks, l_now=l_now, freq=freq, cap=cap)


_orig_activated = F.activated


def activated_high_index_first(p, K):
    p = np.asarray(p, dtype=np.float64)
    return int(bin(_orig_activated(p[::-1], K))[2:].zfill(len(p))[::-1], 2) if len(p) else 0


def activated_one_short(p, K):
    return _orig_activated(p, max(K - 1, 0))


_orig_guide_row = F.guide_row
_orig_blend_rows = F.blend_rows


def guide_keeps_missing(maps, dtype, idx_row, score_row, blend, l):
    if blend != F.BLEND_SCORE:
        return _orig_guide_row(maps, dtype, idx_row, score_row, blend, l)
    rows = np.stack([F.widen(maps[idx_row[i]], dtype)[l] for i in range(len(idx_row))])   # -1 reads maps[-1]
    return F.blend_rows(rows, list(score_row))


def guide_top1_weight_for_all(maps, dtype, idx_row, score_row, blend, l):
    if blend != F.BLEND_SCORE:
        return _orig_guide_row(maps, dtype, idx_row, score_row, blend, l)
    valid = [i for i in range(len(idx_row)) if idx_row[i] >= 0]
    rows = np.stack([F.widen(maps[idx_row[i], l], dtype) for i in valid])
    return F.blend_rows(rows, [score_row[0]] * len(valid))      # every row weighted by the best score


def blend_nan_weight_kept(rows, scores):
    rows = np.asarray(rows, dtype=np.float64)
    w = [0.0 if float(s) <= 0.0 else float(s) for s in scores]  # NaN is not <= 0: kept as a NaN weight
    if sum(w) == 0.0:
        w = [1.0] * len(w)
    num = np.zeros(rows.shape[1])
    den = 0.0
    for i in range(rows.shape[0]):
        num = num + w[i] * rows[i]
        den = den + w[i]
    return num / den


def merge_forgets_earlier_chunks(best_i, best_s, new_i, new_s, k):
    return F.rank(new_s, k, new_i)


_orig_traj_many = F.trajectory_scores_many


def cols_missing_sqrt(V, U):
    dots = V @ U
    nv = np.einsum("ij,ij->i", V, V)[:, None]          # squared norm used as the norm
    nu = np.sqrt(np.einsum("ij,ij->j", U, U))[None, :]
    with np.errstate(invalid="ignore", divide="ignore"):
        s = dots / (nv * nu)
    s[((nv == 0) | (nu == 0)) & ~np.isnan(dots)] = 0.0
    return s


def cols_query_norm_of_first(V, U):
    dots = V @ U
    nv = np.sqrt(np.einsum("ij,ij->i", V, V))[:, None]
    nu = math.sqrt(float(U[:, 0] @ U[:, 0]))             # every column divided by the first one's norm
    with np.errstate(invalid="ignore", divide="ignore"):
        s = dots / (nv * nu)
    s[(nv[:, 0] == 0) | (nu == 0)] = 0.0
    return s


def traj_many_prefix_off_by_one(maps64, Q64, p):
    return _orig_traj_many(maps64, Q64, min(p + 1, maps64.shape[1]))


def traj_many_layers_transposed(maps64, Q64, p):
    n, L, E = maps64.shape
    V = np.ascontiguousarray(maps64.transpose(0, 2, 1)).reshape(n, L * E)[:, :p * E]   # expert-major flattening
    U = np.ascontiguousarray(Q64).reshape(Q64.shape[0], L * E)[:, :p * E].T
    return F._cosine_cols(V, U)


MUTANTS = [
    ("select_row", strict_threshold_select),
    ("select_row", high_index_first_select),
    ("select_row", sum_before_test_select),
    ("select_row", no_cap_select),
    ("select_row", ascending_select),
    ("trajectory_scores", prefix_off_by_one),
    ("trajectory_scores", prefix_over_experts),
    ("_cosine_many", missing_sqrt),
    ("_cosine_many", no_query_norm),
    ("rank", rank_high_index_first),
    ("rank", rank_ascending),
    ("blend_rows", unnormalised_blend),
    ("blend_rows", softmax_weight_blend),
    ("threshold", unclipped_delta),
    ("threshold", score_as_delta),
    ("redundancy", redundancy_swapped_weights),
    ("redundancy", redundancy_partial_depth),
    ("dedup_slots", dedup_reuses_victims),
    ("dedup_slots", dedup_least_redundant),
    ("dedup_slots", dedup_never_appends),
    ("research_schedule", research_one_layer_late),
    ("research_schedule", research_all_layers),
    ("priority_order", priority_distance_off_by_one),
    ("priority_order", priority_ascending),
    ("priority_order", evict_by_ratio),
    ("activated", activated_high_index_first),
    ("activated", activated_one_short),
    ("guide_row", guide_keeps_missing),
    ("guide_row", guide_top1_weight_for_all),
    ("blend_rows", blend_nan_weight_kept),
    ("_merge", merge_forgets_earlier_chunks),
    ("_cosine_cols", cols_missing_sqrt),
    ("_cosine_cols", cols_query_norm_of_first),
    ("trajectory_scores_many", traj_many_prefix_off_by_one),
    ("trajectory_scores_many", traj_many_layers_transposed),
]


@pytest.mark.parametrize("name,mutant", MUTANTS, ids=lambda x: getattr(x, "__name__", str(x)))
def test_planted_mistake_is_caught(monkeypatch, name, mutant):
    monkeypatch.setattr(F, name, mutant)
    failed = []
    for check in C.ALL_CHECKS:
        try:
            check()
        except Exception:  # noqa: BLE001 - any failure of a pin counts as caught
            failed.append(check.__name__)
    assert failed, f"no pin catches the planted mistake {mutant.__name__}"
