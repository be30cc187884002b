"""GPU-vs-oracle parity harness shared by the GPU tests, smoke() and bench.py.

Runs one workload through the C ABI (via the package binding) and through the
CPU oracle on the same generated arrays, then compares:

* scores: every returned score is within SCORE_TOL (absolute on the cosine,
  i.e. relative to |u| |v|) of the oracle's float64 score of the same index;
* indices: the j-th returned index must be the oracle's j-th index unless the
  oracle's j-th score is within the near-tie margin 2 * SCORE_TOL of a
  neighbour; inside a near-tie any index whose oracle score is within the
  margin of the true j-th score is accepted (and counted);
* prefetch sets: bit-exact against the oracle's selection run on the GPU's
  own indices and scores (both sides sum in float64 in the same order).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

import oracle
import synth

SCORE_TOL = 1e-5


def to_device(arr: np.ndarray, dtype: str):
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    elif dtype == "f32":
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr))
    return t.cuda()


@dataclasses.dataclass
class GpuResult:
    idx: np.ndarray
    score: np.ndarray
    mask: np.ndarray
    count: np.ndarray
    flags: int


def run_gpu(s: synth.Spec, a: Dict[str, np.ndarray], cap: Optional[int] = None, tau_mode: Optional[int] = None,
            tau: Optional[float] = None, k_min: Optional[int] = None, k_max: Optional[int] = None,
            insert_chunks: int = 1, max_depth: Optional[int] = None) -> GpuResult:
    import torch
    import paper_2502_05370_amd as fm
    n = a["maps"].shape[0]
    store = fm.Store(cap if cap is not None else max(n, 1), s.L, s.E, s.d_emb, s.map_dtype)
    maps = to_device(a["maps"], s.map_dtype)
    embs = to_device(a["embs"], "bf16") if s.d_emb else None
    bounds = np.linspace(0, n, insert_chunks + 1).astype(int)
    for lo, hi in zip(bounds[:-1], bounds[1:]):
        if hi > lo:
            store.insert(maps[lo:hi], embs[lo:hi] if embs is not None else None)
    B = s.B
    idx = torch.empty((B, s.k), dtype=torch.int32, device="cuda")
    score = torch.empty((B, s.k), dtype=torch.float32, device="cuda")
    if s.B_sem:
        fm.match_semantic(store, to_device(a["q_sem"], "bf16"), s.k, out=(idx[:s.B_sem], score[:s.B_sem]))
    if s.B_traj:
        fm.match_trajectory(store, to_device(a["q_traj"], s.map_dtype), to_device(a["depth"], "i32"), s.k,
                            max_depth=max_depth if max_depth is not None else s.L,
                            out=(idx[s.B_sem:], score[s.B_sem:]))
    mask, count = fm.select_prefetch(
        store, idx, score, to_device(a["lb"], "i32"), to_device(a["le"], "i32"),
        tau=s.tau if tau is None else tau, k_min=s.k_min if k_min is None else k_min,
        k_max=s.k_max if k_max is None else k_max, mode=s.tau_mode if tau_mode is None else tau_mode,
        blend=s.blend)
    flags = store.check()
    torch.cuda.synchronize()
    return GpuResult(idx.cpu().numpy().astype(np.int64), score.cpu().numpy().astype(np.float64),
                     mask.cpu().numpy().view(np.uint64), count.cpu().numpy(), flags)


def oracle_match(s: synth.Spec, a: Dict[str, np.ndarray], rows: Optional[np.ndarray] = None):
    """Oracle top-k for the queries in ``rows`` (all by default), in batch order."""
    B = s.B
    rows = np.arange(B) if rows is None else np.asarray(rows)
    idx = np.full((len(rows), s.k), -1, dtype=np.int64)
    sc = np.full((len(rows), s.k), -np.inf)
    sem = rows[rows < s.B_sem]
    tra = rows[rows >= s.B_sem] - s.B_sem
    pos = {int(r): i for i, r in enumerate(rows)}
    if sem.size:
        i, v = oracle.match_semantic(a["embs"], a["q_sem"][sem], s.k)
        for j, r in enumerate(sem):
            idx[pos[int(r)]], sc[pos[int(r)]] = i[j], v[j]
    if tra.size:
        i, v = oracle.match_trajectory(a["maps"], s.map_dtype, a["q_traj"][tra], a["depth"][tra], s.k)
        for j, r in enumerate(tra):
            idx[pos[int(r + s.B_sem)]], sc[pos[int(r + s.B_sem)]] = i[j], v[j]
    return idx, sc


def oracle_score_of(s: synth.Spec, a: Dict[str, np.ndarray], row: int, y: int) -> float:
    """Oracle float64 score of query ``row`` against stored index ``y``."""
    if row < s.B_sem:
        return oracle.cosine(oracle.widen(a["q_sem"][row], "bf16"), oracle.widen(a["embs"][y], "bf16"))
    b = row - s.B_sem
    p = int(np.clip(a["depth"][b], 1, s.L))
    return oracle.cosine(oracle.widen(a["q_traj"][b, :p], s.map_dtype), oracle.widen(a["maps"][y, :p], s.map_dtype))


@dataclasses.dataclass
class MatchReport:
    checked: int = 0
    near_ties: int = 0
    failures: list = dataclasses.field(default_factory=list)
    max_score_err: float = 0.0


def compare_match(s, a, gpu_idx, gpu_score, orc_idx, orc_score, rows) -> MatchReport:
    rep = MatchReport()
    margin = 2 * SCORE_TOL
    for i, r in enumerate(rows):
        rep.checked += 1
        gi, gs = gpu_idx[r], gpu_score[r]
        oi, os_ = orc_idx[i], orc_score[i]
        valid = [j for j in range(s.k) if oi[j] >= 0]
        if list(gi[len(valid):]) != [-1] * (s.k - len(valid)):
            rep.failures.append((int(r), "missing slots", list(gi), list(oi)))
            continue
        if len(set(int(x) for x in gi[:len(valid)])) != len(valid):
            rep.failures.append((int(r), "duplicate indices", list(gi)))
            continue
        for j in valid:
            y = int(gi[j])
            if y < 0:
                rep.failures.append((int(r), j, "index -1 where the oracle has a match"))
                continue
            ref = oracle_score_of(s, a, int(r), y)
            if np.isnan(ref) and np.isnan(gs[j]):
                continue
            err = abs(gs[j] - ref)
            rep.max_score_err = max(rep.max_score_err, float(err))
            if not err <= SCORE_TOL:
                rep.failures.append((int(r), j, "score", float(gs[j]), ref))
            if y == oi[j]:
                continue
            if ref >= os_[j] - margin:
                rep.near_ties += 1
            else:
                rep.failures.append((int(r), j, "index", y, int(oi[j]), ref, float(os_[j])))
    return rep


def compare_select(s, a, g: GpuResult, tau_mode=None, tau=None, k_min=None, k_max=None):
    mode = s.tau_mode if tau_mode is None else tau_mode
    mask, count = oracle.select_prefetch(
        a["maps"], s.map_dtype, g.idx, g.score.astype(np.float32).astype(np.float64), a["lb"], a["le"], mode,
        s.tau if tau is None else tau, s.k_min if k_min is None else k_min,
        s.k_max if k_max is None else k_max, s.blend)
    bad = np.argwhere((mask != g.mask) | (count != g.count))
    return bad, mask, count


# ---------------------------------------------------------------- deduplicating inserts (Section 4.4)

# RDY combines two float32 scores with weights summing to 1 and rounds once
# to float32, so its error stays within the score tolerance plus 2^-24.
RDY_TOL = SCORE_TOL + 2.0 ** -24


@dataclasses.dataclass
class DedupReport:
    replaced: int = 0
    near_ties: int = 0
    exact: bool = True
    failures: list = dataclasses.field(default_factory=list)


def compare_dedup(slots, old_maps, old_embs, cap, new_maps, new_embs, dtype, d) -> DedupReport:
    """Check GPU slots of a deduplicating insert against the oracle.

    Appended slots must be exact.  Replacements are replayed in batch order:
    each GPU victim must be a pre-batch entry not taken before, and its oracle
    RDY must be within the near-tie margin 2 * RDY_TOL of the best oracle RDY
    among the entries still available; where no near-tie exists this makes the
    victim the oracle's.  A new iteration may be dropped (-1) only when no
    entry is left."""
    rep = DedupReport()
    slots = np.asarray(slots, dtype=np.int64)
    size = old_maps.shape[0]
    m = new_maps.shape[0]
    free = max(0, cap - size)
    n_app = min(m, free)
    if not np.array_equal(slots[:n_app], size + np.arange(n_app)):
        rep.failures.append(("appended slots", slots[:n_app].tolist()))
        return rep
    rest = np.arange(n_app, m)
    ref = oracle.insert_dedup(old_maps, old_embs, cap, new_maps, new_embs, dtype, d)
    rep.exact = bool(np.array_equal(ref, slots))
    if rest.size == 0:
        return rep
    rdy = oracle.redundancy(old_maps, old_embs, new_maps[rest], None if new_embs is None else new_embs[rest],
                            dtype, d) if size > 0 else np.zeros((rest.size, 0))
    taken = np.zeros(size, dtype=bool)
    margin = 2 * RDY_TOL
    for i, x in enumerate(rest):
        y = int(slots[x])
        avail = np.flatnonzero(~taken)
        if avail.size == 0:
            if y != -1:
                rep.failures.append((int(x), "slot given with nothing left", y))
            continue
        if y < 0 or y >= size or taken[y]:
            rep.failures.append((int(x), "invalid victim", y))
            continue
        rep.replaced += 1
        row = rdy[i, avail]
        best_y, _ = oracle.rank(row, 1, avail)
        best = rdy[i, best_y[0]]
        if y != best_y[0]:
            if np.isnan(best) or not rdy[i, y] >= best - margin:
                rep.failures.append((int(x), "victim", y, float(rdy[i, y]), int(best_y[0]), float(best)))
            else:
                rep.near_ties += 1
        taken[y] = True
    return rep


def apply_slots(old, new, slots, cap):
    """The store contents after writing ``new`` rows at ``slots`` (appends extend)."""
    size = old.shape[0]
    grow = int(max([s + 1 for s in slots if s >= 0] + [size]))
    out = np.concatenate([old, np.zeros((grow - size,) + old.shape[1:], dtype=old.dtype)])
    for x, y in enumerate(slots):
        if y >= 0:
            out[y] = new[x]
    return out


# ---------------------------------------------------------------- incremental re-search (Section 4.2.2)

def compare_topk(gpu_idx, gpu_score, orc_idx, orc_score, score_of) -> MatchReport:
    """compare_match for any search: ``score_of(row, y)`` is the oracle's
    float64 score of stored index y for query row."""
    rep = MatchReport()
    margin = 2 * SCORE_TOL
    for r in range(orc_idx.shape[0]):
        rep.checked += 1
        gi, gs, oi, os_ = gpu_idx[r], gpu_score[r], orc_idx[r], orc_score[r]
        k = oi.shape[0]
        valid = [j for j in range(k) if oi[j] >= 0]
        if list(gi[len(valid):]) != [-1] * (k - len(valid)):
            rep.failures.append((r, "missing slots", list(gi), list(oi)))
            continue
        if len(set(int(x) for x in gi[:len(valid)])) != len(valid):
            rep.failures.append((r, "duplicate indices", list(gi)))
            continue
        for j in valid:
            y = int(gi[j])
            ref = score_of(r, y)
            if np.isnan(ref) and np.isnan(gs[j]):
                continue
            err = abs(gs[j] - ref)
            rep.max_score_err = max(rep.max_score_err, float(err))
            if not err <= SCORE_TOL:
                rep.failures.append((r, j, "score", float(gs[j]), ref))
            if y == oi[j]:
                continue
            if ref >= os_[j] - margin:
                rep.near_ties += 1
            else:
                rep.failures.append((r, j, "index", y, int(oi[j]), ref, float(os_[j])))
    return rep


def compare_depth(maps, dtype, Q, p, gpu_idx, gpu_score, rows=None) -> MatchReport:
    """GPU top-k of queries Q (all at prefix depth p) against the oracle."""
    rows = np.arange(Q.shape[0]) if rows is None else np.asarray(rows)
    k = gpu_idx.shape[1]
    oi, os_ = oracle.match_trajectory(maps, dtype, Q[rows], np.full(len(rows), p), k)

    def score_of(r, y):
        return oracle.cosine(oracle.widen(Q[rows[r], :p], dtype), oracle.widen(maps[y, :p], dtype))

    return compare_topk(gpu_idx[rows], gpu_score[rows], oi, os_, score_of)
