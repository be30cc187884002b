"""Parity at the full workload sizes, in the launch configuration the
benchmark times.

The whole batch runs through the C ABI on the GPU.  The oracle then checks
the queries of each kind against the whole store: all of them where the
batch is small (workloads 1 and 2), else 32 per kind (the first, the last and
30 drawn at random); the prefetch sets of every row are checked against the
oracle's selection on the GPU's own matches; and properties that hold at any
size are checked for every row.
"""
import numpy as np
import pytest

import oracle
import synth
from parity import (RDY_TOL, SCORE_TOL, compare_match, compare_select, oracle_match, run_gpu, to_device)

pytestmark = pytest.mark.gpu


PER_KIND = 32


def _sample_rows(s, seed=0):
    rng = np.random.default_rng(seed)
    rows = []
    for lo, n in ((0, s.B_sem), (s.B_sem, s.B_traj)):
        if n <= PER_KIND * 2:
            rows += list(range(lo, lo + n))
        elif n:
            mid = rng.choice(np.arange(lo + 1, lo + n - 1), size=PER_KIND - 2, replace=False)
            rows += [lo, lo + n - 1] + mid.tolist()
    return np.array(sorted(rows))


def _check_all_rows(s, g):
    idx, score = g.idx, g.score
    k = min(s.k, s.n)
    assert np.all((idx[:, :k] >= 0) & (idx[:, :k] < s.n))
    for b in range(s.B):
        assert len(set(idx[b, :k].tolist())) == k, b
    assert np.all(np.abs(score[:, :k]) <= 1.0 + SCORE_TOL)
    assert np.all(np.diff(score[:, :k], axis=1) <= 0.0)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_full_size_sampled(cfg):
    s = synth.spec(cfg)
    print(f"full-size workload {s.name}: generating", flush=True)
    a = synth.generate(s)
    max_depth = int(np.clip(a["depth"], 1, s.L).max()) if s.B_traj else None
    print("  GPU match + select", flush=True)
    g = run_gpu(s, a, max_depth=max_depth)
    assert g.flags == 0
    _check_all_rows(s, g)
    rows = _sample_rows(s)
    print(f"  oracle on rows {rows.tolist()}", flush=True)
    oi, osc = oracle_match(s, a, rows)
    rep = compare_match(s, a, g.idx, g.score, oi, osc, rows)
    assert not rep.failures, rep.failures[:5]
    print(f"  near ties {rep.near_ties}, max score error {rep.max_score_err:.2e}; selection of all rows", flush=True)
    bad, _, _ = compare_select(s, a, g)
    assert bad.size == 0, bad[:5]


def test_dedup_full_size_sampled():
    """Batch of 256 new iterations into the full 100,000-entry store with
    d = 4096 embeddings, prefetch distance 3 (the benchmarked insert)."""
    import paper_2502_05370_amd as fm
    s = synth.spec(3).scaled(B_traj=0, B_sem=0)
    m, d = 256, 3
    print("full-size dedup: generating", flush=True)
    a = synth.generate(s)
    b = synth.generate_new(s, m, a)
    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16"))
    slots = store.insert_dedup(to_device(b["new_maps"], s.map_dtype), to_device(b["new_embs"], "bf16"), d)
    assert store.check() == 0
    slots = slots.cpu().numpy().astype(np.int64)
    assert store.size == s.n
    # every new iteration replaced a distinct pre-batch entry
    assert np.all((slots >= 0) & (slots < s.n)) and len(set(slots.tolist())) == m
    # exact copies replace their originals unless an earlier one took it
    for x in np.flatnonzero(b["dup_src"] >= 0):
        if b["dup_src"][x] not in slots[:x]:
            assert slots[x] == b["dup_src"][x], x
    # sampled rows: the victim is the most redundant entry still available,
    # up to near-ties of RDY
    rng = np.random.default_rng(1)
    sample = sorted({0, 1, 2, m - 1} | set(rng.integers(3, m - 1, size=3).tolist()))
    for x in sample:
        print(f"  oracle RDY row {x}", flush=True)
        r = oracle.redundancy(a["maps"], a["embs"], b["new_maps"][x:x + 1], b["new_embs"][x:x + 1],
                              s.map_dtype, d)[0]
        avail = np.ones(s.n, dtype=bool)
        avail[slots[:x]] = False
        cand = np.flatnonzero(avail)
        best = oracle.rank(r[cand], 1, cand)[0][0]
        y = int(slots[x])
        assert avail[y]
        assert y == best or r[y] >= r[best] - 2 * RDY_TOL, (x, y, r[y], best, r[best])
