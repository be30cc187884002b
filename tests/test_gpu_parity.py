"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded inputs, at sizes the oracle finishes in seconds that still span
several workgroup tiles and a ragged tail."""
import numpy as np
import pytest
import torch

import oracle
import synth
import dataclasses

from parity import (SCORE_TOL, compare_match, compare_select, compare_topk, oracle_match, run_gpu, to_device)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X GPU")]

# (config, n, B_traj, B_sem): several tiles per store, query counts off the 16-grid
SMALL = [
    (1, 1000, 8, 0),
    (2, 3001, 64, 0),
    (2, 517, 37, 0),
    (3, 2050, 0, 40),
    (4, 4003, 100, 0),
    (5, 2501, 30, 20),
]


def _check(s, a, g, rows=None, **sel):
    rows = np.arange(s.B) if rows is None else rows
    oi, os_ = oracle_match(s, a, rows)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, rows)
    assert not rep.failures, rep.failures[:5]
    bad, _, _ = compare_select(s, a, g, **sel)
    assert bad.size == 0, bad[:10]
    return rep


@pytest.mark.parametrize("cfg,n,bt,bs", SMALL, ids=lambda v: str(v))
def test_config_small(cfg, n, bt, bs):
    print(f"config {cfg} n={n} B_traj={bt} B_sem={bs}", flush=True)
    s = synth.spec(cfg).scaled(n=n, B_traj=bt, B_sem=bs)
    a = synth.generate(s)
    g = run_gpu(s, a)
    assert g.flags == 0
    rep = _check(s, a, g)
    print(f"  near ties {rep.near_ties}, max score err {rep.max_score_err:.2e}", flush=True)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_dense_scores_all_candidates(cfg):
    """Every score the scan computes (not only the winners) is within tolerance."""
    import paper_2502_05370_amd as fm
    s = synth.spec(cfg).scaled(n=700, B_traj=min(synth.spec(cfg).B_traj, 19), B_sem=min(synth.spec(cfg).B_sem, 9))
    a = synth.generate(s)
    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16") if s.d_emb else None)
    if s.B_traj:
        got = fm.debug_scores(store, q=to_device(a["q_traj"], s.map_dtype), depth=to_device(a["depth"], "i32")).cpu().numpy()
        M = oracle.widen(a["maps"], s.map_dtype)
        Q = oracle.widen(a["q_traj"], s.map_dtype)
        for b in range(s.B_traj):
            ref = oracle.trajectory_scores(M, Q[b], int(a["depth"][b]))
            assert np.max(np.abs(got[b] - ref)) <= SCORE_TOL, b
    if s.B_sem:
        got = fm.debug_scores(store, q_sem=to_device(a["q_sem"], "bf16")).cpu().numpy()
        X = oracle.widen(a["embs"], "bf16")
        Q = oracle.widen(a["q_sem"], "bf16")
        for b in range(s.B_sem):
            ref = oracle.semantic_scores(X, Q[b])
            assert np.max(np.abs(got[b] - ref)) <= SCORE_TOL, b


def test_self_match_and_duplicates():
    """A query equal to a stored map (full depth) scores 1 and, with exact
    duplicates planted, the lowest index wins."""
    s = synth.spec(2).scaled(n=1200, B_traj=20)
    a = synth.generate(s)
    a["maps"][900] = a["maps"][300]
    a["maps"][1100] = a["maps"][300]
    a["q_traj"][3] = a["maps"][300]
    a["depth"][3] = s.L
    a["lb"][3] = s.L
    g = run_gpu(s, a)
    assert g.idx[3, 0] == 300
    assert abs(g.score[3, 0] - 1.0) <= SCORE_TOL
    _check(s, a, g)


def test_empty_store_and_k_larger_than_store():
    import paper_2502_05370_amd as fm
    s = synth.spec(4).scaled(n=3, B_traj=5)
    a = synth.generate(s)
    store = fm.Store(64, s.L, s.E)
    q = to_device(a["q_traj"], "f32")
    d = to_device(a["depth"], "i32")
    idx, sc = fm.match_trajectory(store, q, d, k=4)
    assert (idx.cpu() == -1).all() and torch.isinf(sc.cpu()).all()
    store.insert(to_device(a["maps"], "f32"))
    idx, sc = fm.match_trajectory(store, q, d, k=4)
    idx = idx.cpu().numpy()
    assert (idx[:, 3] == -1).all() and (idx[:, :3] >= 0).all()
    oi, os_ = oracle.match_trajectory(a["maps"], "f32", a["q_traj"], a["depth"], 4)
    assert np.array_equal(idx[:, :3], oi[:, :3])
    mask, cnt = fm.select_prefetch(store, torch.full((5, 4), -1, dtype=torch.int32, device="cuda"),
                                   sc, to_device(a["lb"], "i32"), to_device(a["le"], "i32"), tau=0.5, k_max=4)
    assert (mask.cpu() == 0).all() and (cnt.cpu() == 0).all()


def test_batches_beyond_one_launch_and_incremental_inserts():
    s = synth.spec(1).scaled(n=1500, B_traj=1100)
    a = synth.generate(s)
    g = run_gpu(s, a, cap=2000, insert_chunks=3)
    rows = np.r_[0:40, 1000:1100]
    _check(s, a, g, rows=rows)


def test_depth_clamping_sets_flag():
    s = synth.spec(1).scaled(n=300, B_traj=6)
    a = synth.generate(s)
    a["depth"][:] = [0, 1, 5, 31, 40, -3]
    g = run_gpu(s, a, max_depth=20)
    assert g.flags & 0x1
    a2 = dict(a)
    a2["depth"] = np.clip(a["depth"], 1, 20)
    oi, os_ = oracle_match(s, a2)
    rep = compare_match(s, a2, g.idx, g.score, oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures


def test_value_range_flag():
    """float32 values beyond 8 in magnitude (gate probabilities are at most 1)
    set FM_FLAG_VALUE_RANGE, from a stored map at insert and from a query
    row at staging; values at the limit and queries past their depth do not."""
    import paper_2502_05370_amd as fm
    s = synth.spec(2).scaled(n=200, B_traj=5)
    a = synth.generate(s)
    # at the limit, in a stored map and in an observed query layer: clean
    a["maps"][3, 2, 5] = 8.0
    a["q_traj"][0, 0, 0] = -8.0
    g = run_gpu(s, a)
    assert not (g.flags & fm._lib.FM_FLAG_VALUE_RANGE)
    # past a query's depth: never staged, clean
    a2 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in a.items()}
    d = int(np.clip(a2["depth"][1], 1, s.L))
    if d < s.L:
        a2["q_traj"][1, d, 0] = 100.0
        g = run_gpu(s, a2)
        assert not (g.flags & fm._lib.FM_FLAG_VALUE_RANGE)
    # inside a query's prefix: flagged
    a3 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in a.items()}
    a3["q_traj"][2, 0, 7] = 9.0
    g = run_gpu(s, a3)
    assert g.flags & fm._lib.FM_FLAG_VALUE_RANGE
    # in a stored map: flagged at insert
    a4 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in a.items()}
    a4["maps"][7, s.L - 1, 0] = -9.5
    g = run_gpu(s, a4)
    assert g.flags & fm._lib.FM_FLAG_VALUE_RANGE


@pytest.mark.parametrize("tau", [0.0, 0.1, 0.3, 0.5, 0.7, 0.9, 0.99, 1.0])
def test_threshold_sweep_fixed(tau):
    s = synth.spec(2).scaled(n=800, B_traj=24)
    a = synth.generate(s)
    g = run_gpu(s, a, tau=tau, k_min=0, k_max=s.E)
    bad, _, _ = compare_select(s, a, g, tau=tau, k_min=0, k_max=s.E)
    assert bad.size == 0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_dynamic_threshold(cfg):
    base = synth.spec(cfg)
    s = base.scaled(n=600, B_traj=min(base.B_traj, 24), B_sem=min(base.B_sem, 12))
    a = synth.generate(s)
    K = {1: 2, 2: 4, 3: 2, 4: 2, 5: 4}[cfg]
    g = run_gpu(s, a, tau_mode=1, k_min=K, k_max=s.E)
    bad, _, _ = compare_select(s, a, g, tau_mode=1, k_min=K, k_max=s.E)
    assert bad.size == 0


def test_layer_ranges_and_index_flag():
    import paper_2502_05370_amd as fm
    s = synth.spec(1).scaled(n=50, B_traj=4)
    a = synth.generate(s)
    store = fm.Store(50, s.L, s.E)
    store.insert(to_device(a["maps"], "f32"))
    idx = torch.tensor([[3], [7], [60], [9]], dtype=torch.int32, device="cuda")
    sc = torch.tensor([[0.9], [0.5], [0.9], [0.2]], dtype=torch.float32, device="cuda")
    lb = torch.tensor([5, 30, 0, -4], dtype=torch.int32, device="cuda")
    le = torch.tensor([2, 40, 32, 3], dtype=torch.int32, device="cuda")
    mask, cnt = fm.select_prefetch(store, idx, sc, lb, le, tau=0.6, k_min=1, k_max=8)
    assert store.check() & 0x2
    m = mask.cpu().numpy().view(np.uint64)
    c = cnt.cpu().numpy()
    ref_m, ref_c = oracle.select_prefetch(a["maps"], "f32", np.array([[3], [7], [-1], [9]]),
                                          np.array([[0.9], [0.5], [0.9], [0.2]]),
                                          np.array([5, 30, 0, -4]), np.array([2, 40, 32, 3]), 0, 0.6, 1, 8, 0)
    assert np.array_equal(m, ref_m) and np.array_equal(c, ref_c)


def test_extreme_shapes():
    """E = 64 (full mask width), E = 1 (every score 1: the lowest indices win),
    L = 1, single query, single map: indices and scores against the oracle with
    the near-tie rules, and the prefetch sets."""
    import paper_2502_05370_amd as fm
    rng = np.random.default_rng(5)
    for (n, L, E, B) in [(333, 3, 64, 17), (40, 5, 1, 3), (100, 1, 12, 1), (1, 4, 8, 2)]:
        print(f"n={n} L={L} E={E} B={B}", flush=True)
        maps = rng.dirichlet(np.ones(E), size=(n, L)).astype(np.float32)
        q = rng.dirichlet(np.ones(E), size=(B, L)).astype(np.float32)
        depth = rng.integers(1, L + 1, size=B).astype(np.int32)
        store = fm.Store(n, L, E)
        store.insert(to_device(maps, "f32"))
        idx, sc = fm.match_trajectory(store, to_device(q, "f32"), to_device(depth, "i32"), k=2)
        lb = np.zeros(B, dtype=np.int32)
        le = np.full(B, L, dtype=np.int32)
        mask, cnt = fm.select_prefetch(store, idx, sc, to_device(lb, "i32"), to_device(le, "i32"), tau=0.75,
                                       k_min=0, k_max=E)
        oi, os_ = oracle.match_trajectory(maps, "f32", q, depth, 2)
        gi = idx.cpu().numpy().astype(np.int64)
        gs = sc.cpu().numpy().astype(np.float64)

        def score_of(r, y):
            p = int(depth[r])
            return oracle.cosine(oracle.widen(q[r, :p], "f32"), oracle.widen(maps[y, :p], "f32"))

        rep = compare_topk(gi, gs, oi, os_, score_of)
        assert not rep.failures, rep.failures[:5]
        if E == 1:
            # every stored map equals every query (one value 1.0 per layer),
            # so all maps score the same: ties go to the lowest store indices,
            # which no rounding can change
            assert np.array_equal(gi, oi) and np.array_equal(gi[:, :2], np.tile([0, 1], (B, 1)))
        rm, rc = oracle.select_prefetch(maps, "f32", gi, gs, lb, le, 0, 0.75, 0, E, 0)
        assert np.array_equal(mask.cpu().numpy().view(np.uint64), rm) and np.array_equal(cnt.cpu().numpy(), rc)


def test_insert_overflow_is_rejected():
    """An insert past the capacity fails with FM_ERR_FULL, enqueues nothing and
    leaves the size and the stored maps unchanged (Section 4.4: the store
    holds at most C iterations)."""
    import paper_2502_05370_amd as fm
    s = synth.spec(2).scaled(n=150, B_traj=9)
    a = synth.generate(s)
    store = fm.Store(100, s.L, s.E)
    maps = to_device(a["maps"], "f32")
    store.insert(maps[:60])
    q, d = to_device(a["q_traj"], "f32"), to_device(a["depth"], "i32")
    i0, s0 = fm.match_trajectory(store, q, d, k=3)
    with pytest.raises(fm.FmError) as e:
        store.insert(maps[60:101])                     # 60 + 41 > 100
    assert e.value.status == fm._lib.FM_ERR_FULL
    assert store.size == 60
    i1, s1 = fm.match_trajectory(store, q, d, k=3)
    assert torch.equal(i0, i1) and torch.equal(s0, s1)
    oi, _ = oracle.match_trajectory(a["maps"][:60], "f32", a["q_traj"], a["depth"], 3)
    assert np.array_equal(i1.cpu().numpy(), oi)
    store.insert(maps[60:100])                         # exactly to capacity
    assert store.size == 100
    with pytest.raises(fm.FmError) as e:
        store.insert(maps[100:101])
    assert e.value.status == fm._lib.FM_ERR_FULL and store.size == 100


@pytest.mark.parametrize("k", [2, 4, 8])
def test_semantic_top_k(k):
    """Semantic search keeping k matches (the 4- and 8-entry lists of the scan)
    against the oracle, on a workload-3 shaped store."""
    s = dataclasses.replace(synth.spec(3).scaled(n=2050, B_sem=40), k=k)
    a = synth.generate(s)
    g = run_gpu(s, a)
    _check(s, a, g)


@pytest.mark.parametrize("cfg,n,bt,bs", [(2, 1500, 37, 0), (5, 1500, 70, 0), (4, 1200, 40, 0)])
@pytest.mark.parametrize("k", [5, 8])
def test_trajectory_top_8(cfg, n, bt, bs, k):
    """Trajectory search keeping 5 or 8 matches (the 8-entry lists) on float32
    E = 60, bfloat16 E = 60 and float32 E = 16 stores."""
    s = dataclasses.replace(synth.spec(cfg).scaled(n=n, B_traj=bt, B_sem=bs), k=k)
    a = synth.generate(s)
    g = run_gpu(s, a)
    _check(s, a, g)


def test_zero_and_nan_rows():
    import paper_2502_05370_amd as fm
    s = synth.spec(4).scaled(n=200, B_traj=6)
    a = synth.generate(s)
    a["maps"][10] = 0.0                   # zero norm: cosine 0
    a["maps"][11, 0, 0] = np.nan          # NaN: ranks last
    a["q_traj"][0] = a["maps"][11]
    a["depth"][0] = 3
    g = run_gpu(s, a)
    assert 11 not in g.idx[0]
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures
