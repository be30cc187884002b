"""GPU parity of the top-1 trajectory scan of bfloat16 stores for batches of
more than 128 queries (the kernel the mixed 1M-map bf16 batch runs): the HIP
path through the C ABI against the CPU oracle on the same seeded inputs.

The cases cover the layer geometries of bf16 stores (8, 16, 20, 32, 60 and 64
experts: several layers per k-step, one layer in one or two k-steps, padding
quads), odd and even stage counts per slice, one to four query groups, a store
long enough for several slices per workgroup, ragged tails, a batch beyond one
launch, uniform and geometric depth mixes, and dense scores."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth

from parity import SCORE_TOL, compare_match, oracle_match, run_gpu, to_device

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X GPU")]


def _bf16_spec(cfg, E, L, n, B_traj, depth_max, law="uniform"):
    base = synth.spec(cfg)
    return dataclasses.replace(base, E=E, L=L, n=n, B_traj=B_traj, B_sem=0, d_emb=0, map_dtype=synth.BF16,
                               depth_law=law, depth_max=depth_max, k=1, blend=0)


# (name, base config, E, L, n, B_traj, depth_max, depth law, max_depth passed to the search)
CASES = [
    ("qwen_e60_two_groups", 5, 60, 24, 5003, 300, 23, "uniform", 24),
    ("qwen_e60_one_group_full_depth", 5, 60, 24, 2049, 129, 24, "uniform", 24),
    ("e64_three_groups", 5, 64, 24, 3001, 513, 24, "uniform", 24),
    ("e8_odd_stages", 1, 8, 32, 6007, 200, 10, "uniform", 10),
    ("e16_geometric", 4, 16, 32, 3001, 257, 31, "geometric", 32),
    ("e20_padding_quads_odd", 2, 20, 24, 1777, 160, 13, "uniform", 13),
    ("e32_four_groups", 1, 32, 32, 2500, 1024, 31, "uniform", 31),
    ("e60_depth_one", 5, 60, 24, 999, 140, 1, "uniform", 1),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_traj_mm_matches_oracle(case):
    name, cfg, E, L, n, bt, dmax, law, max_depth = case
    print(f"{name}: E={E} L={L} n={n} B_traj={bt} depth<={dmax} max_depth={max_depth}", flush=True)
    s = _bf16_spec(cfg, E, L, n, bt, dmax, law)
    a = synth.generate(s)
    g = run_gpu(s, a, max_depth=max_depth)
    assert g.flags == 0
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures[:5]
    print(f"  near ties {rep.near_ties}, max score err {rep.max_score_err:.2e}", flush=True)


def test_traj_mm_several_slices_per_workgroup():
    """A store long enough that every workgroup walks several slices."""
    s = _bf16_spec(5, 60, 24, 70001, 300, 23)
    print(f"E=60 n={s.n} B_traj={s.B_traj}", flush=True)
    a = synth.generate(s)
    g = run_gpu(s, a, max_depth=23)
    rows = np.arange(s.B)
    oi, os_ = oracle_match(s, a, rows)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, rows)
    assert not rep.failures, rep.failures[:5]
    print(f"  near ties {rep.near_ties}, max score err {rep.max_score_err:.2e}", flush=True)


def test_traj_mm_batch_beyond_one_launch():
    """1100 queries: one launch of 1024 on the bf16 top-1 scan, then 76 on the general scan."""
    s = _bf16_spec(5, 60, 24, 1500, 1100, 23)
    print(f"E=60 n={s.n} B_traj={s.B_traj}", flush=True)
    a = synth.generate(s)
    g = run_gpu(s, a, max_depth=24)
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures[:5]


@pytest.mark.parametrize("E,dmax", [(60, 23), (8, 9)])
def test_traj_mm_dense_scores(E, dmax):
    """Every score of a 150-query bf16 batch (not only the winners) is within tolerance."""
    import paper_2502_05370_amd as fm
    s = _bf16_spec(5 if E == 60 else 1, E, 24 if E == 60 else 32, 700, 150, dmax)
    print(f"dense E={E} n={s.n} B_traj={s.B_traj} depth<={dmax}", flush=True)
    a = synth.generate(s)
    store = fm.Store(s.n, s.L, s.E, 0, s.map_dtype)
    store.insert(to_device(a["maps"], s.map_dtype), None)
    got = fm.debug_scores(store, q=to_device(a["q_traj"], s.map_dtype), depth=to_device(a["depth"], "i32"),
                          max_depth=dmax).cpu().numpy()
    M = oracle.widen(a["maps"], s.map_dtype)
    Q = oracle.widen(a["q_traj"], s.map_dtype)
    for b in range(s.B_traj):
        ref = oracle.trajectory_scores(M, Q[b], int(a["depth"][b]))
        assert np.max(np.abs(got[b] - ref)) <= SCORE_TOL, b


def test_traj_mm_zero_and_nan_rows():
    """Zero maps score 0, a map with a NaN in every query's prefix ranks last."""
    s = _bf16_spec(5, 60, 24, 600, 200, 23)
    a = synth.generate(s)
    a["maps"][10] = 0
    a["maps"][11, 0, 0] = synth.bf16_bits(np.array([np.nan], dtype=np.float32))[0]
    a["q_traj"][0] = a["maps"][11]
    a["depth"][0] = 3
    a["q_traj"][1] = 0                     # zero query: every cosine is 0, the first map wins
    g = run_gpu(s, a, max_depth=24)
    assert g.idx[0, 0] != 11
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures[:5]


def test_traj_mm_signed_and_scaled_queries():
    """Queries of either sign and of norms far from 1 (bf16 values scaled by
    powers of two, exactly): a query whose cosines are all negative keeps its
    least negative map, and the ranking does not depend on the query's norm."""
    s = _bf16_spec(5, 60, 24, 3001, 300, 23)
    a = synth.generate(s)
    q = a["q_traj"].view(np.uint16).astype(np.uint32) << 16
    qf = q.view(np.float32).reshape(a["q_traj"].shape).copy()
    qf[0::3] *= -1.0          # every cosine of these queries is <= 0
    qf[1::3] *= 64.0          # |q| >> 1
    qf[2::6] *= 1.0 / 64.0    # |q| << 1
    a["q_traj"] = synth.bf16_bits(qf.reshape(-1)).reshape(a["q_traj"].shape)
    print(f"signed/scaled E=60 n={s.n} B_traj={s.B_traj}", flush=True)
    g = run_gpu(s, a, max_depth=24)
    assert g.flags == 0
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures[:5]
    assert np.all(g.score[0::3, 0] <= 0.0)
