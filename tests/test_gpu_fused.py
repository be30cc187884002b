"""GPU: the match-and-select calls (fm_match_semantic_select,
fm_match_trajectory_select) give exactly what a match call followed by
fm_select_prefetch on the same rows gives (matches, scores, sets, counts),
for every scan kernel they can follow (semantic top-1 and top-k, trajectory
bf16 top-1 and the general scan with per-group list counts), FIXED and
DYNAMIC thresholds, the similarity blend and a batch beyond one launch; the
separate calls are themselves checked against the oracle in the other
parity tests, and one case here is checked against it directly."""
import dataclasses

import numpy as np
import pytest
import torch

import synth

from parity import compare_match, compare_select, oracle_match, to_device, GpuResult

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X GPU")]


def _run_both(s, a, max_depth=None, mode=None, blend=None):
    import paper_2502_05370_amd as fm
    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16") if s.d_emb else None)
    lb, le = to_device(a["lb"], "i32"), to_device(a["le"], "i32")
    mode = s.tau_mode if mode is None else mode
    blend = s.blend if blend is None else blend
    sel = dict(tau=s.tau, k_min=s.k_min, k_max=s.k_max, mode=mode, blend=blend)
    ws = fm.Workspace(store)
    sep, fus = [], []
    if s.B_sem:
        q = to_device(a["q_sem"], "bf16")
        idx, score = fm.match_semantic(store, q, s.k, workspace=ws)
        mask, count = fm.select_prefetch(store, idx, score, lb[:s.B_sem], le[:s.B_sem], **sel)
        sep.append((idx, score, mask, count))
        fus.append(fm.match_semantic_select(store, q, lb[:s.B_sem], le[:s.B_sem], k=s.k, workspace=ws, **sel))
    if s.B_traj:
        q = to_device(a["q_traj"], s.map_dtype)
        depth = to_device(a["depth"], "i32")
        md = s.L if max_depth is None else max_depth
        idx, score = fm.match_trajectory(store, q, depth, s.k, max_depth=md, workspace=ws)
        mask, count = fm.select_prefetch(store, idx, score, lb[s.B_sem:], le[s.B_sem:], **sel)
        sep.append((idx, score, mask, count))
        fus.append(fm.match_trajectory_select(store, q, depth, lb[s.B_sem:], le[s.B_sem:], k=s.k, max_depth=md,
                                              workspace=ws, **sel))
    flags = store.check()
    torch.cuda.synchronize()
    cat = lambda parts, i: torch.cat([p[i] for p in parts]).cpu().numpy()  # noqa: E731
    return [cat(sep, i) for i in range(4)], [cat(fus, i) for i in range(4)], flags


def _assert_identical(sep, fus):
    for name, x, y in zip(("idx", "score", "mask", "count"), sep, fus):
        if name == "score":
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), name
        else:
            assert np.array_equal(x, y), name


CASES = [
    # (name, config, n, B_traj, B_sem, k)
    ("traj_f32_general_scan", 2, 3001, 64, 0, 1),
    ("traj_f32_groups_top4_blend", 4, 4003, 300, 0, 4),
    ("traj_bf16_mm_and_sem_mm", 5, 2501, 300, 200, 1),
    ("traj_bf16_small_batch", 5, 1500, 70, 20, 1),
    ("sem_top8", 3, 2050, 0, 40, 8),
    ("traj_f32_top8", 1, 1000, 37, 0, 8),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fused_equals_separate(case):
    name, cfg, n, bt, bs, k = case
    print(f"{name}: config {cfg} n={n} B_traj={bt} B_sem={bs} k={k}", flush=True)
    s = dataclasses.replace(synth.spec(cfg).scaled(n=n, B_traj=bt, B_sem=bs), k=k)
    a = synth.generate(s)
    sep, fus, flags = _run_both(s, a)
    assert flags == 0
    _assert_identical(sep, fus)


@pytest.mark.parametrize("mode,blend", [(1, 0), (1, 1), (0, 1)])
def test_fused_threshold_modes_and_blend(mode, blend):
    s = dataclasses.replace(synth.spec(4).scaled(n=2000, B_traj=150), k=4)
    print(f"config 4 mode={mode} blend={blend}", flush=True)
    a = synth.generate(s)
    sep, fus, _ = _run_both(s, a, mode=mode, blend=blend)
    _assert_identical(sep, fus)


def test_fused_batch_beyond_one_launch():
    """1030 semantic and 1100 trajectory queries: a launch of 1024 on the
    top-1 scans, then the rest (6 semantic queries on the 128-query shape, 76
    trajectory queries on the general scan); fused equals separate, and both
    halves match the oracle on every row."""
    s = synth.spec(5).scaled(n=1500, B_traj=1100, B_sem=1030)
    print(f"config 5 n={s.n} B_traj={s.B_traj} B_sem={s.B_sem}", flush=True)
    a = synth.generate(s)
    sep, fus, flags = _run_both(s, a)
    _assert_identical(sep, fus)
    assert flags == 0
    idx, score, mask, count = fus
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, idx.astype(np.int64), score.astype(np.float64), oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures[:5]
    g = GpuResult(idx.astype(np.int64), score.astype(np.float64), mask.view(np.uint64), count, flags)
    bad, _, _ = compare_select(s, a, g)
    assert bad.size == 0, bad[:10]


def test_fused_against_oracle():
    s = synth.spec(5).scaled(n=2501, B_traj=300, B_sem=200)
    print(f"config 5 n={s.n} B_traj={s.B_traj} B_sem={s.B_sem} against the oracle", flush=True)
    a = synth.generate(s)
    _, fus, flags = _run_both(s, a)
    assert flags == 0
    idx, score, mask, count = fus
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, idx.astype(np.int64), score.astype(np.float64), oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures[:5]
    g = GpuResult(idx.astype(np.int64), score.astype(np.float64), mask.view(np.uint64), count, flags)
    bad, _, _ = compare_select(s, a, g)
    assert bad.size == 0, bad[:10]
