"""GPU parity of the incremental trajectory re-search (Section 4.2.2)
through the C ABI: after every observed layer the step's top-k must match the
oracle's Eq. 5 search at that prefix depth (scores within 1e-5, indices exact
outside near-ties), for every layer of a pass."""
import numpy as np
import pytest

import oracle
import synth
from parity import SCORE_TOL, compare_depth, to_device

pytestmark = pytest.mark.gpu


def _pass(cfg, n, B, k, layers=None, cap=None, insert=True):
    import paper_2502_05370_amd as fm
    s = synth.spec(cfg).scaled(n=n, B_traj=B, B_sem=0)
    a = synth.generate(s)
    store = fm.Store(cap or n, s.L, s.E, s.d_emb, s.map_dtype)
    if insert:
        store.insert(to_device(a["maps"], s.map_dtype),
                     to_device(a["embs"], "bf16") if s.d_emb else None)
    tp = fm.TrajPass(store, B)
    q = to_device(a["q_traj"], s.map_dtype)
    out = []
    for layer in range(s.L if layers is None else layers):
        idx, score = tp.step(q[:, layer], layer, k)
        out.append((idx.cpu().numpy().astype(np.int64), score.cpu().numpy().astype(np.float64)))
    flags = store.check()
    return s, a, store, out, flags


CASES = [
    # (workload, stored maps, batch, k)
    (1, 1000, 8, 1),       # Mixtral 32 x 8 float32
    (2, 3001, 64, 1),      # Qwen 24 x 60 float32, one full chunk of queries
    (2, 517, 100, 2),      # two chunks (64 + 36), ragged store
    (4, 2050, 40, 4),      # Phi 32 x 16, top-4
    (5, 1500, 20, 8),      # bf16 store, top-8
]


@pytest.mark.parametrize("cfg,n,B,k", CASES)
def test_every_layer_matches_oracle(cfg, n, B, k):
    print(f"step pass cfg={cfg} n={n} B={B} k={k}", flush=True)
    s, a, store, out, flags = _pass(cfg, n, B, k)
    assert flags == 0
    near = 0
    for layer, (idx, score) in enumerate(out):
        rep = compare_depth(a["maps"], s.map_dtype, a["q_traj"], layer + 1, idx, score)
        assert not rep.failures, (layer, rep.failures[:3])
        near += rep.near_ties
    print(f"  layers={len(out)} near_ties={near}")


def test_step_agrees_with_match_call():
    """The step at depth p and fm_match_trajectory at depth p score every
    stored map alike (dense scores of the match kernels vs the step's top-8)."""
    import paper_2502_05370_amd as fm
    import torch
    s, a, store, out, _ = _pass(2, 800, 16, 8)
    for layer in (0, 5, s.L - 1):
        depth = torch.full((16,), layer + 1, dtype=torch.int32, device="cuda")
        dense = fm.debug_scores(store, q=to_device(a["q_traj"], s.map_dtype), depth=depth).cpu().numpy()
        idx, score = out[layer]
        for b in range(16):
            assert np.max(np.abs(dense[b, idx[b]] - score[b])) <= 2 * SCORE_TOL


def test_stale_state_is_flagged():
    import paper_2502_05370_amd as fm
    s = synth.spec(2).scaled(n=300, B_traj=4, B_sem=0)
    a = synth.generate(s)
    store = fm.Store(400, s.L, s.E, 0, s.map_dtype)
    store.insert(to_device(a["maps"][:200], s.map_dtype))
    tp = fm.TrajPass(store, 4)
    q = to_device(a["q_traj"], s.map_dtype)
    tp.step(q[:, 0], 0)
    tp.step(q[:, 1], 1)
    assert store.check() == 0
    # a layer skipped
    tp.step(q[:, 3], 3)
    assert store.check() == fm.FM_FLAG_STATE_STALE
    # the store grew since layer 0
    tp.step(q[:, 0], 0)
    store.insert(to_device(a["maps"][200:], s.map_dtype))
    tp.step(q[:, 1], 1)
    assert store.check() == fm.FM_FLAG_STATE_STALE
    # a new pass on the grown store is clean and correct
    for layer in range(3):
        idx, score = tp.step(q[:, layer], layer, 2)
    assert store.check() == 0
    rep = compare_depth(a["maps"], s.map_dtype, a["q_traj"], 3, idx.cpu().numpy().astype(np.int64),
                        score.cpu().numpy().astype(np.float64))
    assert not rep.failures, rep.failures


def test_empty_store_and_small_shapes():
    import paper_2502_05370_amd as fm
    # empty store: no matches
    s, a, store, out, _ = _pass(1, 10, 3, 2, layers=2, insert=False)
    for idx, score in out:
        assert np.all(idx == -1) and np.all(np.isneginf(score))
    # one stored map, one query; k larger than the store
    s, a, store, out, _ = _pass(1, 1, 1, 4, layers=4)
    for layer, (idx, score) in enumerate(out):
        assert idx[0, 0] == 0 and np.all(idx[0, 1:] == -1)
        rep = compare_depth(a["maps"], s.map_dtype, a["q_traj"], layer + 1, idx, score)
        assert not rep.failures


@pytest.mark.parametrize("L,E", [(1, 64), (3, 1), (5, 37), (64, 4)])
def test_extreme_shapes(L, E):
    import paper_2502_05370_amd as fm
    rng = np.random.default_rng(L * 100 + E)
    n, B = 133, 19
    z = rng.standard_normal((n + B, L, E))
    p = np.exp(z) / np.exp(z).sum(-1, keepdims=True)
    maps, Q = p[:n].astype(np.float32), p[n:].astype(np.float32)
    store = fm.Store(n, L, E, 0, "f32")
    store.insert(to_device(maps, "f32"))
    tp = fm.TrajPass(store, B)
    q = to_device(Q, "f32")
    for layer in range(L):
        idx, score = tp.step(q[:, layer], layer, 3)
        rep = compare_depth(maps, "f32", Q, layer + 1, idx.cpu().numpy().astype(np.int64),
                            score.cpu().numpy().astype(np.float64))
        assert not rep.failures, (layer, rep.failures[:3])
    assert store.check() == 0


def test_full_size_pass_sampled():
    """Workload 2 at full size (50,000 maps, 64 queries): a whole pass of 24
    steps; sampled queries against the oracle at a few depths, properties of
    every row at every depth."""
    s, a, store, out, flags = _pass(2, 50_000, 64, 1)
    assert flags == 0
    for idx, score in out:
        assert np.all((idx[:, 0] >= 0) & (idx[:, 0] < s.n)) and np.all(np.abs(score) <= 1 + SCORE_TOL)
    rows = [0, 17, 40, 63]
    for layer in (0, 7, s.L - 1):
        print(f"  oracle depth {layer + 1}", flush=True)
        idx, score = out[layer]
        rep = compare_depth(a["maps"], s.map_dtype, a["q_traj"], layer + 1, idx, score, rows=rows)
        assert not rep.failures, (layer, rep.failures[:3])
    # the deepest step recovers the map each query was drawn from
    assert np.mean(out[-1][0][:, 0] == a["src"]) > 0.9
