"""GPU parity of the deduplicating insert (Section 4.4) through the C ABI.

Every case builds a store on the GPU, inserts a batch of new iterations with
fm_store_insert_dedup and compares the slots with the oracle (appends exact,
victims exact outside near-ties of RDY), then checks what the store holds
afterwards by scoring queries against it with the scan kernels and comparing
with the oracle run on the updated CPU arrays.
"""
import numpy as np
import pytest

import oracle
import synth
from parity import SCORE_TOL, apply_slots, compare_dedup, to_device

pytestmark = pytest.mark.gpu


def _store(s, a, cap, size):
    import paper_2502_05370_amd as fm
    store = fm.Store(cap, s.L, s.E, s.d_emb, s.map_dtype)
    if size:
        store.insert(to_device(a["maps"][:size], s.map_dtype),
                     to_device(a["embs"][:size], "bf16") if s.d_emb else None)
    return store


def _insert(store, s, maps, embs, d):
    slots = store.insert_dedup(to_device(maps, s.map_dtype), to_device(embs, "bf16") if s.d_emb else None, d)
    flags = store.check()
    return slots.cpu().numpy().astype(np.int64), flags


def _check_contents(s, store, maps, embs, probe_maps, probe_embs, seed=0):
    """Scores of probe queries against the GPU store match the oracle on the
    CPU copy of what the store should now hold."""
    import paper_2502_05370_amd as fm
    assert store.size == maps.shape[0]
    rng = np.random.default_rng(seed)
    depth = rng.integers(1, s.L + 1, size=probe_maps.shape[0]).astype(np.int32)
    depth[0] = s.L
    got = fm.debug_scores(store, q=to_device(probe_maps, s.map_dtype), depth=to_device(depth, "i32")).cpu().numpy()
    M = oracle.widen(maps, s.map_dtype)
    for i in range(probe_maps.shape[0]):
        ref = oracle.trajectory_scores(M, oracle.widen(probe_maps[i], s.map_dtype), int(depth[i]))
        assert np.max(np.abs(got[i] - ref)) <= SCORE_TOL, i
    if s.d_emb:
        got = fm.debug_scores(store, q_sem=to_device(probe_embs, "bf16")).cpu().numpy()
        X = oracle.widen(embs, "bf16")
        for i in range(probe_embs.shape[0]):
            ref = oracle.semantic_scores(X, oracle.widen(probe_embs[i], "bf16"))
            assert np.max(np.abs(got[i] - ref)) <= SCORE_TOL, i


CASES = [
    # (workload, stored, capacity, new, prefetch distance)
    (3, 1500, 1500, 40, 3),      # Mixtral maps + d=4096 embeddings, full store, Section 6 distance
    (5, 1200, 1300, 150, 6),     # Qwen bf16 + d=2048: 100 appended, then 50 replaced
    (2, 2000, 2000, 64, 0),      # Qwen float32, no embeddings: trajectory only
    (4, 3001, 3001, 33, 0),      # Phi-3.5 shape
    (3, 700, 700, 24, 32),       # d = L: semantic only
    (1, 517, 517, 100, 0),       # many replacements on a small store
    (3, 1203, 1203, 40, 5),      # folded semantic + trajectory rows of a length not a multiple of 4
]


@pytest.mark.parametrize("cfg,n,cap,m,d", CASES)
def test_dedup_matches_oracle(cfg, n, cap, m, d):
    print(f"dedup cfg={cfg} n={n} cap={cap} m={m} d={d}", flush=True)
    s = synth.spec(cfg).scaled(n=n, B_traj=0, B_sem=0)
    a = synth.generate(s)
    b = synth.generate_new(s, m, a)
    store = _store(s, a, cap, n)
    embs_new = b.get("new_embs")
    slots, flags = _insert(store, s, b["new_maps"], embs_new, d)
    assert flags == 0
    rep = compare_dedup(slots, a["maps"], a.get("embs"), cap, b["new_maps"], embs_new, s.map_dtype, d)
    assert not rep.failures, rep.failures[:5]
    assert rep.replaced == min(m - max(0, cap - n), n)
    print(f"  replaced={rep.replaced} near_ties={rep.near_ties} exact={rep.exact}")
    # exact copies of stored iterations replace their originals (RDY = 1)
    dup = b["dup_src"]
    first_rep = max(0, cap - n)
    seen = set()
    for x in range(first_rep, m):
        if dup[x] >= 0 and dup[x] not in seen:
            assert slots[x] == dup[x], (x, slots[x], dup[x])
        seen.add(int(slots[x]))
    maps = apply_slots(a["maps"], b["new_maps"], slots, cap)
    embs = apply_slots(a["embs"], embs_new, slots, cap) if s.d_emb else None
    _check_contents(s, store, maps, embs, b["new_maps"][:12], embs_new[:6] if s.d_emb else None)


def test_repeated_copies_exhaust_candidate_lists():
    """20 copies of one stored map: after the 8 best entries are taken, the
    later copies rescan their whole row."""
    s = synth.spec(1).scaled(n=300, B_traj=0, B_sem=0)
    a = synth.generate(s)
    new = np.repeat(a["maps"][7:8], 20, axis=0)
    store = _store(s, a, 300, 300)
    slots, _ = _insert(store, s, new, None, 0)
    rep = compare_dedup(slots, a["maps"], None, 300, new, None, s.map_dtype, 0)
    assert not rep.failures, rep.failures[:5]
    assert slots[0] == 7 and len(set(slots.tolist())) == 20
    _check_contents(s, store, apply_slots(a["maps"], new, slots, 300), None, new[:2], None)


def test_semantic_weight_with_repeated_embeddings():
    """Copies of one stored iteration with d = 3 on the d = 4096 workload
    (both score kernels and the weighted merge)."""
    s = synth.spec(3).scaled(n=400, B_traj=0, B_sem=0)
    a = synth.generate(s)
    idx = np.array([11] * 12 + [5, 11, 5])
    store = _store(s, a, 400, 400)
    slots, _ = _insert(store, s, a["maps"][idx], a["embs"][idx], 3)
    rep = compare_dedup(slots, a["maps"], a["embs"], 400, a["maps"][idx], a["embs"][idx], s.map_dtype, 3)
    assert not rep.failures, rep.failures[:5]
    assert slots[0] == 11 and slots[12] == 5


def test_empty_and_tiny_stores():
    s = synth.spec(2).scaled(n=8, B_traj=0, B_sem=0)
    a = synth.generate(s)
    b = synth.generate_new(s, 8, a, dup_frac=0.0)
    # empty store of capacity 3: three appends, the rest dropped
    store = _store(s, a, 3, 0)
    slots, _ = _insert(store, s, b["new_maps"][:5], None, 0)
    assert slots.tolist() == [0, 1, 2, -1, -1] and store.size == 3
    # full store of 5 and a batch of 8: every entry replaced once, then dropped
    store = _store(s, a, 5, 5)
    slots, _ = _insert(store, s, b["new_maps"], None, 0)
    assert sorted(slots[:5].tolist()) == [0, 1, 2, 3, 4] and slots[5:].tolist() == [-1, -1, -1]
    rep = compare_dedup(slots, a["maps"][:5], None, 5, b["new_maps"], None, s.map_dtype, 0)
    assert not rep.failures, rep.failures
    # room for the whole batch: plain appends
    store = _store(s, a, 100, 8)
    slots, _ = _insert(store, s, b["new_maps"][:5], None, 0)
    assert slots.tolist() == [8, 9, 10, 11, 12] and store.size == 13
    # a store of one
    store = _store(s, a, 1, 1)
    slots, _ = _insert(store, s, b["new_maps"][:1], None, 0)
    assert slots.tolist() == [0] and store.size == 1
    _check_contents(s, store, b["new_maps"][:1], None, b["new_maps"][:1], None)


def test_consecutive_batches():
    """A second batch sees what the first one wrote."""
    s = synth.spec(5).scaled(n=600, B_traj=0, B_sem=0)
    a = synth.generate(s)
    b = synth.generate_new(s, 96, a, dup_frac=0.2)
    store = _store(s, a, 600, 600)
    slots1, _ = _insert(store, s, b["new_maps"][:48], b["new_embs"][:48], 6)
    maps = apply_slots(a["maps"], b["new_maps"][:48], slots1, 600)
    embs = apply_slots(a["embs"], b["new_embs"][:48], slots1, 600)
    slots2, _ = _insert(store, s, b["new_maps"][48:], b["new_embs"][48:], 6)
    rep = compare_dedup(slots2, maps, embs, 600, b["new_maps"][48:], b["new_embs"][48:], s.map_dtype, 6)
    assert not rep.failures, rep.failures[:5]
    maps = apply_slots(maps, b["new_maps"][48:], slots2, 600)
    embs = apply_slots(embs, b["new_embs"][48:], slots2, 600)
    _check_contents(s, store, maps, embs, b["new_maps"][40:52], b["new_embs"][44:50])


def test_invalid_arguments_enqueue_nothing():
    import paper_2502_05370_amd as fm
    s = synth.spec(2).scaled(n=16, B_traj=0, B_sem=0)
    a = synth.generate(s)
    store = _store(s, a, 16, 16)
    maps = to_device(a["maps"][:2], s.map_dtype)
    for d in (-1, s.L + 1, 1):   # out of range, and d > 0 without embeddings
        with pytest.raises(fm.FmError):
            store.insert_dedup(maps, None, d)
    big = to_device(np.repeat(a["maps"][:1], 1025, axis=0), s.map_dtype)
    with pytest.raises(fm.FmError):
        store.insert_dedup(big, None, 0)
    assert store.size == 16
    _check_contents(s, store, a["maps"], None, a["maps"][:2], None)
