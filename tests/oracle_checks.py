"""Checks that pin the CPU oracle to facts fixed outside of it.

Each check reaches the oracle through ``oracle.finemoe`` attribute lookups at
call time, so the mutant tests can swap a function for a deliberately wrong
one (on the CPU) and confirm that at least one check fails.
"""
import json
import math
import os

import numpy as np

import oracle.brute as brute
import oracle.finemoe as F

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rand_maps(rng, n, L, E, zero_frac=0.0):
    z = rng.standard_normal((n, L, E))
    p = np.exp(z)
    if zero_frac:
        p[rng.random(p.shape) < zero_frac] = 0.0
        p[..., 0] += 1e-3
    p /= p.sum(-1, keepdims=True)
    return p.astype(np.float32)


# ------------------------------------------------------------------ cosine / trajectory / semantic

def check_cosine_vs_fsum(seed=0):
    rng = np.random.default_rng(seed)
    for _ in range(50):
        d = int(rng.integers(1, 40))
        u = rng.standard_normal(d)
        v = rng.standard_normal(d)
        if rng.random() < 0.3:
            v = np.abs(v)
        ref = brute.cosine_fsum(list(u), list(v))
        got = F.cosine(u, v)
        assert abs(got - ref) <= 1e-14, (got, ref)
        got_many = F._cosine_many(v[None, :], u)[0]
        assert abs(got_many - ref) <= 1e-14, (got_many, ref)
    assert F.cosine(np.zeros(5), np.ones(5)) == 0.0
    assert F.cosine(np.ones(5), np.zeros(5)) == 0.0


def check_cosine_vs_torch(seed=1):
    import torch
    rng = np.random.default_rng(seed)
    V = rng.standard_normal((64, 33))
    u = rng.standard_normal(33)
    ref = torch.nn.functional.cosine_similarity(
        torch.from_numpy(V), torch.from_numpy(u)[None, :].expand(64, 33), dim=1, eps=0.0).numpy()
    got = F._cosine_many(V, u)
    assert np.max(np.abs(got - ref)) <= 1e-14


def check_self_match(seed=2):
    rng = np.random.default_rng(seed)
    maps = _rand_maps(rng, 40, 6, 5)
    m64 = F.widen(maps, "f32")
    for y in (0, 17, 39):
        for p in (1, 3, 6):
            s = F.trajectory_scores(m64, m64[y], p)
            assert abs(s[y] - 1.0) <= 1e-15, s[y]
            assert np.all(s <= 1.0 + 1e-15)
            i, sc = F.match_trajectory(maps, "f32", maps[y:y + 1], np.array([p]), 1)
            assert i[0, 0] == y and abs(sc[0, 0] - 1.0) <= 1e-15


def check_disjoint_support():
    L, E = 3, 6
    store = np.zeros((2, L, E), dtype=np.float32)
    store[0, :, 3:] = 1.0 / 3
    store[1, :, :3] = 1.0 / 3
    q = np.zeros((L, E), dtype=np.float32)
    q[:, :3] = [0.5, 0.25, 0.25]
    s = F.trajectory_scores(F.widen(store, "f32"), F.widen(q, "f32"), L)
    assert s[0] == 0.0
    assert s[1] > 0.9


def check_depth_special_cases(seed=3):
    rng = np.random.default_rng(seed)
    n, L, E = 30, 5, 4
    maps = F.widen(_rand_maps(rng, n, L, E), "f32")
    q = F.widen(_rand_maps(rng, 1, L, E)[0], "f32")
    full = F.trajectory_scores(maps, q, L)
    one = F.trajectory_scores(maps, q, 1)
    for y in range(n):
        ref_full = brute.cosine_fsum(list(q.ravel()), list(maps[y].ravel()))
        ref_one = brute.cosine_fsum(list(q[0]), list(maps[y, 0]))
        assert abs(full[y] - ref_full) <= 1e-14
        assert abs(one[y] - ref_one) <= 1e-14
    for p in range(1, L + 1):
        s = F.trajectory_scores(maps, q, p)
        for y in range(0, n, 7):
            ref = brute.cosine_fsum(list(q[:p].ravel()), list(maps[y, :p].ravel()))
            assert abs(s[y] - ref) <= 1e-14


def check_unobserved_layers_ignored(seed=4):
    rng = np.random.default_rng(seed)
    n, L, E = 25, 6, 4
    maps = _rand_maps(rng, n, L, E)
    Q = _rand_maps(rng, 3, L, E)
    depth = np.array([1, 3, 5])
    i0, s0 = F.match_trajectory(maps, "f32", Q, depth, 3)
    Q2 = Q.copy()
    for b, p in enumerate(depth):
        Q2[b, p:] = np.nan
    i1, s1 = F.match_trajectory(maps, "f32", Q2, depth, 3)
    assert np.array_equal(i0, i1) and np.array_equal(s0, s1)


def check_semantic_vs_fsum(seed=5):
    rng = np.random.default_rng(seed)
    import synth
    X = synth.bf16_bits(rng.standard_normal((20, 16)).astype(np.float32))
    Qs = synth.bf16_bits(rng.standard_normal((3, 16)).astype(np.float32))
    idx, sc = F.match_semantic(X, Qs, 2)
    X64 = F.widen(X, "bf16")
    Q64 = F.widen(Qs, "bf16")
    for b in range(3):
        ref = [brute.cosine_fsum(list(Q64[b]), list(X64[y])) for y in range(20)]
        best = brute.best_matches(ref, 2)
        assert list(idx[b]) == best
        for j in range(2):
            assert abs(sc[b, j] - ref[best[j]]) <= 1e-14


def check_match_vs_bruteforce(seed=6):
    rng = np.random.default_rng(seed)
    n, L, E = 60, 4, 4
    maps = _rand_maps(rng, n, L, E)
    maps[40] = maps[12]           # exact duplicate: the lower index must win
    maps[41] = maps[12]
    Q = _rand_maps(rng, 4, L, E)
    Q[0] = maps[12]
    depth = np.array([4, 1, 2, 3])
    idx, sc = F.match_trajectory(maps, "f32", Q, depth, 4)
    m64 = F.widen(maps, "f32")
    q64 = F.widen(Q, "f32")
    for b in range(4):
        p = depth[b]
        ref = [brute.cosine_fsum(list(q64[b, :p].ravel()), list(m64[y, :p].ravel())) for y in range(n)]
        best = brute.best_matches(ref, 4)
        assert list(idx[b]) == best, (b, list(idx[b]), best)
        for j in range(4):
            assert abs(sc[b, j] - ref[best[j]]) <= 1e-14
    assert list(idx[0, :3]) == [12, 40, 41]


def check_rank_rules():
    s = np.array([0.5, 0.9, np.nan, 0.9, 0.1, 0.9])
    i, v = F.rank(s, 6)
    assert list(i) == [1, 3, 5, 0, 4, 2]
    i, v = F.rank(s, 8)
    assert list(i[6:]) == [-1, -1] and np.all(np.isneginf(v[6:]))
    i, v = F.rank(np.zeros(0), 2)
    assert list(i) == [-1, -1]
    rng = np.random.default_rng(7)
    for _ in range(20):
        n = int(rng.integers(1, 256))
        s = np.round(rng.random(n), 2)          # many exact ties
        k = int(rng.integers(1, 9))
        i, v = F.rank(s, k)
        assert list(i) == brute.best_matches(list(s), k)


# ------------------------------------------------------------------ selection

def check_uniform_golden():
    g = golden("uniform4.json")
    p = np.array(g["p"])
    for case in g["cases"]:
        m, c, _ = F.select_row(p, case["tau"], 0, 4)
        assert c == case["kstar"], (case, c)
        assert m == (1 << c) - 1, (case, m)


def check_delta_golden():
    g = golden("delta.json")
    for case in g["cases"]:
        t = F.threshold(F.TAU_DYNAMIC, 0.0, case["score"])
        assert abs(t - case["delta"]) <= 1e-15, (case, t)
    assert F.threshold(F.TAU_FIXED, 0.8, 0.3) == float(np.float32(0.8))


def check_select_vs_enumeration(seed=8):
    rng = np.random.default_rng(seed)
    for _ in range(300):
        E = int(rng.integers(1, 11))
        p = rng.dirichlet(np.full(E, float(rng.choice([0.3, 1.0, 5.0]))))
        if rng.random() < 0.3:
            p = np.round(p * 8) / 8           # ties and exact dyadic sums
        tau = float(rng.choice([0.0, 0.1, 0.5, 0.8, 0.9, 0.99, 1.0, rng.random()]))
        k_min = int(rng.integers(0, E + 1))
        k_max = int(rng.integers(k_min, E + 1))
        m, c, order = F.select_row(p, tau, k_min, k_max)
        kk, S = brute.prefetch_set(list(p), tau, k_min, k_max)
        assert c == kk, (p, tau, k_min, k_max, c, kk)
        assert m == sum(1 << j for j in S), (p, tau, m, S)
        m0, c0, _ = F.select_row(p, tau, 0, E)
        assert c0 == brute.min_cardinality(list(p), tau)
        chosen = [j for j in range(E) if (m0 >> j) & 1]
        assert math.fsum(p[j] for j in chosen) == brute.max_sum_of_size(list(p), c0)


def check_select_nesting_and_minimality(seed=9):
    rng = np.random.default_rng(seed)
    for _ in range(200):
        E = int(rng.integers(2, 64))
        p = rng.dirichlet(np.full(E, 0.5))
        taus = np.sort(rng.random(4))
        prev = 0
        for t in taus:
            m, c, order = F.select_row(p, float(t), 0, E)
            assert (prev & ~m) == 0, "sets must grow with tau"
            prev = m
            chosen = [int(order[i]) for i in range(c)]
            total = math.fsum(p[j] for j in chosen)
            if c < E:
                assert total >= t - 1e-12
            if c > 0:
                assert math.fsum(p[j] for j in chosen[:-1]) < t + 1e-12
        m, c, _ = F.select_row(p, 1.5, 0, E)
        assert c == E and m == (1 << E) - 1
        m, c, _ = F.select_row(p, 0.999, 2, 3)
        assert 2 <= c <= 3


def check_blend():
    a = np.array([0.5, 0.25, 0.25])
    b = np.array([0.0, 0.5, 0.5])
    got = F.blend_rows(np.stack([a, b]), [0.5, 0.25])
    ref = (2 * a + b) / 3
    assert np.max(np.abs(got - ref)) <= 1e-16
    assert np.array_equal(F.blend_rows(a[None, :], [0.7]), a)
    assert np.max(np.abs(F.blend_rows(np.stack([a, a, a]), [0.9, 0.3, 0.1]) - a)) <= 1e-16
    got = F.blend_rows(np.stack([a, b]), [-0.5, 0.0])     # all weights clipped to 0: plain mean
    assert np.max(np.abs(got - (a + b) / 2)) <= 1e-16
    got = F.blend_rows(np.stack([a, b]), [0.9, -0.2])     # negative weight is dropped
    assert np.array_equal(got, a)
    rng = np.random.default_rng(10)
    rows = rng.dirichlet(np.ones(16), size=4)
    got = F.blend_rows(rows, rng.random(4))
    assert abs(got.sum() - 1.0) <= 1e-14 and np.all(got >= 0)


def check_select_prefetch_layout(seed=11):
    rng = np.random.default_rng(seed)
    n, L, E = 10, 5, 6
    maps = _rand_maps(rng, n, L, E)
    idx = np.array([[3], [-1], [7]])
    score = np.array([[0.9], [-np.inf], [0.2]])
    lb = np.array([1, 0, 4])
    le = np.array([4, 5, 9])
    mask, cnt = F.select_prefetch(maps, "f32", idx, score, lb, le, F.TAU_FIXED, 0.5, 1, 6, F.BLEND_NONE)
    assert np.all(mask[0, [0, 4]] == 0) and np.all(cnt[0, 1:4] > 0)
    assert np.all(mask[1] == 0) and np.all(cnt[1] == 0)
    assert np.all(mask[2, :4] == 0) and cnt[2, 4] > 0
    for l in range(1, 4):
        m, c, _ = F.select_row(F.widen(maps[3, l], "f32"), float(np.float32(0.5)), 1, 6)
        assert mask[0, l] == m and cnt[0, l] == c
    # dynamic threshold: score 0.9 -> delta 0.1 -> small sets, score 0.2 -> delta 0.8
    mask, cnt = F.select_prefetch(maps, "f32", idx, score, lb, le, F.TAU_DYNAMIC, 0.0, 0, 6, F.BLEND_NONE)
    m, c, _ = F.select_row(F.widen(maps[7, 4], "f32"), 1.0 - 0.2, 0, 6)
    assert mask[2, 4] == m and cnt[2, 4] == c


# ------------------------------------------------------------------ per-layer re-search (Section 4.2.2)

def check_research_schedule_depths():
    """Target layer l uses layers 1 .. l-d: map 2 agrees with the query on
    layer 1 only, map 1 on layers 1-2, map 0 on layers 1-3; each wins from
    the layer whose prefix first tells it apart."""
    L, E, d = 5, 4, 2
    q = np.zeros((1, L, E), np.float32)
    for l in range(L):
        q[0, l, l % E] = 1.0
    maps = np.zeros((3, L, E), np.float32)
    for y, agree in enumerate((3, 2, 1)):
        for l in range(L):
            maps[y, l, l % E if l < agree else (l + 1) % E] = 1.0
    res = F.research_schedule(maps, "f32", q, 3, d)
    assert sorted(res) == list(range(d + 1, L + 1))
    # p = 1: all three agree (score 1), lowest index first
    assert list(res[d + 1][0][0]) == [0, 1, 2] and np.allclose(res[d + 1][1][0], 1.0)
    # p = 2: maps 0 and 1 agree on both layers, map 2 on one of two
    assert list(res[d + 2][0][0]) == [0, 1, 2]
    assert abs(res[d + 2][1][0][2] - 0.5) <= 1e-15
    # p = 3: only map 0 agrees on all three layers
    assert res[d + 3][0][0][0] == 0 and abs(res[d + 3][1][0][1] - 2.0 / 3.0) <= 1e-15
    assert abs(res[d + 3][1][0][2] - 1.0 / 3.0) <= 1e-15


def check_research_schedule_vs_fsum(seed=17):
    rng = np.random.default_rng(seed)
    L, E, d = 6, 5, 1
    maps = _rand_maps(rng, 9, L, E, zero_frac=0.2)
    Q = _rand_maps(rng, 3, L, E)
    res = F.research_schedule(maps, "f32", Q, 2, d)
    assert len(res) == L - d
    for l, (idx, sc) in res.items():
        p = l - d
        for b in range(3):
            ref = [brute.cosine_fsum(F.widen(Q[b, :p], "f32").ravel(), F.widen(maps[y, :p], "f32").ravel())
                   for y in range(9)]
            assert list(idx[b]) == brute.best_matches(ref, 2), (l, b)
            assert all(abs(sc[b][j] - ref[idx[b][j]]) <= 1e-14 for j in range(2))


# ------------------------------------------------------------------ store deduplication (Section 4.4)

def _bf16(x):
    """bf16 bit patterns of float values (round to nearest even)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def _store(rng, n, L, E, d_emb, dtype="f32"):
    maps = _rand_maps(rng, n, L, E, zero_frac=0.2)
    if dtype == "bf16":
        maps = _bf16(maps)
    embs = _bf16(rng.standard_normal((n, d_emb)))
    return maps, embs


def check_redundancy_vs_fsum(seed=12):
    rng = np.random.default_rng(seed)
    for dtype in ("f32", "bf16"):
        L, E, d_emb = 4, 5, 8
        old_maps, old_embs = _store(rng, 7, L, E, d_emb, dtype)
        new_maps, new_embs = _store(rng, 3, L, E, d_emb, dtype)
        for d in range(L + 1):
            got = F.redundancy(old_maps, old_embs, new_maps, new_embs, dtype, d)
            assert got.shape == (3, 7)
            for x in range(3):
                for y in range(7):
                    ref = brute.redundancy_fsum(F.widen(old_maps[y], dtype).tolist(), F.widen(old_embs[y], "bf16"),
                                                F.widen(new_maps[x], dtype).tolist(), F.widen(new_embs[x], "bf16"), d)
                    assert abs(got[x, y] - ref) <= 1e-14, (dtype, d, x, y, got[x, y], ref)


def check_redundancy_closed_forms(seed=13):
    rng = np.random.default_rng(seed)
    L, E, d_emb = 6, 4, 16
    maps, embs = _store(rng, 5, L, E, d_emb)
    for d in range(L + 1):
        # an iteration is fully redundant with itself
        r = F.redundancy(maps, embs, maps[2:3], embs[2:3], "f32", d)
        assert abs(r[0, 2] - 1.0) <= 1e-15, (d, r[0, 2])
    # disjoint expert supports and orthogonal embeddings: nothing in common
    a = np.zeros((1, L, E), np.float32)
    b = np.zeros((1, L, E), np.float32)
    a[0, :, :2] = 0.5
    b[0, :, 2:] = 0.5
    ea = _bf16(np.eye(d_emb)[:1])
    eb = _bf16(np.eye(d_emb)[1:2])
    for d in range(L + 1):
        assert F.redundancy(a, ea, b, eb, "f32", d)[0, 0] == 0.0
    # the two halves weigh d/L and (L-d)/L: same map, orthogonal embeddings
    for d in range(L + 1):
        r = F.redundancy(a, ea, a, eb, "f32", d)[0, 0]
        assert abs(r - (L - d) / L) <= 1e-15, (d, r)
        r = F.redundancy(a, ea, b, ea, "f32", d)[0, 0]
        assert abs(r - d / L) <= 1e-15, (d, r)
    # a map that differs only in its last layer still counts that layer
    c = a.copy()
    c[0, L - 1] = b[0, L - 1]
    r = F.redundancy(a, ea, c, ea, "f32", 0)[0, 0]
    assert abs(r - (L - 1) / L) <= 1e-15, r


def check_dedup_vs_enumeration(seed=14):
    rng = np.random.default_rng(seed)
    for _ in range(300):
        size = int(rng.integers(0, 6))
        cap = size + int(rng.integers(0, 3))
        m = int(rng.integers(0, 5))
        rdy = np.round(rng.uniform(-1, 1, (m, size)), 1)   # coarse values give ties
        got = F.dedup_slots(rdy, size, cap)
        ref = brute.dedup_by_enumeration(rdy.tolist(), size, cap)
        assert list(got) == ref, (size, cap, rdy, list(got), ref)


def check_dedup_duplicates(seed=15):
    rng = np.random.default_rng(seed)
    L, E, d_emb = 4, 6, 8
    maps, embs = _store(rng, 12, L, E, d_emb)
    pick = [5, 2, 5]
    new_maps = np.concatenate([maps[pick], _store(rng, 1, L, E, d_emb)[0]])
    new_embs = np.concatenate([embs[pick], _store(rng, 1, L, E, d_emb)[1]])
    for d in (0, 1, L):
        slots = F.insert_dedup(maps, embs, 12, new_maps, new_embs, "f32", d)
        # exact copies replace their originals; the second copy of 5 takes its
        # next most redundant entry, and every victim is distinct
        assert slots[0] == 5 and slots[1] == 2, slots
        rdy = [[brute.redundancy_fsum(F.widen(maps[y], "f32").tolist(), F.widen(embs[y], "bf16"),
                                      F.widen(new_maps[x], "f32").tolist(), F.widen(new_embs[x], "bf16"), d)
                for y in range(12)] for x in range(4)]
        rest = [y for y in range(12) if y not in (5, 2)]
        assert slots[2] == max(rest, key=lambda y: (rdy[2][y], -y)), slots
        rest = [y for y in rest if y != slots[2]]
        assert slots[3] == max(rest, key=lambda y: (rdy[3][y], -y)), slots
        assert len(set(slots.tolist())) == 4


def check_dedup_appends_first():
    rng = np.random.default_rng(16)
    L, E, d_emb = 3, 4, 8
    maps, embs = _store(rng, 3, L, E, d_emb)
    new_maps, new_embs = _store(rng, 4, L, E, d_emb)
    # room for two: appended at 3 and 4, the other two replace stored entries
    slots = F.insert_dedup(maps, embs, 5, new_maps, new_embs, "f32", 1)
    assert list(slots[:2]) == [3, 4] and all(0 <= y < 3 for y in slots[2:]) and slots[2] != slots[3], slots
    # room for all: nothing is replaced
    assert list(F.insert_dedup(maps, embs, 10, new_maps, new_embs, "f32", 1)) == [3, 4, 5, 6]
    # empty store smaller than the batch: the overflow is dropped
    empty_m, empty_e = maps[:0], embs[:0]
    assert list(F.insert_dedup(empty_m, empty_e, 2, new_maps[:3], new_embs[:3], "f32", 1)) == [0, 1, -1]
    # full store smaller than the batch: every entry is replaced once, then drop
    slots = F.insert_dedup(maps, embs, 3, new_maps, new_embs, "f32", 1)
    assert sorted(slots[:3].tolist()) == [0, 1, 2] and slots[3] == -1, slots
    # no embeddings needed when d = 0
    slots = F.insert_dedup(maps, None, 3, new_maps[:1], None, "f32", 0)
    assert 0 <= slots[0] < 3


# ------------------------------------------------------------------ priorities (Section 4.5)

def _f32(x):
    return float(np.float32(x))


def check_priority_closed_forms():
    L, E = 4, 3
    maps = np.zeros((1, L, E), np.float32)
    maps[0, 1] = [0.5, 0.3, 0.2]
    maps[0, 2] = [0.6, 0.25, 0.15]
    maps[0, 3] = [0.4, 0.4, 0.2]
    idx, score = np.array([[0]]), np.array([[0.9]])
    full = (1 << E) - 1
    masks = np.array([[full] * L], dtype=np.uint64)
    # prefetch from layer 0: p / distance, layers 1, 2, 3 at distances 1, 2, 3
    order, pri, cnt = F.priority_order(maps, "f32", idx, score, F.BLEND_NONE, F.PRI_PREFETCH, masks, l_now=[0])
    assert cnt[0] == 9
    exp = sorted([(_f32(maps[0, l, j] / (l - 0.0)), l * E + j) for l in (1, 2, 3) for j in range(E)],
                 key=lambda t: (-t[0], t[1]))
    assert [int(o) for o in order[0, :9]] == [e for _, e in exp]
    # the nearest layer's 0.5 outranks the next layer's 0.6 (0.6 / 2 = 0.3)
    assert order[0, 0] == 1 * E + 0 and abs(pri[0, 0] - 0.5) == 0.0
    assert list(order[0, 9:]) == [-1] * (L * E - 9) and np.all(np.isneginf(pri[0, 9:]))
    # equal priorities (layer 3: 0.4 and 0.4 at distance 3) keep expert order
    pos = {int(e): i for i, e in enumerate(order[0, :9])}
    assert pos[3 * E + 0] < pos[3 * E + 1]
    # layers at or before the current one are never listed
    order, pri, cnt = F.priority_order(maps, "f32", idx, score, F.BLEND_NONE, F.PRI_PREFETCH, masks, l_now=[2])
    assert cnt[0] == 3 and set(int(e) for e in order[0, :3]) == {9, 10, 11}
    assert abs(pri[0, 0] - _f32(0.4)) == 0.0
    # eviction: 1 / (p * freq), least used and least likely first; zero use first of all
    freq = np.ones((L, E), np.float32)
    freq[2, 1] = 0.0
    freq[1, 0] = 10.0
    cache = np.array([0, 0b011, 0b110, 0], dtype=np.uint64)
    order, pri, cnt = F.priority_order(maps, "f32", idx, score, F.BLEND_NONE, F.PRI_EVICT, cache, freq=freq)
    assert cnt[0] == 4
    assert int(order[0, 0]) == 2 * E + 1 and np.isposinf(pri[0, 0])
    assert [int(e) for e in order[0, 1:4]] == [2 * E + 2, 1 * E + 1, 1 * E + 0]
    assert abs(pri[0, 3] - _f32(1.0 / (0.5 * 10.0))) == 0.0
    # a query without a match lists nothing; a cap keeps the first entries
    order, pri, cnt = F.priority_order(maps, "f32", np.array([[-1]]), np.array([[-np.inf]]), F.BLEND_NONE,
                                       F.PRI_PREFETCH, masks, l_now=[0], cap=2)
    assert cnt[0] == 0 and list(order[0]) == [-1, -1]
    order, pri, cnt = F.priority_order(maps, "f32", idx, score, F.BLEND_NONE, F.PRI_PREFETCH, masks, l_now=[0],
                                       cap=2)
    assert cnt[0] == 9 and [int(o) for o in order[0]] == [e for _, e in exp[:2]]


def check_priority_vs_brute(seed=18):
    rng = np.random.default_rng(seed)
    for trial in range(40):
        L, E, n, k = int(rng.integers(1, 6)), int(rng.integers(1, 9)), 5, 3
        maps = _rand_maps(rng, n, L, E, zero_frac=0.3)
        if trial % 3 == 0:
            maps = np.round(maps * 4) / 4   # ties
        if trial % 7 == 0:
            maps[1, 0, 0] = np.nan
        idx = rng.permutation(n)[:k][None, :]
        score = np.sort(rng.uniform(-0.2, 1, k))[::-1][None, :]
        blend = F.BLEND_SCORE if trial % 2 else F.BLEND_NONE
        rows = [F.guide_row(maps, "f32", idx[0], score[0], blend, l) for l in range(L)]
        masks = rng.integers(0, 1 << E, size=(1, L)).astype(np.uint64)
        l_now = int(rng.integers(-1, L))
        order, pri, cnt = F.priority_order(maps, "f32", idx, score, blend, F.PRI_PREFETCH, masks, l_now=[l_now])
        bits = [int(masks[0, l]) if l > l_now else 0 for l in range(L)]
        ref = brute.priority_list(rows, bits, lambda l, j, p: _f32(p / (l - l_now)))
        assert cnt[0] == len(ref) and [int(o) for o in order[0, :cnt[0]]] == [e for _, e in ref], trial
        freq = rng.integers(0, 4, size=(L, E)).astype(np.float32)
        cache = rng.integers(0, 1 << E, size=L).astype(np.uint64)
        order, pri, cnt = F.priority_order(maps, "f32", idx, score, blend, F.PRI_EVICT, cache, freq=freq)

        def evict(l, j, p):
            prod = p * float(freq[l, j])
            return _f32(math.nan if math.isnan(prod) else (math.inf if prod == 0.0 else 1.0 / prod))

        ref = brute.priority_list(rows, [int(c) for c in cache], evict)
        assert cnt[0] == len(ref) and [int(o) for o in order[0, :cnt[0]]] == [e for _, e in ref], trial
        got = pri[0, :cnt[0]]
        assert all((math.isnan(a) and math.isnan(b)) or a == b for a, b in zip(got.tolist(), [v for v, _ in ref]))


# ------------------------------------------------------------------ misses (Section 3)

def check_misses_closed_forms():
    Q = np.array([[[0.5, 0.3, 0.1, 0.1], [0.25, 0.25, 0.25, 0.25]]], np.float32)
    full = np.array([[0b1111, 0b1111]], np.uint64)
    empty = np.zeros((1, 2), np.uint64)
    lb, le = np.array([0]), np.array([2])
    assert F.miss_counts(Q, "f32", full, 2, lb, le).tolist() == [[0, 0]]
    assert F.miss_counts(Q, "f32", empty, 2, lb, le).tolist() == [[2, 2]]
    # layer 0 activates {0, 1}; the set {0, 2} misses expert 1
    assert F.miss_counts(Q, "f32", np.array([[0b0101, 0]], np.uint64), 2, lb, np.array([1])).tolist() == [[1, 0]]
    # equal probabilities activate the lower indices {0, 1}
    assert F.activated(Q[0, 1], 2) == 0b0011
    assert F.miss_counts(Q, "f32", np.array([[0, 0b1100]], np.uint64), 2, np.array([1]), le).tolist() == [[0, 2]]
    # K = E: every expert is activated
    assert F.activated(Q[0, 0], 4) == 0b1111
    assert F.activated(np.array([np.nan, 0.1, 0.2]), 1) == 0b100


def check_misses_vs_enumeration(seed=19):
    rng = np.random.default_rng(seed)
    for _ in range(200):
        E = int(rng.integers(1, 9))
        K = int(rng.integers(1, E + 1))
        p = rng.dirichlet(np.ones(E))
        if rng.random() < 0.3:
            p = np.round(p * 4) / 4
        chosen = int(rng.integers(0, 1 << E))
        Q = p.astype(np.float32)[None, None, :]
        got = int(F.miss_counts(Q, "f32", np.array([[chosen]], np.uint64), K, np.array([0]), np.array([1]))[0, 0])
        ref = brute.misses_by_enumeration(F.widen(Q[0, 0], "f32").tolist(), K, chosen)
        assert got == ref, (p, K, chosen, got, ref)


# ------------------------------------------------------------------ blend glue and chunked search

def _maps_as_lists(maps):
    return F.widen(maps, "f32").tolist()


def check_guide_row_blend(seed=20):
    """BLEND_SCORE guiding rows against the fsum blend: each weight goes with
    its own match's row, missing matches (index -1) are skipped even when
    their score is finite, a NaN score weighs 0, and all-zero weights give
    the plain mean of the valid rows."""
    rng = np.random.default_rng(seed)
    n, L, E = 12, 4, 5
    maps = _rand_maps(rng, n, L, E)
    ml = _maps_as_lists(maps)
    cases = [
        ([3, 7, 1, 9], [0.9, 0.6, 0.3, 0.05]),        # distinct weights per match
        ([5, 2, -1, -1], [0.8, 0.4, -np.inf, -np.inf]),  # missing matches
        ([4, -1, -1, -1], [-0.2, -np.inf, -np.inf, -np.inf]),  # no positive weight: mean of the valid row
        ([6, 8, -1], [-0.1, 0.0, 0.7]),               # missing match with a finite score is not used
        ([0, 11, 2], [np.nan, 0.5, 0.25]),            # NaN weighs 0
        ([1, 10], [np.nan, np.nan]),                  # every weight 0: plain mean
        ([9, 3, 0], [0.7, -0.3, 0.2]),                # a negative weight is dropped
    ]
    for idx_row, sc_row in cases:
        idx_row = np.array(idx_row)
        sc_row = np.array(sc_row, dtype=np.float64)
        for l in range(L):
            got = F.guide_row(maps, "f32", idx_row, sc_row, F.BLEND_SCORE, l)
            ref = brute.guide_fsum(ml, idx_row.tolist(), sc_row.tolist(), True, l)
            assert not np.any(np.isnan(got)), (idx_row, sc_row)
            assert np.max(np.abs(got - np.array(ref))) <= 4e-16, (idx_row, sc_row, l, got, ref)
            best = F.guide_row(maps, "f32", idx_row, sc_row, F.BLEND_NONE, l)
            assert np.array_equal(best, np.array(ml[idx_row[0]][l]))
    # a single valid match reproduces its row whatever its score (w * x / w
    # within one rounding of x)
    for sc in (0.9, 0.0, -0.5, np.nan):
        got = F.guide_row(maps, "f32", np.array([7, -1]), np.array([sc, -np.inf]), F.BLEND_SCORE, 2)
        ref = F.widen(maps[7, 2], "f32")
        assert np.all(np.abs(got - ref) <= 2.0 ** -52 * ref), (sc, got, ref)


def check_select_prefetch_blend(seed=21):
    """select_prefetch with BLEND_SCORE against the fsum blend and subset
    enumeration of Eq. 6-8, over ragged match lists."""
    rng = np.random.default_rng(seed)
    n, L, E, k = 15, 5, 6, 4
    maps = _rand_maps(rng, n, L, E, zero_frac=0.2)
    ml = _maps_as_lists(maps)
    B = 6
    idx = np.full((B, k), -1, dtype=np.int64)
    score = np.full((B, k), -np.inf)
    for b in range(B):
        m = int(rng.integers(1, k + 1))
        idx[b, :m] = rng.permutation(n)[:m]
        score[b, :m] = np.sort(rng.uniform(-0.3, 1.0, m))[::-1]
    score[2, 1] = np.nan
    lb = rng.integers(0, L, size=B)
    le = np.full(B, L)
    for tau in (0.3, 0.6, 0.85):
        mask, cnt = F.select_prefetch(maps, "f32", idx, score, lb, le, F.TAU_FIXED, tau, 1, E, F.BLEND_SCORE)
        t = float(np.float32(tau))
        for b in range(B):
            for l in range(L):
                if l < lb[b]:
                    assert mask[b, l] == 0 and cnt[b, l] == 0
                    continue
                p = brute.guide_fsum(ml, idx[b].tolist(), score[b].tolist(), True, l)
                kk, S = brute.prefetch_set(p, t, 1, E)
                assert cnt[b, l] == kk, (tau, b, l)
                assert int(mask[b, l]) == sum(1 << j for j in S), (tau, b, l)


def check_chunked_search(seed=22):
    """Searches over several store chunks (chunk size set to 7 for 60 stored
    iterations) against brute force over the whole store; duplicates planted
    across chunk boundaries keep the lowest index."""
    rng = np.random.default_rng(seed)
    old = F._CHUNK
    F._CHUNK = 7
    try:
        n, L, E = 60, 4, 5
        maps = _rand_maps(rng, n, L, E)
        maps[45] = maps[3]
        maps[59] = maps[3]
        Q = _rand_maps(rng, 5, L, E)
        Q[0] = maps[3]
        Q[1] = maps[58]
        depth = np.array([4, 2, 1, 3, 4])
        idx, sc = F.match_trajectory(maps, "f32", Q, depth, 3)
        m64 = F.widen(maps, "f32")
        q64 = F.widen(Q, "f32")
        for b in range(5):
            p = int(depth[b])
            ref = [brute.cosine_fsum(list(q64[b, :p].ravel()), list(m64[y, :p].ravel())) for y in range(n)]
            best = brute.best_matches(ref, 3)
            assert list(idx[b]) == best, (b, list(idx[b]), best)
            assert all(abs(sc[b, j] - ref[best[j]]) <= 1e-14 for j in range(3))
        assert list(idx[0]) == [3, 45, 59] and idx[1, 0] == 58
        X = _bf16(rng.standard_normal((n, 16)))
        X[33] = X[8]
        Qs = _bf16(rng.standard_normal((3, 16)))
        Qs[2] = X[8]
        idx, sc = F.match_semantic(X, Qs, 4)
        X64 = F.widen(X, "bf16")
        Q64 = F.widen(Qs, "bf16")
        for b in range(3):
            ref = [brute.cosine_fsum(list(Q64[b]), list(X64[y])) for y in range(n)]
            assert list(idx[b]) == brute.best_matches(ref, 4), b
        assert list(idx[2, :2]) == [8, 33]
        # fewer stored iterations than k across chunks: -1 / -inf fill
        idx, sc = F.match_trajectory(maps[:9], "f32", Q[:1], depth[:1], 12)
        assert list(idx[0, 9:]) == [-1, -1, -1] and np.all(np.isneginf(sc[0, 9:]))
        assert sorted(idx[0, :9].tolist()) == list(range(9))
        # redundancy over several chunks against the fsum pair formula
        old_maps, old_embs = maps[:20], _bf16(rng.standard_normal((20, 8)))
        new_maps, new_embs = maps[40:43], _bf16(rng.standard_normal((3, 8)))
        r = F.redundancy(old_maps, old_embs, new_maps, new_embs, "f32", 2)
        om, nm = F.widen(old_maps, "f32"), F.widen(new_maps, "f32")
        oe, ne = F.widen(old_embs, "bf16"), F.widen(new_embs, "bf16")
        for x in range(3):
            for y in range(20):
                ref = brute.redundancy_fsum(om[y].tolist(), oe[y].tolist(), nm[x].tolist(), ne[x].tolist(), 2)
                assert abs(r[x, y] - ref) <= 1e-14, (x, y)
    finally:
        F._CHUNK = old


ALL_CHECKS = [
    check_cosine_vs_fsum, check_cosine_vs_torch, check_self_match, check_disjoint_support,
    check_depth_special_cases, check_unobserved_layers_ignored, check_semantic_vs_fsum,
    check_match_vs_bruteforce, check_rank_rules, check_uniform_golden, check_delta_golden,
    check_select_vs_enumeration, check_select_nesting_and_minimality, check_blend,
    check_select_prefetch_layout, check_redundancy_vs_fsum, check_redundancy_closed_forms,
    check_dedup_vs_enumeration, check_dedup_duplicates, check_dedup_appends_first,
    check_research_schedule_depths, check_research_schedule_vs_fsum,
    check_priority_closed_forms, check_priority_vs_brute,
    check_misses_closed_forms, check_misses_vs_enumeration,
    check_guide_row_blend, check_select_prefetch_blend, check_chunked_search,
]
