"""GPU parity of the Section 4.5 priority ordering through the C ABI.

The order, the float32 priorities and the candidate counts must equal the
oracle's bit for bit (both sides round the float64 priority to float32 and
order on it), given the GPU's own matches and prefetch sets."""
import numpy as np
import pytest

import oracle
import synth
from parity import run_gpu, to_device

pytestmark = pytest.mark.gpu


def _gpu_order(store, g, s, kind, masks, l_now=None, freq=None, cap=None):
    import paper_2502_05370_amd as fm
    import torch
    idx = torch.from_numpy(g.idx.astype(np.int32)).cuda()
    score = torch.from_numpy(g.score.astype(np.float32)).cuda()
    m = torch.from_numpy(np.ascontiguousarray(masks).view(np.int64)).cuda()
    ln = torch.from_numpy(np.asarray(l_now, dtype=np.int32)).cuda() if l_now is not None else None
    fr = torch.from_numpy(np.asarray(freq, dtype=np.float32)).cuda() if freq is not None else None
    order, pri, count = fm.priority_order(store, idx, score, m, l_now=ln, freq=fr, kind=kind, blend=s.blend, cap=cap)
    return order.cpu().numpy(), pri.cpu().numpy(), count.cpu().numpy()


def _check(s, a, g, got, kind, masks, l_now=None, freq=None, cap=None):
    order, pri, count = oracle.priority_order(a["maps"], s.map_dtype, g.idx, g.score.astype(np.float32), s.blend,
                                              kind, masks, l_now=l_now, freq=freq, cap=cap)
    go, gp, gc = got
    assert np.array_equal(gc, count), (gc[:8], count[:8])
    assert np.array_equal(go, order), np.argwhere(go != order)[:5]
    same = (gp == pri) | (np.isnan(gp) & np.isnan(pri))
    assert same.all(), np.argwhere(~same)[:5]


def _store_and_match(cfg, n, bt, bs, **kw):
    import paper_2502_05370_amd as fm
    s = synth.spec(cfg).scaled(n=n, B_traj=bt, B_sem=bs, **kw)
    a = synth.generate(s)
    g = run_gpu(s, a)
    # run_gpu's store is gone; rebuild one with the same contents for the ordering call
    store = fm.Store(n, s.L, s.E, s.d_emb, s.map_dtype)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16") if s.d_emb else None)
    return s, a, g, store


@pytest.mark.parametrize("cfg,n,bt,bs", [(1, 1000, 8, 0), (2, 3001, 64, 0), (3, 2050, 0, 40), (4, 4003, 100, 0),
                                         (5, 2501, 30, 20)])
def test_prefetch_order_matches_oracle(cfg, n, bt, bs):
    s, a, g, store = _store_and_match(cfg, n, bt, bs)
    l_now = a["lb"].astype(np.int64) - 1      # the layer before the first selected one
    got = _gpu_order(store, g, s, oracle.PRI_PREFETCH, g.mask, l_now=l_now)
    _check(s, a, g, got, oracle.PRI_PREFETCH, g.mask, l_now=l_now)
    assert store.check() == 0
    # a cap keeps the first entries; l_now beyond the set lists nothing
    cap = 5
    got = _gpu_order(store, g, s, oracle.PRI_PREFETCH, g.mask, l_now=l_now, cap=cap)
    _check(s, a, g, got, oracle.PRI_PREFETCH, g.mask, l_now=l_now, cap=cap)
    late = np.full(s.B, s.L - 1)
    got = _gpu_order(store, g, s, oracle.PRI_PREFETCH, g.mask, l_now=late)
    assert np.all(got[2] == 0) and np.all(got[0] == -1)


@pytest.mark.parametrize("cfg,n,bt,bs", [(2, 3001, 64, 0), (4, 4003, 100, 0), (5, 2501, 30, 20)])
def test_evict_order_matches_oracle(cfg, n, bt, bs):
    s, a, g, store = _store_and_match(cfg, n, bt, bs)
    rng = np.random.default_rng(cfg)
    cache = rng.integers(0, 1 << 62, size=s.L, dtype=np.int64).astype(np.uint64) & np.uint64((1 << s.E) - 1)
    freq = rng.integers(0, 20, size=(s.L, s.E)).astype(np.float32)   # zeros: never visited
    got = _gpu_order(store, g, s, oracle.PRI_EVICT, cache, freq=freq)
    _check(s, a, g, got, oracle.PRI_EVICT, cache, freq=freq)


def test_full_width_and_special_values():
    """E = 64 and L = 64 with every expert selected (4096 candidates, the
    largest sort), a NaN probability, a query without a match and an index
    past the store."""
    import paper_2502_05370_amd as fm
    import torch
    L, E, n = 64, 64, 40
    rng = np.random.default_rng(5)
    z = rng.standard_normal((n, L, E))
    maps = (np.exp(z) / np.exp(z).sum(-1, keepdims=True)).astype(np.float32)
    maps[3, 10, 7] = np.nan
    maps[4] = np.round(maps[4] * 8) / 8          # many equal priorities
    store = fm.Store(n, L, E, 0, "f32")
    store.insert(to_device(maps, "f32"))
    s = synth.spec(1).scaled(n=n, B_traj=4, B_sem=0, L=L, E=E)

    class G:
        idx = np.array([[3], [4], [-1], [n + 5]])
        score = np.array([[0.9], [0.5], [-np.inf], [0.2]])
    full = np.full((4, L), np.uint64((1 << 64) - 1), dtype=np.uint64)
    l_now = np.array([-1, 20, 0, 0])
    got = _gpu_order(store, G, s, oracle.PRI_PREFETCH, full, l_now=l_now)
    assert got[2][0] == L * E and got[2][1] == (L - 21) * E and got[2][2] == 0 and got[2][3] == 0
    assert store.check() == fm.FM_FLAG_INDEX_RANGE
    # the oracle on the valid queries (the out-of-range one lists nothing)
    G.idx = G.idx[:3]
    G.score = G.score[:3]
    got = tuple(x[:3] for x in got)
    _check(s, {"maps": maps}, G, got, oracle.PRI_PREFETCH, full[:3], l_now=l_now[:3])
    freq = np.ones((L, E), np.float32)
    got = _gpu_order(store, G, s, oracle.PRI_EVICT, full[0], freq=freq)
    _check(s, {"maps": maps}, G, got, oracle.PRI_EVICT, full[0], freq=freq)
