"""GPU parity of the Section 3 miss indicator through the C ABI, on the
pipeline the capacity study runs: fresh iterations are matched against a
store (trajectory at their depth, semantic by embedding), their prefetch sets
selected, and the activated experts (top-K of their own gate probabilities)
outside the sets counted.  Counts must equal the oracle's exactly."""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from parity import to_device

pytestmark = pytest.mark.gpu

MODELS = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "models.json")))["models"]
K_OF = {1: MODELS["mixtral_8x7b"]["K"], 2: MODELS["qwen1.5_moe"]["K"], 3: MODELS["mixtral_8x7b"]["K"],
        4: MODELS["phi3.5_moe"]["K"], 5: MODELS["qwen1.5_moe"]["K"]}


def _pipeline(cfg, n, m):
    import paper_2502_05370_amd as fm
    import torch
    s = synth.spec(cfg).scaled(n=n, B_traj=0, B_sem=0)
    a = synth.generate(s)
    new = synth.generate_new(s, m, a, dup_frac=0.0)
    store = fm.Store(n, s.L, s.E, s.d_emb, s.map_dtype)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16") if s.d_emb else None)
    rng = np.random.default_rng(cfg)
    depth = rng.integers(1, s.L, size=m).astype(np.int32)
    q = to_device(new["new_maps"], s.map_dtype)
    idx, score = fm.match_trajectory(store, q, to_device(depth, "i32"), s.k)
    lb, le = depth.copy(), np.full(m, s.L, np.int32)
    if s.d_emb:   # the first half searched by embedding, guiding every layer
        h = m // 2
        fm.match_semantic(store, to_device(new["new_embs"][:h], "bf16"), s.k, out=(idx[:h], score[:h]))
        lb[:h] = 0
    lbt, let = to_device(lb, "i32"), to_device(le, "i32")
    mask, _ = fm.select_prefetch(store, idx, score, lbt, let, tau=s.tau, k_min=s.k_min, k_max=s.k_max,
                                 mode=s.tau_mode, blend=s.blend)
    miss = fm.miss_count(store, q, mask, K_OF[cfg], lbt, let)
    torch.cuda.synchronize()
    return s, new, mask.cpu().numpy().view(np.uint64), miss.cpu().numpy(), lb, le


@pytest.mark.parametrize("cfg,n,m", [(1, 1000, 24), (2, 3001, 64), (3, 2050, 40), (4, 4003, 100), (5, 2501, 50)])
def test_misses_match_oracle(cfg, n, m):
    s, new, mask, miss, lb, le = _pipeline(cfg, n, m)
    ref = oracle.miss_counts(new["new_maps"], s.map_dtype, mask, K_OF[cfg], lb, le)
    assert np.array_equal(miss, ref), np.argwhere(miss != ref)[:5]
    # a sanity property of the pipeline: most activated experts are prefetched
    rows = sum(int(h - l) for l, h in zip(lb, le))
    assert ref.sum() < 0.5 * K_OF[cfg] * rows


def test_miss_edge_cases():
    import paper_2502_05370_amd as fm
    L, E = 3, 64
    rng = np.random.default_rng(0)
    q = rng.dirichlet(np.ones(E), size=(5, L)).astype(np.float32)
    q[1, 0, :] = 0.25                 # all equal: the lowest K indices are activated
    q[2, 1, 7] = np.nan               # NaN ranks last
    store = fm.Store(4, L, E, 0, "f32")
    masks = rng.integers(0, 1 << 62, size=(5, L), dtype=np.int64).astype(np.uint64)
    masks[3] = np.uint64((1 << 64) - 1)   # everything prefetched
    masks[4] = 0                          # nothing prefetched
    lb = np.array([0, 0, 0, 1, -5], np.int32)
    le = np.array([3, 3, 2, 9, 3], np.int32)
    for K in (1, 4, 64):
        got = fm.miss_count(store, to_device(q, "f32"), to_device(masks.view(np.int64), "i64"), K,
                            to_device(lb, "i32"), to_device(le, "i32")).cpu().numpy()
        ref = oracle.miss_counts(q, "f32", masks, K, lb, le)
        assert np.array_equal(got, ref), (K, got, ref)
    with pytest.raises(fm.FmError):
        fm.miss_count(store, to_device(q, "f32"), to_device(masks.view(np.int64), "i64"), 65,
                      to_device(lb, "i32"), to_device(le, "i32"))
