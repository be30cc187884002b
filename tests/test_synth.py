"""The seeded input generator: determinism, row sums, bf16 rounding, shapes."""
import numpy as np
import pytest
import torch

import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 3.0e38, 1e-40, np.inf, -np.inf], dtype=np.float32)])
    ours = synth.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = synth.bf16_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_small_workloads_shapes_and_invariants(cfg):
    s = synth.spec(cfg).scaled(n=300, B_traj=min(synth.spec(cfg).B_traj, 16),
                               B_sem=min(synth.spec(cfg).B_sem, 8))
    a = synth.generate(s)
    assert a["maps"].shape == (300, s.L, s.E)
    p = synth.values_f32(a["maps"], s.map_dtype).astype(np.float64)
    assert np.all(p >= 0)
    tol = s.E * (2.0 ** -8 if s.map_dtype == "bf16" else 2.0 ** -24)
    assert np.max(np.abs(p.sum(-1) - 1.0)) <= tol
    if s.B_traj:
        q = synth.values_f32(a["q_traj"], s.map_dtype).astype(np.float64)
        assert np.max(np.abs(q.sum(-1) - 1.0)) <= tol
        assert a["depth"].min() >= 1 and a["depth"].max() <= s.depth_max
        assert np.array_equal(a["lb"][s.B_sem:], a["depth"])
    if s.d_emb:
        e = synth.bf16_to_f32(a["embs"]).astype(np.float64)
        nrm = np.linalg.norm(e, axis=1)
        assert np.max(np.abs(nrm - 1.0)) <= 2.0 ** -8
    assert a["lb"].shape == (s.B,) and np.all(a["le"] == s.L)


def test_determinism():
    s = synth.spec(4).scaled(n=500, B_traj=32)
    d1 = synth.digests(synth.generate(s))
    d2 = synth.digests(synth.generate(s))
    assert d1 == d2
    s2 = synth.spec(2).scaled(n=500, B_traj=32)
    assert synth.digests(synth.generate(s2))["maps"] != d1["maps"]


def test_geometric_depths_skew_shallow():
    s = synth.spec(4)
    d = synth.generate(s.scaled(n=64))["depth"]
    assert d.shape == (512,) and d.min() >= 1 and d.max() <= 31
    assert 4.5 < d.mean() < 9.0


@pytest.mark.parametrize("cfg", [2, 3, 5])
def test_new_iterations(cfg):
    s = synth.spec(cfg).scaled(n=200, B_traj=0, B_sem=0)
    a = synth.generate(s)
    b = synth.generate_new(s, 64, a, dup_frac=0.25)
    assert b["new_maps"].shape == (64, s.L, s.E) and b["new_maps"].dtype == a["maps"].dtype
    dup = b["dup_src"]
    assert 0 < int((dup >= 0).sum()) < 64
    for x in np.flatnonzero(dup >= 0):
        assert np.array_equal(b["new_maps"][x], a["maps"][dup[x]])
        if s.d_emb:
            assert np.array_equal(b["new_embs"][x], a["embs"][dup[x]])
    p = synth.values_f32(b["new_maps"], s.map_dtype).astype(np.float64)
    tol = s.E * (2.0 ** -8 if s.map_dtype == "bf16" else 2.0 ** -24)
    assert np.max(np.abs(p.sum(-1) - 1.0)) <= tol
    # deterministic
    c = synth.generate_new(s, 64, a, dup_frac=0.25)
    assert all(np.array_equal(b[k], c[k]) for k in b)
