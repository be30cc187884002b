"""GPU parity of the top-1 semantic scan (k_sem_mm) on inputs at the edges of
its ranking: queries of either sign and of norms far from 1 (bf16 values
scaled by powers of two, exactly), a zero query (every cosine 0: the first
map), a query with a NaN (every cosine NaN), zero and NaN stored embeddings;
with query groups of 128 (one group) and 256 (two groups, a ragged tail),
through the C ABI against the CPU oracle on the same seeded inputs."""
import dataclasses

import numpy as np
import pytest
import torch

import synth

from parity import compare_match, oracle_match, run_gpu

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X GPU")]


def _widen(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


@pytest.mark.parametrize("B", [100, 300])
def test_sem_mm_signed_scaled_zero_and_nan(B):
    s = dataclasses.replace(synth.spec(5).scaled(n=3001, B_traj=0, B_sem=B), k=1)
    print(f"semantic top-1 edges: d={s.d_emb} n={s.n} B_sem={s.B_sem}", flush=True)
    a = synth.generate(s)
    q = _widen(a["q_sem"]).copy()
    q[0::5] *= -1.0
    q[1::5] *= 64.0
    q[2::5] *= 1.0 / 64.0
    q[3] = 0.0                   # zero query
    q[4, 7] = np.nan             # NaN query
    a["q_sem"] = synth.bf16_bits(q.reshape(-1)).reshape(a["q_sem"].shape)
    e = _widen(a["embs"]).copy()
    e[10] = 0.0                  # zero norm: cosine 0
    e[11, 3] = np.nan            # NaN: ranks last
    a["embs"] = synth.bf16_bits(e.reshape(-1)).reshape(a["embs"].shape)
    g = run_gpu(s, a)
    assert g.flags == 0
    oi, os_ = oracle_match(s, a)
    rep = compare_match(s, a, g.idx, g.score, oi, os_, np.arange(s.B))
    assert not rep.failures, rep.failures[:5]
    assert g.idx[3, 0] == 0 and g.score[3, 0] == 0.0
    assert g.idx[4, 0] == 0 and np.isnan(g.score[4, 0])
    assert not np.any(g.idx[:, 0] == 11)
