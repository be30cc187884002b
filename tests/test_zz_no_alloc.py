"""fm_match_trajectory_noalloc (the trajectory search whose workspace is the
library's own device array) against fm_match_trajectory with a caller
workspace, through the C ABI: identical indices and scores on two calls in
a row, the second with a smaller batch and depth bound, and both against the
oracle (Eq. 5 top-k)."""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
import synth
from parity import compare_topk, to_device

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X GPU")]


def _call(lib, fn, store, q, depth, max_depth, B, k, ws=None):
    idx = torch.full((B, k), -7, dtype=torch.int32, device="cuda")
    sc = torch.full((B, k), 7.0, dtype=torch.float32, device="cuda")
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    args = [store.handle, C.c_void_p(q.data_ptr()), C.c_void_p(depth.data_ptr()), max_depth, B, k,
            C.c_void_p(idx.data_ptr()), C.c_void_p(sc.data_ptr())]
    if ws is not None:
        args += [ws.ptr, ws.nbytes]
    st = getattr(lib, fn)(*(args + [stream]))
    assert st == 0, (fn, st, lib.fm_last_error())
    torch.cuda.synchronize()
    return idx.cpu().numpy().astype(np.int64), sc.cpu().numpy().astype(np.float64)


def _oracle_check(maps, dtype, q, depth, gi, gs):
    oi, os_ = oracle.match_trajectory(maps, dtype, q, depth, gi.shape[1])

    def score_of(r, y):
        p = int(np.clip(depth[r], 1, q.shape[1]))
        return oracle.cosine(oracle.widen(q[r, :p], dtype), oracle.widen(maps[y, :p], dtype))

    rep = compare_topk(gi, gs, oi, os_, score_of)
    assert not rep.failures, rep.failures[:5]


# (the bf16 top-1 case of more than 128 queries runs the depth-band scan on the first call)
@pytest.mark.parametrize("cfg,n,B1,B2,k", [(2, 3001, 150, 37, 1), (5, 2500, 300, 20, 4), (4, 1800, 64, 9, 4),
                                           (5, 2500, 300, 20, 1)])
def test_noalloc_matches_workspace_call(cfg, n, B1, B2, k):
    import paper_2502_05370_amd as fm
    print(f"noalloc cfg={cfg} n={n} B={B1},{B2} k={k}", flush=True)
    lib = fm._lib.load()
    s = synth.spec(cfg).scaled(n=n, B_traj=B1, B_sem=0)
    a = synth.generate(s)
    store = fm.Store(n, s.L, s.E, 0, s.map_dtype)
    store.insert(to_device(a["maps"], s.map_dtype))
    ws = fm.Workspace(store)
    q_all = to_device(a["q_traj"], s.map_dtype)
    d_all = np.clip(a["depth"], 1, s.L).astype(np.int32)
    # first call: the whole batch; second: fewer queries with a lower depth bound
    for B, dmax in ((B1, s.L), (B2, max(2, s.L // 2))):
        q = q_all[:B].contiguous()
        d_np = np.minimum(d_all[:B], dmax)
        depth = to_device(d_np, "i32")
        ni, ns = _call(lib, "fm_match_trajectory_noalloc", store, q, depth, dmax, B, k)
        wi, wsc = _call(lib, "fm_match_trajectory", store, q, depth, dmax, B, k, ws=ws)
        assert np.array_equal(ni, wi), B
        assert np.array_equal(ns.view(np.int64), wsc.view(np.int64)), B
        _oracle_check(a["maps"], s.map_dtype, a["q_traj"][:B], d_np, ni, ns)
    assert store.check() == 0


def test_noalloc_argument_errors():
    import paper_2502_05370_amd as fm
    lib = fm._lib.load()
    s = synth.spec(1).scaled(n=100, B_traj=4)
    a = synth.generate(s)
    store = fm.Store(100, s.L, s.E)
    store.insert(to_device(a["maps"], "f32"))
    q = to_device(a["q_traj"], "f32")
    depth = to_device(a["depth"], "i32")
    idx = torch.empty((4, 1), dtype=torch.int32, device="cuda")
    sc = torch.empty((4, 1), dtype=torch.float32, device="cuda")
    p = lambda t: C.c_void_p(t.data_ptr())
    assert lib.fm_match_trajectory_noalloc(store.handle, p(q), p(depth), 0, 4, 1, p(idx), p(sc), None) == 1
    assert lib.fm_match_trajectory_noalloc(store.handle, p(q), p(depth), s.L, 4, 9, p(idx), p(sc), None) == 1
    assert lib.fm_match_trajectory_noalloc(store.handle, None, p(depth), s.L, 4, 1, p(idx), p(sc), None) == 1
    assert lib.fm_match_trajectory_noalloc(None, p(q), p(depth), s.L, 4, 1, p(idx), p(sc), None) == 1
