"""The Python binding rejects tensors whose device, dtype, shape or layout
the kernels would misread, before anything reaches the C ABI (CPU only: a
stand-in store object carries the shape; no call reaches the library)."""
import types

import pytest
import torch

import paper_2502_05370_amd as fm

DEV = torch.device("cuda", 0)


def _store(L=4, E=8, d_emb=128, dtype="f32"):
    return types.SimpleNamespace(L=L, E=E, d_emb=d_emb, map_dtype=dtype, dtype_code=fm._DTYPES[dtype], device=DEV,
                                 handle=None)


def _meta(shape, dtype):
    # tensors on the meta device: right shape and dtype, wrong device
    return torch.empty(shape, dtype=dtype, device="meta")


def test_wrong_device_rejected():
    s = _store()
    with pytest.raises(ValueError, match="is on"):
        fm.match_trajectory(s, torch.zeros(3, 4, 8), torch.ones(3, dtype=torch.int32))
    with pytest.raises(ValueError, match="is on"):
        fm.match_semantic(s, torch.zeros(3, 128, dtype=torch.bfloat16))


def test_checks_in_order(monkeypatch):
    """With the device check satisfied (the helper is asked about tensors on
    the store's device), dtype, shape and layout are each rejected."""
    s = _store()
    s.device = torch.device("cpu")
    q = torch.zeros(3, 4, 8)
    with pytest.raises(ValueError, match="int32"):
        fm.match_trajectory(s, q, torch.ones(3, dtype=torch.int64))          # torch's default integer type
    with pytest.raises(ValueError, match="shape"):
        fm.match_trajectory(s, torch.zeros(3, 3, 8), torch.ones(3, dtype=torch.int32))   # fewer than L layers
    with pytest.raises(ValueError, match="shape"):
        fm.match_trajectory(s, q, torch.ones(2, dtype=torch.int32))
    with pytest.raises(ValueError, match="float32"):
        fm.match_trajectory(s, q.double(), torch.ones(3, dtype=torch.int32))
    with pytest.raises(ValueError, match="contiguous"):
        fm.match_trajectory(s, torch.zeros(3, 8, 4).transpose(1, 2), torch.ones(3, dtype=torch.int32))
    small = (torch.empty(3, 1, dtype=torch.int32), torch.empty(3, 1))
    with pytest.raises(ValueError, match="out\\[0\\]"):
        fm.match_trajectory(s, q, torch.ones(3, dtype=torch.int32), k=2, out=small)
    with pytest.raises(ValueError, match="bfloat16"):
        fm.match_semantic(s, torch.zeros(3, 128))
    with pytest.raises(ValueError, match="shape"):
        fm.match_semantic(s, torch.zeros(3, 64, dtype=torch.bfloat16))
    idx = torch.zeros(3, 1, dtype=torch.int32)
    sc = torch.zeros(3, 1)
    lb = torch.zeros(3, dtype=torch.int32)
    with pytest.raises(ValueError, match="int32"):
        fm.select_prefetch(s, idx.long(), sc, lb, lb)
    with pytest.raises(ValueError, match="layer_end"):
        fm.select_prefetch(s, idx, sc, lb, torch.zeros(3, dtype=torch.int64))
    with pytest.raises(ValueError, match="out\\[0\\]"):
        fm.select_prefetch(s, idx, sc, lb, lb, out=(torch.empty(3, 2, dtype=torch.int64),
                                                    torch.empty(3, 4, dtype=torch.uint8)))
    with pytest.raises(ValueError, match="masks"):
        fm.priority_order(s, idx, sc, torch.zeros(3, 2, dtype=torch.int64), l_now=lb)
    with pytest.raises(ValueError, match="l_now"):
        fm.priority_order(s, idx, sc, torch.zeros(3, 4, dtype=torch.int64), l_now=None)
    with pytest.raises(ValueError, match="freq"):
        fm.priority_order(s, idx, sc, torch.zeros(4, dtype=torch.int64), kind=fm.FM_PRI_EVICT,
                          freq=torch.zeros(4, 7))
    with pytest.raises(ValueError, match="masks"):
        fm.miss_count(s, q, torch.zeros(3, 4, dtype=torch.int32), 2, lb, lb)
    with pytest.raises(ValueError, match="required"):
        fm.match_trajectory(s, q, None)
    with pytest.raises(TypeError):
        fm.match_trajectory(s, q, [1, 2, 3])
