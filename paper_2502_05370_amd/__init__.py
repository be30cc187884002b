"""FineMoE expert-map matching and prefetch selection on MI355X (gfx950).

A thin Python binding over the C ABI of ``libfinemoe_map.so``
(include/finemoe_map.h).  PyTorch provides device memory and streams only:
every step of the path (store residency, semantic and trajectory search,
ranking, blending, thresholding and selection) runs in the library's HIP
kernels.  There is no CPU fallback; the import fails if the library has not
been built.

    store = Store(cap, L, E, d_emb=0, map_dtype="f32")
    store.insert(maps, embs=None)                       # maps [n][L][E] on the GPU
    slots = store.insert_dedup(maps, embs, d)           # Section 4.4, replaces when full
    idx, score = match_trajectory(store, q, depth, k=1) # Eq. 5
    idx, score = match_semantic(store, q_sem, k=1)      # Eq. 4
    tp = TrajPass(store, B)                             # Section 4.2.2, one pass
    idx, score = tp.step(q_layer, layer, k=1)           # after each observed layer
    mask, count = select_prefetch(store, idx, score, layer_begin, layer_end,
                                  tau=0.8, k_min=1, k_max=8)   # Eq. 6-8
    order, pri, n = priority_order(store, idx, score, mask, l_now=l_now)  # Section 4.5
"""
from __future__ import annotations

import ctypes as C
from typing import Optional, Tuple

import torch

from . import _lib
from ._lib import (FM_BF16, FM_BLEND_NONE, FM_BLEND_SCORE, FM_F32, FM_FLAG_DEPTH_CLAMPED,  # noqa: F401
                   FM_FLAG_INDEX_RANGE, FM_FLAG_STATE_STALE, FM_PRI_EVICT, FM_PRI_PREFETCH, FM_TAU_DYNAMIC, FM_TAU_FIXED, FmError, SelectParams)

_lib.load()

__all__ = ["Store", "Workspace", "match_semantic", "match_trajectory", "match_trajectory_noalloc", "select_prefetch", "priority_order",
           "miss_count",
           "debug_scores",
           "map_bytes", "store_bytes", "workspace_bytes", "dedup_scratch_bytes", "traj_state_bytes", "TrajPass",
           "FmError"]

_DTYPES = {"f32": FM_F32, "bf16": FM_BF16}
_TORCH = {FM_F32: torch.float32, FM_BF16: torch.bfloat16}


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _need(t, name: str, dtype, shape, device) -> torch.Tensor:
    """Check a tensor handed to the library: on the store's device,
    contiguous, of the expected dtype and shape (None in ``shape`` matches any
    size).  The kernels read and write through raw pointers, so a wrong
    layout would be read out of bounds instead of failing; raise instead."""
    if t is None:
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the store is on {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != len(shape) or any(w is not None and g != w for g, w in zip(t.shape, shape)):
        want = "x".join("*" if w is None else str(w) for w in shape)
        raise ValueError(f"{name} must have shape [{want}], got {list(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _dev(store: "Store") -> torch.device:
    return store.device


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _aligned_bytes(nbytes: int, device) -> torch.Tensor:
    """A 256-byte aligned uint8 device tensor of ``nbytes`` bytes."""
    raw = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-raw.data_ptr()) % 256
    return raw[off:off + nbytes]


def map_bytes(cap: int, L: int, E: int, map_dtype: str = "f32") -> int:
    return int(_lib.load().fm_map_bytes(cap, L, E, _DTYPES[map_dtype]))


def store_bytes(cap: int, L: int, E: int, d_emb: int = 0, map_dtype: str = "f32") -> int:
    return int(_lib.load().fm_store_bytes(cap, L, E, d_emb, _DTYPES[map_dtype]))


def workspace_bytes(L: int, E: int, d_emb: int = 0, map_dtype: str = "f32", B_max: int = 1024,
                    k_max: int = 8) -> int:
    return int(_lib.load().fm_workspace_bytes(L, E, d_emb, _DTYPES[map_dtype], B_max, k_max))


def dedup_scratch_bytes(cap: int, n_max: int) -> int:
    return int(_lib.load().fm_dedup_scratch_bytes(cap, n_max))


class Workspace:
    """Device scratch for match calls (every call rewrites what it reads).
    Calls sharing one workspace must be ordered."""

    def __init__(self, store: "Store", B_max: int = 1024, k_max: int = 8, device=None):
        self.nbytes = workspace_bytes(store.L, store.E, store.d_emb, store.map_dtype, B_max, k_max)
        if self.nbytes == 0:
            raise ValueError(f"invalid workspace request B_max={B_max} k_max={k_max}")
        device = store.device if device is None else device
        self.buf = _aligned_bytes(self.nbytes, device)

    @property
    def ptr(self):
        return C.c_void_p(self.buf.data_ptr())


class Store:
    """Expert Map Store held in one device buffer owned by this object."""

    def __init__(self, cap: int, L: int, E: int, d_emb: int = 0, map_dtype: str = "f32", device="cuda"):
        self.cap, self.L, self.E, self.d_emb = int(cap), int(L), int(E), int(d_emb)
        self.map_dtype = map_dtype
        self.dtype_code = _DTYPES[map_dtype]
        self.device = torch.device(device)
        if self.device.type == "cuda" and self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        nbytes = store_bytes(cap, L, E, d_emb, map_dtype)
        if nbytes == 0:
            raise ValueError(f"invalid store shape cap={cap} L={L} E={E} d_emb={d_emb}")
        with torch.cuda.device(self.device):
            self.buf = _aligned_bytes(nbytes, self.device)
            desc = _lib.StoreDesc(self.cap, self.L, self.E, self.d_emb, self.dtype_code,
                                  C.c_void_p(self.buf.data_ptr()), nbytes)
            h = C.c_void_p()
            _lib.check(_lib.load().fm_store_build(C.byref(h), C.byref(desc)), "fm_store_build")
        self.handle = h
        self.workspace = None
        self._dedup_scratch = None

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value and _lib is not None and _lib._LIB is not None:
            _lib._LIB.fm_store_destroy(h)
            self.handle = None

    @property
    def size(self) -> int:
        n = C.c_int32()
        _lib.check(_lib.load().fm_store_size(self.handle, C.byref(n)), "fm_store_size")
        return n.value

    def insert(self, maps: torch.Tensor, embs: Optional[torch.Tensor] = None, stream=None,
               return_slots: bool = False):
        """Append maps [n][L][E] (and embeddings [n][d_emb] bf16) already on the device."""
        dev = _dev(self)
        maps = _need(maps.contiguous(), "maps", _TORCH[self.dtype_code], (None, self.L, self.E), dev)
        n = maps.shape[0]
        if embs is not None:
            embs = _need(embs.contiguous(), "embs", torch.bfloat16, (n, self.d_emb), dev)
        slots = torch.empty(n, dtype=torch.int32, device=dev) if return_slots else None
        _lib.check(_lib.load().fm_store_insert(self.handle, _ptr(maps), _ptr(embs), n, _ptr(slots),
                                               _stream(stream)), "fm_store_insert")
        return slots

    def insert_dedup(self, maps: torch.Tensor, embs: Optional[torch.Tensor], d: int,
                     workspace: Optional["Workspace"] = None, scratch: Optional[torch.Tensor] = None,
                     stream=None) -> torch.Tensor:
        """Insert with deduplication (Section 4.4): append while there is room,
        then replace the most redundant stored iterations (RDY with prefetch
        distance d).  Returns the slot of each new iteration (int32, -1 if
        dropped) on the device."""
        dev = _dev(self)
        maps = _need(maps.contiguous(), "maps", _TORCH[self.dtype_code], (None, self.L, self.E), dev)
        n = maps.shape[0]
        if embs is not None:
            embs = _need(embs.contiguous(), "embs", torch.bfloat16, (n, self.d_emb), dev)
        ws = workspace if workspace is not None else self.ensure_workspace()
        if scratch is None:
            need = dedup_scratch_bytes(self.cap, max(n, 1))
            if self._dedup_scratch is None or self._dedup_scratch.numel() < need:
                self._dedup_scratch = _aligned_bytes(need, self.device)
            scratch = self._dedup_scratch
        slots = torch.empty(n, dtype=torch.int32, device=self.device)
        _lib.check(_lib.load().fm_store_insert_dedup(self.handle, _ptr(maps), _ptr(embs), n, int(d), _ptr(slots),
                                                     ws.ptr, ws.nbytes, _ptr(scratch), scratch.numel(),
                                                     _stream(stream)), "fm_store_insert_dedup")
        return slots

    def check(self, stream=None) -> int:
        """Synchronise and return the sticky device flags (raises FmError if any)."""
        f = C.c_uint32()
        st = _lib.load().fm_store_check(self.handle, _stream(stream), C.byref(f))
        if st == _lib.FM_ERR_DEVICE:
            return f.value
        _lib.check(st, "fm_store_check")
        return f.value

    def ensure_workspace(self) -> Workspace:
        if self.workspace is None:
            self.workspace = Workspace(self)
        return self.workspace


def traj_state_bytes(cap: int, B_max: int) -> int:
    return int(_lib.load().fm_traj_state_bytes(cap, B_max))


class TrajPass:
    """State of one incremental trajectory re-search pass (Section 4.2.2) of
    B queries: call ``step`` with layer 0, 1, 2, ... as the layers are
    observed; each step returns the Eq. 5 top-k at prefix depth layer + 1."""

    def __init__(self, store: Store, B: int, device=None):
        self.store, self.B = store, int(B)
        self.nbytes = traj_state_bytes(store.cap, self.B)
        if self.nbytes == 0:
            raise ValueError(f"invalid pass size B={B}")
        self.buf = _aligned_bytes(self.nbytes, store.device if device is None else device)

    def step(self, q_layer: torch.Tensor, layer: int, k: int = 1,
             out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None, workspace: Optional[Workspace] = None,
             stream=None):
        """q_layer [B][E] (store dtype): every query's gate probabilities at ``layer``."""
        dev = _dev(self.store)
        if isinstance(q_layer, torch.Tensor):
            q_layer = q_layer.contiguous()
        _need(q_layer, "q_layer", _TORCH[self.store.dtype_code], (self.B, self.store.E), dev)
        if out is None:
            out = (torch.empty((self.B, k), dtype=torch.int32, device=dev),
                   torch.empty((self.B, k), dtype=torch.float32, device=dev))
        idx, score = out
        _need(idx, "out[0] (idx)", torch.int32, (self.B, k), dev)
        _need(score, "out[1] (score)", torch.float32, (self.B, k), dev)
        ws = _ws(self.store, workspace)
        _lib.check(_lib.load().fm_traj_step(self.store.handle, C.c_void_p(self.buf.data_ptr()), self.nbytes,
                                            _ptr(q_layer), int(layer), self.B, k, _ptr(idx), _ptr(score), ws.ptr,
                                            ws.nbytes, _stream(stream)), "fm_traj_step")
        return idx, score


def _ws(store: Store, workspace: Optional[Workspace]) -> Workspace:
    return workspace if workspace is not None else store.ensure_workspace()


def match_trajectory(store: Store, q: torch.Tensor, depth: torch.Tensor, k: int = 1,
                     max_depth: Optional[int] = None, out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                     workspace: Optional[Workspace] = None, stream=None):
    """Eq. 5 search: q [B][L][E] (store dtype), depth [B] int32 -> idx [B][k] int32, score [B][k] float32."""
    dev = _dev(store)
    _need(q, "q", _TORCH[store.dtype_code], (None, store.L, store.E), dev)
    B = q.shape[0]
    _need(depth, "depth", torch.int32, (B,), dev)
    if max_depth is None:
        max_depth = store.L
    if out is None:
        out = (torch.empty((B, k), dtype=torch.int32, device=dev),
               torch.empty((B, k), dtype=torch.float32, device=dev))
    idx, score = out
    _need(idx, "out[0] (idx)", torch.int32, (B, k), dev)
    _need(score, "out[1] (score)", torch.float32, (B, k), dev)
    ws = _ws(store, workspace)
    _lib.check(_lib.load().fm_match_trajectory(store.handle, _ptr(q), _ptr(depth), max_depth, B, k,
                                               _ptr(idx), _ptr(score), ws.ptr, ws.nbytes, _stream(stream)),
               "fm_match_trajectory")
    return idx, score


def match_trajectory_noalloc(store: Store, q: torch.Tensor, depth: torch.Tensor, k: int = 1,
                             max_depth: Optional[int] = None, out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                             stream=None):
    """match_trajectory through the entry point that takes no workspace (the
    library's own device scratch serves as one); ``out`` must be given by
    callers that cannot allocate."""
    dev = _dev(store)
    _need(q, "q", _TORCH[store.dtype_code], (None, store.L, store.E), dev)
    B = q.shape[0]
    _need(depth, "depth", torch.int32, (B,), dev)
    if max_depth is None:
        max_depth = store.L
    if out is None:
        out = (torch.empty((B, k), dtype=torch.int32, device=dev),
               torch.empty((B, k), dtype=torch.float32, device=dev))
    idx, score = out
    _need(idx, "out[0] (idx)", torch.int32, (B, k), dev)
    _need(score, "out[1] (score)", torch.float32, (B, k), dev)
    _lib.check(_lib.load().fm_match_trajectory_noalloc(store.handle, _ptr(q), _ptr(depth), max_depth, B, k,
                                                       _ptr(idx), _ptr(score), _stream(stream)),
               "fm_match_trajectory_noalloc")
    return idx, score


def match_semantic(store: Store, q: torch.Tensor, k: int = 1,
                   out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                   workspace: Optional[Workspace] = None, stream=None):
    """Eq. 4 search: q [B][d_emb] bfloat16 -> idx [B][k] int32, score [B][k] float32."""
    dev = _dev(store)
    _need(q, "q", torch.bfloat16, (None, store.d_emb), dev)
    B = q.shape[0]
    if out is None:
        out = (torch.empty((B, k), dtype=torch.int32, device=dev),
               torch.empty((B, k), dtype=torch.float32, device=dev))
    idx, score = out
    _need(idx, "out[0] (idx)", torch.int32, (B, k), dev)
    _need(score, "out[1] (score)", torch.float32, (B, k), dev)
    ws = _ws(store, workspace)
    _lib.check(_lib.load().fm_match_semantic(store.handle, _ptr(q), B, k, _ptr(idx), _ptr(score), ws.ptr,
                                             ws.nbytes, _stream(stream)), "fm_match_semantic")
    return idx, score


def select_prefetch(store: Store, idx: torch.Tensor, score: torch.Tensor, layer_begin: torch.Tensor,
                    layer_end: torch.Tensor, tau: float = 0.9, k_min: int = 1, k_max: Optional[int] = None,
                    mode: int = FM_TAU_FIXED, blend: int = FM_BLEND_NONE,
                    out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None, stream=None):
    """Eq. 6-8 prefetch sets -> mask [B][L] (int64 holding uint64 bits), count [B][L] uint8."""
    dev = _dev(store)
    _need(idx, "idx", torch.int32, (None, None), dev)
    B, k = idx.shape
    _need(score, "score", torch.float32, (B, k), dev)
    _need(layer_begin, "layer_begin", torch.int32, (B,), dev)
    _need(layer_end, "layer_end", torch.int32, (B,), dev)
    if k_max is None:
        k_max = store.E
    if out is None:
        out = (torch.empty((B, store.L), dtype=torch.int64, device=dev),
               torch.empty((B, store.L), dtype=torch.uint8, device=dev))
    mask, count = out
    _need(mask, "out[0] (mask)", torch.int64, (B, store.L), dev)
    _need(count, "out[1] (count)", torch.uint8, (B, store.L), dev)
    p = SelectParams(mode, tau, k_min, k_max, blend)
    _lib.check(_lib.load().fm_select_prefetch(store.handle, _ptr(idx), _ptr(score), B, k, _ptr(layer_begin),
                                              _ptr(layer_end), C.byref(p), _ptr(mask), _ptr(count),
                                              _stream(stream)), "fm_select_prefetch")
    return mask, count


def _fused_outputs(store: Store, B: int, k: int, layer_begin, layer_end, out, dev):
    _need(layer_begin, "layer_begin", torch.int32, (B,), dev)
    _need(layer_end, "layer_end", torch.int32, (B,), dev)
    if out is None:
        out = (torch.empty((B, k), dtype=torch.int32, device=dev),
               torch.empty((B, k), dtype=torch.float32, device=dev),
               torch.empty((B, store.L), dtype=torch.int64, device=dev),
               torch.empty((B, store.L), dtype=torch.uint8, device=dev))
    idx, score, mask, count = out
    _need(idx, "out[0] (idx)", torch.int32, (B, k), dev)
    _need(score, "out[1] (score)", torch.float32, (B, k), dev)
    _need(mask, "out[2] (mask)", torch.int64, (B, store.L), dev)
    _need(count, "out[3] (count)", torch.uint8, (B, store.L), dev)
    return out


def match_trajectory_select(store: Store, q: torch.Tensor, depth: torch.Tensor, layer_begin: torch.Tensor,
                            layer_end: torch.Tensor, k: int = 1, max_depth: Optional[int] = None, tau: float = 0.9,
                            k_min: int = 1, k_max: Optional[int] = None, mode: int = FM_TAU_FIXED,
                            blend: int = FM_BLEND_NONE, out=None, workspace: Optional[Workspace] = None,
                            stream=None):
    """match_trajectory, then select_prefetch of its rows, in one call -> (idx, score, mask, count)."""
    dev = _dev(store)
    _need(q, "q", _TORCH[store.dtype_code], (None, store.L, store.E), dev)
    B = q.shape[0]
    _need(depth, "depth", torch.int32, (B,), dev)
    if max_depth is None:
        max_depth = store.L
    if k_max is None:
        k_max = store.E
    idx, score, mask, count = out = _fused_outputs(store, B, k, layer_begin, layer_end, out, dev)
    ws = _ws(store, workspace)
    p = SelectParams(mode, tau, k_min, k_max, blend)
    _lib.check(_lib.load().fm_match_trajectory_select(store.handle, _ptr(q), _ptr(depth), max_depth, B, k,
                                                      _ptr(layer_begin), _ptr(layer_end), C.byref(p), _ptr(idx),
                                                      _ptr(score), _ptr(mask), _ptr(count), ws.ptr, ws.nbytes,
                                                      _stream(stream)), "fm_match_trajectory_select")
    return out


def match_semantic_select(store: Store, q: torch.Tensor, layer_begin: torch.Tensor, layer_end: torch.Tensor,
                          k: int = 1, tau: float = 0.9, k_min: int = 1, k_max: Optional[int] = None,
                          mode: int = FM_TAU_FIXED, blend: int = FM_BLEND_NONE, out=None,
                          workspace: Optional[Workspace] = None, stream=None):
    """match_semantic, then select_prefetch of its rows, in one call -> (idx, score, mask, count)."""
    dev = _dev(store)
    _need(q, "q", torch.bfloat16, (None, store.d_emb), dev)
    B = q.shape[0]
    if k_max is None:
        k_max = store.E
    idx, score, mask, count = out = _fused_outputs(store, B, k, layer_begin, layer_end, out, dev)
    ws = _ws(store, workspace)
    p = SelectParams(mode, tau, k_min, k_max, blend)
    _lib.check(_lib.load().fm_match_semantic_select(store.handle, _ptr(q), B, k, _ptr(layer_begin),
                                                    _ptr(layer_end), C.byref(p), _ptr(idx), _ptr(score),
                                                    _ptr(mask), _ptr(count), ws.ptr, ws.nbytes, _stream(stream)),
               "fm_match_semantic_select")
    return out


def priority_order(store: Store, idx: torch.Tensor, score: torch.Tensor, masks: torch.Tensor,
                   l_now: Optional[torch.Tensor] = None, freq: Optional[torch.Tensor] = None,
                   kind: int = FM_PRI_PREFETCH, blend: int = FM_BLEND_NONE, cap: Optional[int] = None,
                   out=None, stream=None):
    """Section 4.5 priorities -> order [B][cap] int32 (l * E + j), pri [B][cap] float32, count [B] int32.
    PREFETCH: masks [B][L] (int64 holding uint64 bits) from select_prefetch, l_now [B] int32.
    EVICT: masks [L] (cached experts), freq [L][E] float32."""
    dev = _dev(store)
    _need(idx, "idx", torch.int32, (None, None), dev)
    B, k = idx.shape
    _need(score, "score", torch.float32, (B, k), dev)
    if isinstance(masks, torch.Tensor):
        masks = masks.contiguous()
    _need(masks, "masks", torch.int64, (B, store.L) if kind == FM_PRI_PREFETCH else (store.L,), dev)
    if kind == FM_PRI_PREFETCH:
        _need(l_now, "l_now", torch.int32, (B,), dev)
    else:
        _need(freq, "freq", torch.float32, (store.L, store.E), dev)
    cap = store.L * store.E if cap is None else int(cap)
    if out is None:
        out = (torch.empty((B, cap), dtype=torch.int32, device=dev),
               torch.empty((B, cap), dtype=torch.float32, device=dev),
               torch.empty((B,), dtype=torch.int32, device=dev))
    order, pri, count = out
    _need(order, "out[0] (order)", torch.int32, (B, cap), dev)
    _need(pri, "out[1] (pri)", torch.float32, (B, cap), dev)
    _need(count, "out[2] (count)", torch.int32, (B,), dev)
    _lib.check(_lib.load().fm_priority_order(store.handle, _ptr(idx), _ptr(score), B, k, blend, kind,
                                             _ptr(masks), _ptr(l_now), _ptr(freq), cap, _ptr(order),
                                             _ptr(pri), _ptr(count), _stream(stream)), "fm_priority_order")
    return order, pri, count


def miss_count(store: Store, q: torch.Tensor, masks: torch.Tensor, K: int, layer_begin: torch.Tensor,
               layer_end: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Section 3 misses: activated experts (top-K of q [B][L][E], store dtype) outside the sets
    masks [B][L] -> [B][L] uint8 for layers in [layer_begin, layer_end)."""
    dev = _dev(store)
    if isinstance(q, torch.Tensor):
        q = q.contiguous()
    _need(q, "q", _TORCH[store.dtype_code], (None, store.L, store.E), dev)
    B = q.shape[0]
    _need(masks, "masks", torch.int64, (B, store.L), dev)
    _need(layer_begin, "layer_begin", torch.int32, (B,), dev)
    _need(layer_end, "layer_end", torch.int32, (B,), dev)
    if out is None:
        out = torch.empty((B, store.L), dtype=torch.uint8, device=dev)
    _need(out, "out", torch.uint8, (B, store.L), dev)
    _lib.check(_lib.load().fm_miss_count(store.handle, _ptr(q), B, int(K), _ptr(masks), _ptr(layer_begin),
                                         _ptr(layer_end), _ptr(out), _stream(stream)), "fm_miss_count")
    return out


def debug_scores(store: Store, q: Optional[torch.Tensor] = None, depth: Optional[torch.Tensor] = None,
                 q_sem: Optional[torch.Tensor] = None, max_depth: Optional[int] = None,
                 workspace: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """Dense float32 scores [B][size] from the same kernels as the match calls (test support)."""
    dev = _dev(store)
    if q is not None:
        _need(q, "q", _TORCH[store.dtype_code], (None, store.L, store.E), dev)
        _need(depth, "depth", torch.int32, (q.shape[0],), dev)
    if q_sem is not None:
        _need(q_sem, "q_sem", torch.bfloat16, (None, store.d_emb), dev)
    B = (q if q is not None else q_sem).shape[0]
    n = store.size
    out = torch.full((B, max(n, 1)), float("nan"), dtype=torch.float32, device=dev)
    ws = _ws(store, workspace)
    _lib.check(_lib.load().fm_debug_scores(store.handle, _ptr(q), _ptr(depth),
                                           max_depth if max_depth is not None else store.L, _ptr(q_sem), B,
                                           _ptr(out), ws.ptr, ws.nbytes, _stream(stream)), "fm_debug_scores")
    return out[:, :n]
