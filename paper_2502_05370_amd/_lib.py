"""ctypes declarations of the C ABI in include/finemoe_map.h.

Loads ``libfinemoe_map.so`` from this package directory (or, for the
sanitizer tests, the library file FM_LIBRARY names).  There is no fallback:
if the library is missing the import fails with a message saying how to
build it.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("FM_LIBRARY") or os.path.join(HERE, "libfinemoe_map.so")

FM_OK, FM_ERR_INVALID, FM_ERR_UNSUPPORTED, FM_ERR_FULL, FM_ERR_HIP, FM_ERR_DEVICE = range(6)
FM_F32, FM_BF16 = 0, 1
FM_TAU_FIXED, FM_TAU_DYNAMIC = 0, 1
FM_BLEND_NONE, FM_BLEND_SCORE = 0, 1
FM_PRI_PREFETCH, FM_PRI_EVICT = 0, 1
FM_FLAG_DEPTH_CLAMPED = 0x1
FM_FLAG_INDEX_RANGE = 0x2
FM_FLAG_STATE_STALE = 0x4
FM_FLAG_VALUE_RANGE = 0x8

STATUS_NAMES = {0: "FM_OK", 1: "FM_ERR_INVALID", 2: "FM_ERR_UNSUPPORTED", 3: "FM_ERR_FULL",
                4: "FM_ERR_HIP", 5: "FM_ERR_DEVICE"}

# Every symbol the header declares, with (restype, argtypes).
_vp = C.c_void_p
_i32 = C.c_int32
_sz = C.c_size_t


class StoreDesc(C.Structure):
    _fields_ = [("cap", C.c_int32), ("L", C.c_int32), ("E", C.c_int32), ("d_emb", C.c_int32),
                ("map_dtype", C.c_int), ("buffer", C.c_void_p), ("buffer_bytes", C.c_size_t)]


class SelectParams(C.Structure):
    _fields_ = [("mode", C.c_int), ("tau", C.c_float), ("k_min", C.c_int32), ("k_max", C.c_int32),
                ("blend", C.c_int)]


SIGNATURES = {
    "fm_map_bytes": (_sz, [_i32, _i32, _i32, C.c_int]),
    "fm_store_bytes": (_sz, [_i32, _i32, _i32, _i32, C.c_int]),
    "fm_workspace_bytes": (_sz, [_i32, _i32, _i32, C.c_int, _i32, _i32]),
    "fm_store_build": (C.c_int, [C.POINTER(_vp), C.POINTER(StoreDesc)]),
    "fm_store_insert": (C.c_int, [_vp, _vp, _vp, _i32, _vp, _vp]),
    "fm_dedup_scratch_bytes": (_sz, [_i32, _i32]),
    "fm_store_insert_dedup": (C.c_int, [_vp, _vp, _vp, _i32, _i32, _vp, _vp, _sz, _vp, _sz, _vp]),
    "fm_store_size": (C.c_int, [_vp, C.POINTER(_i32)]),
    "fm_store_check": (C.c_int, [_vp, _vp, C.POINTER(C.c_uint32)]),
    "fm_store_destroy": (C.c_int, [_vp]),
    "fm_match_semantic": (C.c_int, [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _sz, _vp]),
    "fm_match_trajectory": (C.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp, _sz, _vp]),
    "fm_match_trajectory_noalloc": (C.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp]),
    "fm_select_prefetch": (C.c_int, [_vp, _vp, _vp, _i32, _i32, _vp, _vp, C.POINTER(SelectParams), _vp, _vp, _vp]),
    "fm_match_semantic_select": (C.c_int, [_vp, _vp, _i32, _i32, _vp, _vp, C.POINTER(SelectParams), _vp, _vp, _vp,
                                           _vp, _vp, _sz, _vp]),
    "fm_match_trajectory_select": (C.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp, C.POINTER(SelectParams),
                                             _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "fm_miss_count": (C.c_int, [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "fm_priority_order": (C.c_int, [_vp, _vp, _vp, _i32, _i32, C.c_int, C.c_int, _vp, _vp, _vp, _i32, _vp, _vp, _vp,
                                    _vp]),
    "fm_traj_state_bytes": (_sz, [_i32, _i32]),
    "fm_traj_step": (C.c_int, [_vp, _vp, _sz, _vp, _i32, _i32, _i32, _vp, _vp, _vp, _sz, _vp]),
    "fm_debug_scores": (C.c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _sz, _vp]),
    "fm_debug_scan_events": (C.c_int, [_vp, _vp]),
    "fm_last_error": (C.c_char_p, []),
    "fm_version": (C.c_int32, []),
}


class FmError(RuntimeError):
    def __init__(self, status: int, call: str, message: str):
        self.status = status
        super().__init__(f"{call} -> {STATUS_NAMES.get(status, status)}: {message}")


_LIB = None


def load() -> C.CDLL:
    """Load the built library (once) and declare every entry point."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2502_05370_amd/build.py` "
            "(hipcc for gfx950); there is no CPU fallback")
    lib = C.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def check(status: int, call: str) -> None:
    if status != FM_OK:
        msg = load().fm_last_error()
        raise FmError(status, call, msg.decode() if msg else "")
