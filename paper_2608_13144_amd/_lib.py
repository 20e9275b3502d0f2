"""ctypes view of liblipcache.so (the C ABI declared in include/lipcache.h).

Argument marshalling only.  Loading fails loudly when the library has not
been built; there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblipcache.so")

OK, EINVAL, EDEGENERATE, ENOCONV, ECAPACITY, EUNSUPPORTED, EWORKSPACE, EHIP = range(8)
F32, BF16, F16 = 0, 1, 2
LOOKUP_PRUNE = 0x100
RADIUS_CONSERVATIVE, RADIUS_TIGHT = 0, 1
SELECT_RADIUS_DEDUP, SELECT_PRIORITY, SELECT_KCENTER = 0, 1, 2
BOUNDARY_SCALED, BOUNDARY_GLOBAL, BOUNDARY_INTERCLASS = 0, 1, 2
MISS = -1
STAT_HITS, STAT_RECHECKED, STAT_BAND_PAIRS, STAT_BAND_QUERIES = range(4)
NOALLOC_SCRATCH_BYTES = 32 << 20

# Every function the header declares, with (restype, argtypes).
_vp, _i32, _i64, _f64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_size_t


class LipcacheCache(ctypes.Structure):
    """Mirror of ``lipcache_cache``."""

    _fields_ = [
        ("z", ctypes.c_void_p),
        ("zimg", ctypes.c_void_p),
        ("r", ctypes.c_void_p),
        ("label", ctypes.c_void_p),
        ("norm2", ctypes.c_void_p),
        ("n", ctypes.c_int64),
        ("capacity", ctypes.c_int64),
        ("d", ctypes.c_int32),
        ("store_dtype", ctypes.c_int32),
    ]


_PCACHE = ctypes.POINTER(LipcacheCache)


class LipcacheIndex(ctypes.Structure):
    """Mirror of ``lipcache_index``."""

    _fields_ = [
        ("sorted", LipcacheCache),
        ("perm", ctypes.c_void_p),
        ("offsets", ctypes.c_void_p),
        ("centers", ctypes.c_void_p),
        ("bound", ctypes.c_void_p),
        ("K", ctypes.c_int32),
        ("n_indexed", ctypes.c_int64),
    ]


_PINDEX = ctypes.POINTER(LipcacheIndex)

SIGNATURES = {
    "lipcache_spectral_norm": (_i32, [_vp, _i32, _i32, _i32, _f64, ctypes.POINTER(_f64), ctypes.POINTER(_i32),
                                      _vp, _sz, _vp]),
    "lipcache_spectral_norm_workspace_bytes": (_sz, [_i32, _i32]),
    "lipcache_certify": (_i32, [_vp, _i64, _i32, _vp, _vp, _i32, _f64, _i32, _i32, _vp, _vp, _vp, _vp,
                                _vp, _sz, _vp]),
    "lipcache_certify_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "lipcache_lookup": (_i32, [_PCACHE, _vp, _i64, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "lipcache_lookup_noalloc": (_i32, [_PCACHE, _vp, _i64, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "lipcache_lookup_prunes": (_i32, [_PCACHE, _i32]),
    "lipcache_lookup_workspace_bytes": (_sz, [_i64, _i64, _i32, _i32]),
    "lipcache_insert": (_i32, [_PCACHE, _vp, _vp, _vp, _vp, _i64, ctypes.POINTER(_i64), _vp, _sz, _vp]),
    "lipcache_insert_workspace_bytes": (_sz, [_i64]),
    "lipcache_lookup_filter_dump": (_i32, [_PCACHE, _vp, _i64, _i32, _vp, _vp, _vp, _sz, _vp]),
    "lipcache_construct": (_i32, [_PCACHE, _vp, _vp, _vp, _vp, _vp, _i64, _i32, _i64, _i32, _i32, _vp,
                                  ctypes.POINTER(_i64), _vp, _sz, _vp]),
    "lipcache_construct_workspace_bytes": (_sz, [_PCACHE, _i64, _i32, _i64]),
    "lipcache_boundary_radius": (_i32, [_PCACHE, _i32, _f64, _i32, _vp, _vp, _sz, _vp]),
    "lipcache_boundary_radius_workspace_bytes": (_sz, [_i32, _i32]),
    "lipcache_consistency": (_i32, [_vp, _vp, _i64, _vp, _vp]),
    "lipcache_index_build": (_i32, [_PCACHE, _i32, _i32, _PINDEX, _vp, _sz, _vp]),
    "lipcache_index_build_workspace_bytes": (_sz, [_i64, _i32, _i32]),
    "lipcache_lookup_indexed": (_i32, [_PCACHE, _PINDEX, _vp, _i64, _i32, _vp, _vp, _vp, _vp, _vp,
                                       ctypes.POINTER(_i64), _vp, _sz, _vp]),
    "lipcache_lookup_indexed_workspace_bytes": (_sz, [_i64, _i64, _i32, _i32, _i64]),
    "lipcache_status_string": (ctypes.c_char_p, [_i32]),
    "lipcache_abi_version": (_i32, []),
}

_LIB = None


class LipcacheError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {status_string(status)} (status {status})")
        self.status = status


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the library once; raises if it is missing (no fallback)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run __graft_entry__.build() (hipcc, gfx950)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def status_string(status: int) -> str:
    return load().lipcache_status_string(int(status)).decode()


def check(fn: str, status: int, allow=(OK,)) -> int:
    if status not in allow:
        raise LipcacheError(fn, status)
    return status
