"""MI355X-native certified feature cache (LipCache's certified cache path).

The compute path is the HIP library ``liblipcache.so`` (C ABI in
include/lipcache.h).  Submodules: ``api`` (torch binding), ``_lib`` (ctypes
view of the library), ``workload`` (seeded synthetic inputs), ``build``
(hipcc build of the library).
"""
from ._lib import MISS, LipcacheError  # noqa: F401

__all__ = ["MISS", "LipcacheError"]
