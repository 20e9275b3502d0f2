"""The C ABI on the host: symbols, workspace queries and argument validation.

No call here reaches the device: every case returns from host-side
validation before any HIP call is made.
"""
import ctypes
import os
import re

import pytest

from paper_2608_13144_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lipcache.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="liblipcache.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lipcache_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound():
    lib = L.load()
    names = declared_functions()
    assert len(names) >= 11
    for name in names:
        assert hasattr(lib, name), name
        assert name in L.SIGNATURES, f"binding lacks {name}"
    assert lib.lipcache_abi_version() == 7


def test_status_strings():
    for s in range(8):
        assert L.status_string(s)
    assert "degenerate" in L.status_string(L.EDEGENERATE)


def test_workspace_queries():
    lib = L.load()
    assert lib.lipcache_spectral_norm_workspace_bytes(200, 256) >= 200 * 200 * 8
    assert lib.lipcache_spectral_norm_workspace_bytes(300, 64) >= 64 * 64 * 8
    assert lib.lipcache_certify_workspace_bytes(200, 256, 0) >= 200 * 256 * 8
    assert lib.lipcache_certify_workspace_bytes(200, 256, L.RADIUS_TIGHT) >= 200 * 256 * 8 + 200 * 200 * 8
    assert lib.lipcache_lookup_workspace_bytes(32768, 1 << 20, 256, L.F16) >= 32768 * 16
    assert lib.lipcache_insert_workspace_bytes(65536) >= 2 * 64 * 8


FAKE = ctypes.c_void_p(0x100000)  # never dereferenced: validation fails first


def _cache(**kw):
    c = L.LipcacheCache(FAKE.value, None, FAKE.value, FAKE.value, FAKE.value, 0, 16, 64, L.F32)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_spectral_norm_validation():
    lib = L.load()
    s = ctypes.c_double()
    it = ctypes.c_int32()
    ws = ctypes.create_string_buffer(1 << 16)
    assert lib.lipcache_spectral_norm(None, 4, 4, 10, 1e-12, ctypes.byref(s), ctypes.byref(it), ws, 1 << 16, None) == L.EINVAL
    assert lib.lipcache_spectral_norm(FAKE, 0, 4, 10, 1e-12, ctypes.byref(s), None, ws, 1 << 16, None) == L.EINVAL
    assert lib.lipcache_spectral_norm(FAKE, 4, 4, 0, 1e-12, ctypes.byref(s), None, ws, 1 << 16, None) == L.EINVAL
    assert lib.lipcache_spectral_norm(FAKE, 4, 4, 10, 0.0, ctypes.byref(s), None, ws, 1 << 16, None) == L.EINVAL
    assert lib.lipcache_spectral_norm(FAKE, 4, 4, 10, 1e-12, None, None, ws, 1 << 16, None) == L.EINVAL
    assert lib.lipcache_spectral_norm(FAKE, 2000, 2000, 10, 1e-12, ctypes.byref(s), None, ws, 1 << 16, None) == L.EUNSUPPORTED
    assert lib.lipcache_spectral_norm(FAKE, 4, 4, 10, 1e-12, ctypes.byref(s), None, None, 0, None) == L.EWORKSPACE


def test_certify_validation():
    lib = L.load()
    args = dict(z=FAKE, N=10, d=64, W=FAKE, b=None, C=10, sigma=1.0, mode=0, store=0,
                label=FAKE, r=FAKE, margin=None, norm2=None, ws=FAKE, wsb=1 << 20)

    def call(**over):
        a = dict(args, **over)
        return lib.lipcache_certify(a["z"], a["N"], a["d"], a["W"], a["b"], a["C"], a["sigma"], a["mode"],
                                    a["store"], a["label"], a["r"], a["margin"], a["norm2"], a["ws"], a["wsb"], None)
    assert call(d=33) == L.EINVAL
    assert call(d=16) == L.EINVAL
    assert call(d=2048) == L.EINVAL
    assert call(C=1) == L.EINVAL
    assert call(N=-1) == L.EINVAL
    assert call(sigma=0.0) == L.EINVAL
    assert call(sigma=-1.0) == L.EINVAL
    assert call(store=7) == L.EINVAL
    assert call(mode=9) == L.EINVAL
    assert call(label=None) == L.EINVAL
    assert call(z=ctypes.c_void_p(0x100004)) == L.EINVAL  # misaligned
    assert call(mode=L.RADIUS_TIGHT, wsb=10 * 64 * 8 + 256) == L.EWORKSPACE   # no room for the C x C table
    assert call(ws=None) == L.EWORKSPACE
    assert call(wsb=16) == L.EWORKSPACE
    assert call(ws=ctypes.c_void_p(0x100040)) == L.EWORKSPACE  # not 256-aligned


def test_lookup_validation():
    lib = L.load()

    def call(c, B=8, prec=L.F16, zq=FAKE, label=FAKE, ws=FAKE, wsb=1 << 24):
        return lib.lipcache_lookup(ctypes.byref(c) if c is not None else None, zq, B, prec, label, None, None,
                                   None, None, ws, wsb, None)
    assert call(None) == L.EINVAL
    assert call(_cache(d=48)) == L.EINVAL
    assert call(_cache(store_dtype=3)) == L.EINVAL
    assert call(_cache(n=20)) == L.EINVAL            # n > capacity
    assert call(_cache(z=None)) == L.EINVAL
    assert call(_cache(), B=-1) == L.EINVAL
    assert call(_cache(), prec=5) == L.EINVAL
    assert call(_cache(), prec=L.BF16) == L.EINVAL   # a store type, not a filter precision
    assert call(_cache(), zq=None) == L.EINVAL
    assert call(_cache(), label=None) == L.EINVAL
    assert call(_cache(d=1024), prec=L.F32) == L.EUNSUPPORTED
    assert call(_cache(), ws=None) == L.EWORKSPACE
    assert call(_cache(), wsb=64) == L.EWORKSPACE
    # lookup options: only LIPCACHE_LOOKUP_PRUNE, on a filter precision
    assert call(_cache(), prec=L.F16 | 0x200) == L.EINVAL
    assert call(_cache(), prec=L.BF16 | L.LOOKUP_PRUNE) == L.EINVAL
    assert call(_cache(d=1024), prec=L.F32 | L.LOOKUP_PRUNE) == L.EUNSUPPORTED
    assert call(_cache(), prec=L.F16 | L.LOOKUP_PRUNE, ws=None) == L.EWORKSPACE


def test_pruned_lookup_workspace():
    """The pruned lookup's workspace adds its prefix thresholds: 4 bytes per
    query and per entry (plus padding), and the plain size is unchanged."""
    lib = L.load()
    B, n = 32768, 1 << 20
    plain = lib.lipcache_lookup_workspace_bytes(B, n, 256, L.F16)
    pruned = lib.lipcache_lookup_workspace_bytes(B, n, 256, L.F16 | L.LOOKUP_PRUNE)
    assert pruned >= plain + 4 * B + 4 * n
    assert pruned <= plain + 4 * B + 4 * (n + 2048) + 512
    assert lib.lipcache_lookup_workspace_bytes(B, n, 256, L.F32) == plain


def test_lookup_prunes_rule():
    """Which caches the pruned path serves (host only): the float16 filter
    with an image, 64 <= d <= 512, n >= 32,768; everything else runs the full
    contraction, and a request without the option never prunes."""
    lib = L.load()

    def prunes(prec=L.F16 | L.LOOKUP_PRUNE, **kw):
        base = dict(zimg=FAKE.value, n=40000, capacity=50000, d=256)
        base.update(kw)
        return lib.lipcache_lookup_prunes(ctypes.byref(_cache(**base)), prec)
    assert prunes() == 1
    assert prunes(d=64) == 1 and prunes(d=512) == 1 and prunes(d=96) == 1
    assert prunes(n=32768) == 1 and prunes(n=32767) == 0
    assert prunes(d=32) == 0 and prunes(d=1024) == 0
    assert prunes(zimg=None) == 0
    assert prunes(prec=L.F16) == 0
    assert prunes(prec=L.F32 | L.LOOKUP_PRUNE) == 0
    assert prunes(prec=L.BF16 | L.LOOKUP_PRUNE) == 0
    assert prunes(store_dtype=L.BF16) == 1
    assert lib.lipcache_lookup_prunes(None, L.F16 | L.LOOKUP_PRUNE) == 0


def test_lookup_noalloc_validation():
    """The allocation-free lookup validates like lipcache_lookup and refuses,
    before any device work, a lookup whose workspace exceeds its static array."""
    lib = L.load()

    def call(c, B=8, prec=L.F16, zq=FAKE, label=FAKE):
        return lib.lipcache_lookup_noalloc(ctypes.byref(c) if c is not None else None, zq, B, prec, label, None,
                                           None, None, None, None)
    assert call(None) == L.EINVAL
    assert call(_cache(d=48)) == L.EINVAL
    assert call(_cache(), B=-1) == L.EINVAL
    assert call(_cache(), prec=L.BF16) == L.EINVAL
    assert call(_cache(), label=None) == L.EINVAL
    assert call(_cache(d=1024), prec=L.F32) == L.EUNSUPPORTED
    # the largest n that fits with B = 65,536, and one row more
    B = 65536
    n = 4_500_000
    assert lib.lipcache_lookup_workspace_bytes(B, n, 64, L.F16) <= L.NOALLOC_SCRATCH_BYTES
    big = 1 << 23
    assert lib.lipcache_lookup_workspace_bytes(B, big, 64, L.F16) > L.NOALLOC_SCRATCH_BYTES
    assert call(_cache(n=big, capacity=big), B=B) == L.EWORKSPACE
    assert call(_cache(n=16, capacity=16), B=1 << 24) == L.EWORKSPACE


def test_insert_validation():
    lib = L.load()

    def call(c, k=4, z=FAKE, lab=FAKE, r=FAKE, ws=FAKE, wsb=1 << 20):
        n = ctypes.c_int64(-5)
        st = lib.lipcache_insert(ctypes.byref(c) if c is not None else None, z, lab, r, None, k,
                                 ctypes.byref(n), ws, wsb, None)
        return st, n.value
    assert call(None)[0] == L.EINVAL
    assert call(_cache(), k=-1)[0] == L.EINVAL
    assert call(_cache(d=40))[0] == L.EINVAL
    assert call(_cache(), z=None)[0] == L.EINVAL
    assert call(_cache(), z=ctypes.c_void_p(0x100008))[0] == L.EINVAL   # rows move as 16-byte vectors
    assert call(_cache(), r=None)[0] == L.EINVAL
    assert call(_cache(n=-1))[0] == L.EINVAL
    assert call(_cache(), ws=None)[0] == L.EWORKSPACE
    st, n = call(_cache(), k=0)
    assert st == L.OK and n == 0


def _index(K=4, n_indexed=10, **kw):
    srt = _cache(n=n_indexed, capacity=16)
    ix = L.LipcacheIndex(srt, FAKE.value, FAKE.value, FAKE.value, FAKE.value, K, n_indexed)
    for k, v in kw.items():
        setattr(ix, k, v)
    return ix


def test_index_build_validation():
    lib = L.load()

    def call(c, K=4, iters=2, ix="default", ws=FAKE, wsb=1 << 30):
        ix = _index() if ix == "default" else ix
        return lib.lipcache_index_build(ctypes.byref(c) if c is not None else None, K, iters,
                                        ctypes.byref(ix) if ix is not None else None, ws, wsb, None)
    assert call(None) == L.EINVAL
    assert call(_cache(n=10), ix=None) == L.EINVAL
    assert call(_cache(n=0)) == L.EINVAL                     # nothing to index
    assert call(_cache(n=10), K=0) == L.EINVAL
    assert call(_cache(n=10), K=11) == L.EINVAL              # K > n
    assert call(_cache(n=10), iters=-1) == L.EINVAL
    assert call(_cache(n=10, d=40)) == L.EINVAL
    small = _index()
    small.sorted.capacity = 8
    assert call(_cache(n=10), ix=small) == L.EINVAL          # sorted copy cannot hold the rows
    assert call(_cache(n=10), ix=_index(centers=0x100004)) == L.EINVAL
    assert call(_cache(n=10), ix=_index(perm=None)) == L.EINVAL
    assert call(_cache(n=10), ws=None) == L.EWORKSPACE
    assert call(_cache(n=10), wsb=64) == L.EWORKSPACE
    assert lib.lipcache_index_build_workspace_bytes(1 << 20, 256, 1024) >= (1 << 20) * 4 + 1024 * 256 * 8


def test_lookup_indexed_validation():
    lib = L.load()

    def call(c, ix, B=8, prec=L.F16, ws=FAKE, wsb=1 << 30):
        pairs = ctypes.c_int64(-1)
        st = lib.lipcache_lookup_indexed(ctypes.byref(c), ctypes.byref(ix) if ix is not None else None, FAKE, B,
                                         prec, FAKE, None, None, None, None, ctypes.byref(pairs), ws, wsb, None)
        return st
    c = _cache(n=12)
    assert call(c, None) == L.EINVAL
    assert call(c, _index(K=0)) == L.EINVAL
    assert call(c, _index(n_indexed=13)) == L.EINVAL         # more rows indexed than the cache holds
    bad = _index()
    bad.sorted.n = 9
    assert call(c, bad) == L.EINVAL                          # sorted copy out of step with the index
    bad = _index()
    bad.sorted.d = 128
    assert call(c, bad) == L.EINVAL
    assert call(c, _index(centers=0x100004)) == L.EINVAL
    assert call(_cache(n=12, zimg=FAKE.value), _index()) == L.EINVAL   # image on one side only
    assert call(c, _index(), B=-1) == L.EINVAL
    assert call(c, _index(), prec=7) == L.EINVAL
    assert call(c, _index(), ws=None) == L.EWORKSPACE
    assert call(c, _index(), wsb=64) == L.EWORKSPACE
    assert lib.lipcache_lookup_indexed_workspace_bytes(32768, 1 << 20, 256, 1024, 1 << 20) >= 32768 * 1024 // 8



def test_construct_validation():
    lib = L.load()

    def call(c, N=4, strategy=L.SELECT_RADIUS_DEDUP, budget=8, per_class=0, n_classes=0, z=FAKE, lab=FAKE,
             r=FAKE, prio=None, ws=FAKE, wsb=None):
        if wsb is None:
            wsb = lib.lipcache_construct_workspace_bytes(ctypes.byref(c), max(N, 0), n_classes, budget) if c else 0
        appended = ctypes.c_int64(-5)
        st = lib.lipcache_construct(ctypes.byref(c) if c is not None else None, z, lab, r, None, prio, N,
                                    strategy, budget, per_class, n_classes, None, ctypes.byref(appended), ws,
                                    wsb, None)
        return st, appended.value
    assert call(None)[0] == L.EINVAL
    assert call(_cache(), N=-1)[0] == L.EINVAL
    assert call(_cache(), N=1 << 31)[0] == L.EUNSUPPORTED      # candidate indices are 32-bit
    assert call(_cache(d=48))[0] == L.EINVAL
    assert call(_cache(store_dtype=3))[0] == L.EINVAL
    assert call(_cache(n=17))[0] == L.EINVAL                   # n > capacity
    assert call(_cache(r=None))[0] == L.EINVAL
    assert call(_cache(), strategy=7)[0] == L.EINVAL
    assert call(_cache(), z=None)[0] == L.EINVAL
    assert call(_cache(), r=None)[0] == L.EINVAL
    assert call(_cache(), z=ctypes.c_void_p(0x100008))[0] == L.EINVAL  # rows move as 16-byte vectors
    assert call(_cache(), strategy=L.SELECT_PRIORITY)[0] == L.EINVAL   # priority keys missing
    assert call(_cache(), per_class=-1)[0] == L.EINVAL
    assert call(_cache(), per_class=2, n_classes=0)[0] == L.EINVAL
    assert call(_cache(), per_class=2, n_classes=16385)[0] == L.EINVAL
    assert call(_cache(n=10), budget=7)[0] == L.ECAPACITY      # only 6 free rows
    assert call(_cache(), ws=None)[0] == L.EWORKSPACE
    assert call(_cache(), wsb=64)[0] == L.EWORKSPACE
    assert call(_cache(), budget=0) == (L.OK, 0)               # nothing to append: no launch
    assert call(_cache(), N=0) == (L.OK, 0)


def test_boundary_radius_validation():
    lib = L.load()

    def call(c, mode=L.BOUNDARY_SCALED, factor=0.5, n_classes=0, out=FAKE, ws=None, wsb=0):
        return lib.lipcache_boundary_radius(ctypes.byref(c) if c is not None else None, mode, factor, n_classes,
                                            out, ws, wsb, None)
    assert call(None) == L.EINVAL
    assert call(_cache(n=4), out=None) == L.EINVAL
    assert call(_cache(n=4, d=48)) == L.EINVAL
    assert call(_cache(n=4, store_dtype=3)) == L.EINVAL
    assert call(_cache(n=17)) == L.EINVAL                      # n > capacity
    assert call(_cache(n=4, label=None)) == L.EINVAL
    assert call(_cache(n=4), mode=9) == L.EINVAL
    for bad in (-1.0, float("nan"), float("inf")):
        assert call(_cache(n=4), factor=bad) == L.EINVAL
    assert call(_cache(n=4), mode=L.BOUNDARY_INTERCLASS, n_classes=0) == L.EINVAL
    assert call(_cache(n=4), mode=L.BOUNDARY_INTERCLASS, n_classes=65537) == L.EINVAL
    assert call(_cache(n=4), mode=L.BOUNDARY_INTERCLASS, n_classes=10) == L.EWORKSPACE
    need = lib.lipcache_boundary_radius_workspace_bytes(64, 10)
    assert need >= 10 * 64 * 8
    assert call(_cache(n=4), mode=L.BOUNDARY_INTERCLASS, n_classes=10, ws=FAKE, wsb=need - 1) == L.EWORKSPACE
    assert call(_cache(n=0)) == L.OK                           # empty cache: no launch
    assert call(_cache(n=0), mode=L.BOUNDARY_INTERCLASS, n_classes=10, ws=FAKE, wsb=need) == L.OK


def test_consistency_validation():
    lib = L.load()
    assert lib.lipcache_consistency(FAKE, FAKE, -1, FAKE, None) == L.EINVAL
    assert lib.lipcache_consistency(FAKE, FAKE, 8, None, None) == L.EINVAL
    assert lib.lipcache_consistency(None, FAKE, 8, FAKE, None) == L.EINVAL
    assert lib.lipcache_consistency(FAKE, None, 8, FAKE, None) == L.EINVAL


def test_filter_dump_validation():
    lib = L.load()

    def call(c, B=8, prec=L.F16, g=FAKE, cand=FAKE, ws=FAKE, wsb=1 << 30):
        return lib.lipcache_lookup_filter_dump(ctypes.byref(c) if c is not None else None, FAKE, B, prec, g, cand,
                                               ws, wsb, None)
    assert call(None) == L.EINVAL
    assert call(_cache(n=4, d=48)) == L.EINVAL
    assert call(_cache(n=4), B=-1) == L.EINVAL
    assert call(_cache(n=4), prec=5) == L.EINVAL
    assert call(_cache(n=4), g=None) == L.EINVAL
    assert call(_cache(n=4), cand=None) == L.EINVAL
    big = _cache(n=1 << 20, capacity=1 << 20)
    assert call(big, B=128) == L.EINVAL                        # B * n above 2^26
    assert call(_cache(n=4), ws=None) == L.EWORKSPACE
    assert call(_cache(n=4), wsb=64) == L.EWORKSPACE

def test_binding_refuses_without_library(tmp_path):
    saved = L._LIB
    try:
        L._LIB = None
        with pytest.raises(RuntimeError, match="not built"):
            L.load(str(tmp_path / "missing.so"))
    finally:
        L._LIB = saved
