"""Torch-facing binding of the certified cache library.

PyTorch provides device memory and the current HIP stream; every step of the
path runs in the HIP kernels behind ``liblipcache.so``.  The functions mirror
the C ABI names (``lipcache_spectral_norm`` -> ``spectral_norm`` ...).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import torch

from . import _lib as L

_STORE = {"f32": L.F32, "bf16": L.BF16}
_PRECISION = {"f32": L.F32, "f16": L.F16}
_RADIUS = {"conservative": L.RADIUS_CONSERVATIVE, "tight": L.RADIUS_TIGHT}
_SELECT = {"radius_dedup": L.SELECT_RADIUS_DEDUP, "priority": L.SELECT_PRIORITY, "kcenter": L.SELECT_KCENTER}
_BOUNDARY = {"scaled": L.BOUNDARY_SCALED, "global": L.BOUNDARY_GLOBAL, "interclass": L.BOUNDARY_INTERCLASS}


def _p(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need_cuda(t: torch.Tensor, name: str, dtype: torch.dtype, ndim: int | None = None) -> None:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions")


def workspace(nbytes: int, device: torch.device) -> torch.Tensor:
    """Scratch buffer from torch's allocator (block starts are 512-byte aligned)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


@dataclass
class SpectralNorm:
    sigma: float
    iterations: int
    converged: bool


def spectral_norm(W: torch.Tensor, max_iters: int = 20000, rel_tol: float = 1e-13) -> SpectralNorm:
    """lipcache_spectral_norm: sigma_max(W) by float64 power iteration (sync)."""
    _need_cuda(W, "W", torch.float32, 2)
    lib = L.load()
    C, d = W.shape
    ws = workspace(lib.lipcache_spectral_norm_workspace_bytes(C, d), W.device)
    sigma = ctypes.c_double(0.0)
    iters = ctypes.c_int32(0)
    st = lib.lipcache_spectral_norm(_p(W), C, d, int(max_iters), float(rel_tol), ctypes.byref(sigma),
                                    ctypes.byref(iters), _p(ws), ws.numel(), _stream(W.device))
    L.check("lipcache_spectral_norm", st, allow=(L.OK, L.ENOCONV))
    return SpectralNorm(sigma.value, iters.value, st == L.OK)


@dataclass
class Certified:
    label: torch.Tensor          # int32 [N]
    r: torch.Tensor              # float32 [N]
    margin: torch.Tensor | None  # float32 [N]
    norm2: torch.Tensor | None   # float32 [N]


def certify(z: torch.Tensor, W: torch.Tensor, b: torch.Tensor | None, sigma: float, store: str = "f32",
            radius_mode: str = "conservative", want_margin: bool = False,
            want_norm2: bool = False) -> Certified:
    """lipcache_certify: labels, margins and certified radii of the rows of z (async)."""
    _need_cuda(z, "z", torch.float32, 2)
    _need_cuda(W, "W", torch.float32, 2)
    if b is not None:
        _need_cuda(b, "b", torch.float32, 1)
    lib = L.load()
    N, d = z.shape
    C = W.shape[0]
    dev = z.device
    label = torch.empty(N, dtype=torch.int32, device=dev)
    r = torch.empty(N, dtype=torch.float32, device=dev)
    margin = torch.empty(N, dtype=torch.float32, device=dev) if want_margin else None
    norm2 = torch.empty(N, dtype=torch.float32, device=dev) if want_norm2 else None
    mode = _RADIUS[radius_mode]
    ws = workspace(lib.lipcache_certify_workspace_bytes(C, d, mode), dev)
    st = lib.lipcache_certify(_p(z), N, d, _p(W), _p(b), C, float(sigma), mode, _STORE[store], _p(label),
                              _p(r), _p(margin), _p(norm2), _p(ws), ws.numel(), _stream(dev))
    L.check("lipcache_certify", st)
    return Certified(label, r, margin, norm2)


@dataclass
class LookupResult:
    label: torch.Tensor           # int32 [B], MISS on a miss
    index: torch.Tensor | None    # int64 [B], -1 on a miss
    dist2: torch.Tensor | None    # float32 [B], +inf on a miss
    stats: torch.Tensor           # int64 [4]: hits, re-checked pairs, band pairs, band queries
    band: torch.Tensor | None     # uint8 [B]


class LipCache:
    """The feature cache C = {(z_i, y~_i, r_i)} in device memory (caller-owned tensors)."""

    def __init__(self, d: int, capacity: int, store: str = "f32", device: str | torch.device = "cuda",
                 image: bool = True):
        """``image``: also keep the float16 image of the stored features that
        the f16 filter streams (costs 2 bytes per element; without it the f16
        lookup converts the rows on the fly)."""
        self.d = int(d)
        self.capacity = int(capacity)
        self.store = store
        self.device = torch.device(device)
        zdt = torch.float32 if store == "f32" else torch.bfloat16
        self.z = torch.empty((self.capacity, self.d), dtype=zdt, device=self.device)
        self.zimg = (torch.empty((self.capacity, self.d), dtype=torch.float16, device=self.device)
                     if image else None)
        self.r = torch.empty(self.capacity, dtype=torch.float32, device=self.device)
        self.label = torch.empty(self.capacity, dtype=torch.int32, device=self.device)
        self.norm2 = torch.empty(self.capacity, dtype=torch.float32, device=self.device)
        self.n = 0
        self._ws = None

    def cstruct(self) -> L.LipcacheCache:
        return L.LipcacheCache(self.z.data_ptr(), None if self.zimg is None else self.zimg.data_ptr(),
                               self.r.data_ptr(), self.label.data_ptr(), self.norm2.data_ptr(), self.n,
                               self.capacity, self.d, _STORE[self.store])

    def _workspace(self, nbytes: int) -> torch.Tensor:
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = workspace(nbytes, self.device)
        return self._ws

    def insert(self, z_src: torch.Tensor, label_src: torch.Tensor, r_src: torch.Tensor,
               miss_selector: torch.Tensor | None = None) -> int:
        """lipcache_insert: append selected rows (ascending), all-or-nothing (sync)."""
        _need_cuda(z_src, "z_src", torch.float32, 2)
        _need_cuda(label_src, "label_src", torch.int32, 1)
        _need_cuda(r_src, "r_src", torch.float32, 1)
        if miss_selector is not None:
            _need_cuda(miss_selector, "miss_selector", torch.int32, 1)
        lib = L.load()
        k = z_src.shape[0]
        if z_src.shape[1] != self.d or label_src.shape[0] != k or r_src.shape[0] != k:
            raise ValueError("insert: shapes do not match the cache")
        if miss_selector is not None and miss_selector.shape[0] != k:
            raise ValueError("insert: selector length")
        ws = self._workspace(lib.lipcache_insert_workspace_bytes(k))
        cs = self.cstruct()
        got = ctypes.c_int64(0)
        st = lib.lipcache_insert(ctypes.byref(cs), _p(z_src), _p(label_src), _p(r_src), _p(miss_selector), k,
                                 ctypes.byref(got), _p(ws), ws.numel(), _stream(self.device))
        L.check("lipcache_insert", st)
        self.n = int(cs.n)
        return int(got.value)

    def lookup(self, zq: torch.Tensor, precision: str = "f16", want_index: bool = True,
               want_dist2: bool = True, want_band: bool = True, out: LookupResult | None = None,
               prune: bool = False) -> LookupResult:
        """lipcache_lookup: nearest certified hit per query, or MISS (async).
        ``prune``: LIPCACHE_LOOKUP_PRUNE (prefix pruning; same answers)."""
        _need_cuda(zq, "zq", torch.float32, 2)
        if zq.shape[1] != self.d:
            raise ValueError("lookup: query width differs from the cache's d")
        lib = L.load()
        B = zq.shape[0]
        dev = self.device
        if out is None:
            out = LookupResult(
                torch.empty(B, dtype=torch.int32, device=dev),
                torch.empty(B, dtype=torch.int64, device=dev) if want_index else None,
                torch.empty(B, dtype=torch.float32, device=dev) if want_dist2 else None,
                torch.zeros(4, dtype=torch.int64, device=dev),
                torch.empty(B, dtype=torch.uint8, device=dev) if want_band else None)
        prec = _PRECISION[precision] | (L.LOOKUP_PRUNE if prune else 0)
        ws = self._workspace(lib.lipcache_lookup_workspace_bytes(B, self.n, self.d, prec))
        cs = self.cstruct()
        st = lib.lipcache_lookup(ctypes.byref(cs), _p(zq), B, prec, _p(out.label), _p(out.index), _p(out.dist2),
                                 _p(out.stats), _p(out.band), _p(ws), ws.numel(), _stream(dev))
        L.check("lipcache_lookup", st)
        return out

    def lookup_prunes(self, precision: str = "f16") -> bool:
        """lipcache_lookup_prunes: whether a lookup with ``prune=True`` takes
        the pruned path on this cache (else it runs the full contraction)."""
        cs = self.cstruct()
        return bool(L.load().lipcache_lookup_prunes(ctypes.byref(cs), _PRECISION[precision] | L.LOOKUP_PRUNE))

    def lookup_noalloc(self, zq: torch.Tensor, precision: str = "f16",
                       out: LookupResult | None = None, prune: bool = False) -> LookupResult:
        """lipcache_lookup_noalloc: lookup on the library's static per-GPU
        workspace (no device allocation in the library; async)."""
        _need_cuda(zq, "zq", torch.float32, 2)
        if zq.shape[1] != self.d:
            raise ValueError("lookup_noalloc: query width differs from the cache's d")
        lib = L.load()
        B = zq.shape[0]
        dev = self.device
        if out is None:
            out = LookupResult(torch.empty(B, dtype=torch.int32, device=dev),
                               torch.empty(B, dtype=torch.int64, device=dev),
                               torch.empty(B, dtype=torch.float32, device=dev),
                               torch.zeros(4, dtype=torch.int64, device=dev),
                               torch.empty(B, dtype=torch.uint8, device=dev))
        cs = self.cstruct()
        prec = _PRECISION[precision] | (L.LOOKUP_PRUNE if prune else 0)
        st = lib.lipcache_lookup_noalloc(ctypes.byref(cs), _p(zq), B, prec, _p(out.label),
                                         _p(out.index), _p(out.dist2), _p(out.stats), _p(out.band), _stream(dev))
        L.check("lipcache_lookup_noalloc", st)
        return out

    def serve(self, zq: torch.Tensor, W: torch.Tensor, b: torch.Tensor | None, sigma: float,
              precision: str = "f16", out: LookupResult | None = None):
        """One round of certified serving (Alg. 2): look every query up, certify
        every query with the head (the label and radius a miss is cached with;
        for a bfloat16 store the rounded query is certified), and write the
        misses back.  Returns (lookup result, certified queries, rows appended).
        """
        res = self.lookup(zq, precision=precision, out=out)
        cq = certify(zq, W, b, sigma, store=self.store)
        inserted = self.insert(zq, cq.label, cq.r, res.label)
        return res, cq, inserted

    def construct(self, z: torch.Tensor, label: torch.Tensor, r: torch.Tensor, strategy: str = "radius_dedup",
                  budget: int = -1, per_class: int = 0, n_classes: int = 0, priority: torch.Tensor | None = None,
                  guard_label: torch.Tensor | None = None):
        """lipcache_construct: select candidates (Alg. 1) and append them (sync).

        Returns (rows appended, int64 tensor of the selected candidate indices
        in append order)."""
        _need_cuda(z, "z", torch.float32, 2)
        _need_cuda(label, "label", torch.int32, 1)
        _need_cuda(r, "r", torch.float32, 1)
        if priority is not None:
            _need_cuda(priority, "priority", torch.float32, 1)
        if guard_label is not None:
            _need_cuda(guard_label, "guard_label", torch.int32, 1)
        n = z.shape[0]
        if z.shape[1] != self.d or label.shape[0] != n or r.shape[0] != n:
            raise ValueError("construct: shapes do not match the cache")
        lib = L.load()
        strat = _SELECT[strategy]
        cs = self.cstruct()
        bud = self.capacity - self.n if budget < 0 else int(budget)
        sel = torch.full((max(bud, 1),), -1, dtype=torch.int64, device=self.device)
        ws = self._workspace(lib.lipcache_construct_workspace_bytes(ctypes.byref(cs), n, int(n_classes), int(budget)))
        got = ctypes.c_int64(0)
        st = lib.lipcache_construct(ctypes.byref(cs), _p(z), _p(label), _p(r), _p(guard_label), _p(priority), n,
                                    strat, int(budget), int(per_class), int(n_classes), _p(sel), ctypes.byref(got),
                                    _p(ws), ws.numel(), _stream(self.device))
        L.check("lipcache_construct", st)
        self.n = int(cs.n)
        return int(got.value), sel[: got.value]

    def boundary_radius(self, mode: str, factor: float, n_classes: int = 0) -> torch.Tensor:
        """lipcache_boundary_radius: per-entry radii of a reuse boundary (async)."""
        lib = L.load()
        out = torch.empty(max(self.n, 1), dtype=torch.float32, device=self.device)
        ws = workspace(lib.lipcache_boundary_radius_workspace_bytes(self.d, int(n_classes)), self.device)
        cs = self.cstruct()
        st = lib.lipcache_boundary_radius(ctypes.byref(cs), _BOUNDARY[mode], float(factor), int(n_classes),
                                          _p(out), _p(ws), ws.numel(), _stream(self.device))
        L.check("lipcache_boundary_radius", st)
        return out[: self.n]

    def with_radii(self, r: torch.Tensor) -> "LipCache":
        """A lookup-only view of this cache whose radii are ``r`` (features,
        labels and norms shared)."""
        _need_cuda(r, "r", torch.float32, 1)
        if r.shape[0] < self.n:
            raise ValueError("with_radii: one radius per live entry")
        v = LipCache.__new__(LipCache)
        v.__dict__.update(self.__dict__)
        v.r = r
        v._ws = None
        return v

    def build_index(self, K: int, iters: int = 4) -> "ClusterIndex":
        """lipcache_index_build over the current rows (async; the index owns its arrays)."""
        lib = L.load()
        n, d = self.n, self.d
        if n < 1:
            raise ValueError("build_index: the cache is empty")
        ix = ClusterIndex.__new__(ClusterIndex)
        ix.sorted = LipCache(d, n, store=self.store, device=self.device, image=self.zimg is not None)
        ix.perm = torch.empty(n, dtype=torch.int64, device=self.device)
        ix.offsets = torch.empty(int(K) + 1, dtype=torch.int64, device=self.device)
        ix.centers = torch.empty((int(K), d), dtype=torch.float32, device=self.device)
        ix.bound = torch.empty(int(K), dtype=torch.float32, device=self.device)
        ix.K, ix.n_indexed = int(K), 0
        ws = workspace(lib.lipcache_index_build_workspace_bytes(n, d, int(K)), self.device)
        cs = self.cstruct()
        st_ = ix.cstruct()
        st = lib.lipcache_index_build(ctypes.byref(cs), int(K), int(iters), ctypes.byref(st_), _p(ws), ws.numel(),
                                      _stream(self.device))
        L.check("lipcache_index_build", st)
        ix.n_indexed = int(st_.n_indexed)
        ix.sorted.n = int(st_.sorted.n)
        ix._build_ws = ws  # kept alive until the build has run
        return ix

    def lookup_indexed(self, index: "ClusterIndex", zq: torch.Tensor, precision: str = "f16",
                       out: LookupResult | None = None) -> tuple[LookupResult, int]:
        """lipcache_lookup_indexed: the lookup's outputs through a cluster index
        (sync).  Returns (result, query-entry pairs the filter scanned)."""
        _need_cuda(zq, "zq", torch.float32, 2)
        if zq.shape[1] != self.d:
            raise ValueError("lookup_indexed: query width differs from the cache's d")
        lib = L.load()
        B = zq.shape[0]
        dev = self.device
        if out is None:
            out = LookupResult(torch.empty(B, dtype=torch.int32, device=dev),
                               torch.empty(B, dtype=torch.int64, device=dev),
                               torch.empty(B, dtype=torch.float32, device=dev),
                               torch.zeros(4, dtype=torch.int64, device=dev),
                               torch.empty(B, dtype=torch.uint8, device=dev))
        prec = _PRECISION[precision]
        ws = self._workspace(lib.lipcache_lookup_indexed_workspace_bytes(B, self.n, self.d, index.K, index.n_indexed))
        cs = self.cstruct()
        ic = index.cstruct()
        pairs = ctypes.c_int64(0)
        st = lib.lipcache_lookup_indexed(ctypes.byref(cs), ctypes.byref(ic), _p(zq), B, prec, _p(out.label),
                                         _p(out.index), _p(out.dist2), _p(out.stats), _p(out.band),
                                         ctypes.byref(pairs), _p(ws), ws.numel(), _stream(dev))
        L.check("lipcache_lookup_indexed", st)
        return out, int(pairs.value)

    def filter_dump(self, zq: torch.Tensor, precision: str = "f16"):
        """lipcache_lookup_filter_dump: matrix-core dot products and filter decisions (small sizes)."""
        _need_cuda(zq, "zq", torch.float32, 2)
        lib = L.load()
        B = zq.shape[0]
        g_hat = torch.full((B, self.n), float("nan"), dtype=torch.float32, device=self.device)
        cand = torch.zeros((B, self.n), dtype=torch.uint8, device=self.device)
        prec = _PRECISION[precision]
        ws = self._workspace(lib.lipcache_lookup_workspace_bytes(B, self.n, self.d, prec))
        cs = self.cstruct()
        st = lib.lipcache_lookup_filter_dump(ctypes.byref(cs), _p(zq), B, prec, _p(g_hat), _p(cand), _p(ws),
                                             ws.numel(), _stream(self.device))
        L.check("lipcache_lookup_filter_dump", st)
        return g_hat, cand


class ClusterIndex:
    """Exact cluster index of a LipCache (lipcache_index): the indexed rows in
    cluster order, the cluster offsets, centres and bounds R_c."""

    sorted: LipCache
    perm: torch.Tensor      # int64 [n_indexed]: cache row of sorted row j
    offsets: torch.Tensor   # int64 [K + 1]
    centers: torch.Tensor   # float32 [K, d]
    bound: torch.Tensor     # float32 [K]
    K: int
    n_indexed: int

    def cstruct(self) -> L.LipcacheIndex:
        return L.LipcacheIndex(self.sorted.cstruct(), self.perm.data_ptr(), self.offsets.data_ptr(),
                               self.centers.data_ptr(), self.bound.data_ptr(), self.K, self.n_indexed)


def consistency(lookup_label: torch.Tensor, head_label: torch.Tensor) -> tuple[int, int]:
    """lipcache_consistency: (hits, hits returning the head's own label) (sync)."""
    _need_cuda(lookup_label, "lookup_label", torch.int32, 1)
    _need_cuda(head_label, "head_label", torch.int32, 1)
    if lookup_label.shape != head_label.shape:
        raise ValueError("consistency: shapes differ")
    lib = L.load()
    counts = torch.empty(2, dtype=torch.int64, device=lookup_label.device)
    st = lib.lipcache_consistency(_p(lookup_label), _p(head_label), lookup_label.shape[0], _p(counts),
                                  _stream(lookup_label.device))
    L.check("lipcache_consistency", st)
    h, c = counts.cpu().tolist()
    return int(h), int(c)
