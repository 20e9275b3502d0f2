"""lipcache_lookup_noalloc (static per-GPU workspace) against lipcache_lookup.

Called through the C ABI (ctypes), twice in a row on the same GPU array, the
second time with a smaller batch and a smaller cache, so state the first
call left in the array must not leak into the second: every output (label,
index, d^2 bits, band flags, counters) must equal lipcache_lookup's on the
same inputs bit for bit.  The pruned lookup (LIPCACHE_LOOKUP_PRUNE) is
checked the same way; its prefix thresholds live in the same array.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2608_13144_amd import _lib as L
from paper_2608_13144_amd import workload as wlmod
from gpu_helpers import build_cache, gpu, say

pytestmark = pytest.mark.gpu


def _outputs(B):
    dev = torch.device("cuda:0")
    return [torch.full((B,), 7, dtype=torch.int32, device=dev), torch.full((B,), 7, dtype=torch.int64, device=dev),
            torch.full((B,), 7.0, dtype=torch.float32, device=dev), torch.full((4,), 7, dtype=torch.int64, device=dev),
            torch.full((B,), 7, dtype=torch.uint8, device=dev)]


def _abi(lib, name, c, zq, prec, outs, ws=None):
    p = [ctypes.c_void_p(t.data_ptr()) for t in outs]
    cs = c.cstruct()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if ws is None:
        return lib.lipcache_lookup_noalloc(ctypes.byref(cs), ctypes.c_void_p(zq.data_ptr()), zq.shape[0], prec,
                                           *p, stream)
    return lib.lipcache_lookup(ctypes.byref(cs), ctypes.c_void_p(zq.data_ptr()), zq.shape[0], prec, *p,
                               ctypes.c_void_p(ws.data_ptr()), ws.numel(), stream)


def _same(a, b, what):
    torch.cuda.synchronize()
    for x, y, f in zip(a, b, ("label", "index", "dist2", "stats", "band")):
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), f"{what}: {f} differs"


def _case(name, n_cache, B):
    cfg = wlmod.CONFIGS[name]
    wl = wlmod.make_workload(cfg, seed=0, n_cache=n_cache)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig, store=cfg.store_dtype)
    st = oracle.CacheState(d=cfg.d, capacity=n_cache, store=cfg.store_dtype)
    oracle.insert(st, wl.z, cert.label, cert.r)
    draws = wlmod.draw_queries(wl, 0, batch=B)
    idx = wlmod.near_indices(draws, st.n)
    return st, wlmod.compose_queries(draws, st.z[idx], st.r[idx])


@pytest.mark.parametrize("precision", [L.F16, L.F32, L.F16 | L.LOOKUP_PRUNE])
def test_noalloc_matches_lookup_twice(precision):
    lib = L.load()
    big_st, big_q = _case("mix-d128-c10", 65536, 8192)
    small_st, small_q = _case("tiny-d64-c10", 4096, 1000)
    for st, q, what in ((big_st, big_q, "first call (mix-d128-c10, B = 8192)"),
                        (small_st, small_q, "second call (tiny-d64-c10, B = 1000)")):
        say("noalloc", precision, what)
        c = build_cache(st)
        zq = gpu(q)
        B = q.shape[0]
        need = lib.lipcache_lookup_workspace_bytes(B, c.n, c.d, precision)
        assert need <= L.NOALLOC_SCRATCH_BYTES
        ws = torch.empty(need, dtype=torch.uint8, device="cuda:0")
        ref = _outputs(B)
        assert _abi(lib, "lookup", c, zq, precision, ref, ws) == L.OK
        got = _outputs(B)
        assert _abi(lib, "noalloc", c, zq, precision, got) == L.OK
        _same(got, ref, what)
        assert int(ref[3][0].item()) > 0  # some hits
        del c
        torch.cuda.empty_cache()
