"""The pruned lookup (LIPCACHE_LOOKUP_PRUNE) against the oracle and the full lookup.

The squared distance over the first 32 features is a lower bound of the whole
(Eq. (13) sums non-negative terms), so the prefix filter may only drop blocks
of pairs that hold no hit and no boundary-band pair.  Every block it keeps
goes through the same dot products as the full lookup.  So labels, indices,
distances, band flags and the hit, band-pair and band-query counts must equal
the full lookup's bit for bit, and the oracle's on every unflagged query; only
the number of re-checked pairs may fall (fewer pairs the full filter let
through without being hits).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_13144_amd import _lib as L
from paper_2608_13144_amd import workload as wlmod
from gpu_helpers import build_cache, compare_lookup, gpu, host, oracle_cache, say

pytestmark = pytest.mark.gpu


def same_as_full(c, zq_t, what, precision="f16"):
    """Pruned and full lookups of one batch: identical answers, fewer re-checks."""
    full = c.lookup(zq_t, precision=precision)
    pr = c.lookup(zq_t, precision=precision, prune=True)
    for f in ("label", "index", "dist2", "band"):
        a, b = getattr(full, f), getattr(pr, f)
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"{what}: {f} differs from the full lookup"
    sf, sp = host(full.stats), host(pr.stats)
    for k in (L.STAT_HITS, L.STAT_BAND_PAIRS, L.STAT_BAND_QUERIES):
        assert sf[k] == sp[k], f"{what}: stats[{k}] {sp[k]} vs full {sf[k]}"
    assert sp[L.STAT_RECHECKED] <= sf[L.STAT_RECHECKED], (what, sp.tolist(), sf.tolist())
    return pr, sf, sp


def check_band(res, ref, what):
    """Every boundary-band pair is re-checked: per-query flags and the pair count."""
    band = host(res.band).astype(bool)
    assert np.array_equal(band, ref.n_band > 0), f"{what}: band flags"
    assert int(host(res.stats)[L.STAT_BAND_PAIRS]) == int(ref.n_band.sum()), f"{what}: band pairs"


def mixture_case(d, N, B, store, seed, C=7):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((C, d)) / math.sqrt(d)).astype(np.float32)
    mu = 2.0 * rng.standard_normal((C, d))
    z = (mu[rng.integers(0, C, N)] + 0.5 * rng.standard_normal((N, d))).astype(np.float32)
    sig = oracle.spectral_norm(W).sigma
    cert = oracle.certify(z, W, None, sig, store=store)
    st = oracle_cache(z, cert.label, cert.r, d, store=store)
    pick = rng.integers(0, st.n, B)
    v = rng.standard_normal((B, d))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    u = rng.uniform(0, 2, B)
    zq = (st.z[pick].astype(np.float64) + (u * st.r[pick])[:, None] * v).astype(np.float32)
    zq[1::5] = (mu[rng.integers(0, C, zq[1::5].shape[0])] + 0.5 * rng.standard_normal(zq[1::5].shape)).astype(np.float32)
    return st, zq


@pytest.mark.parametrize("d,N,B,store,image", [
    (64, 40000, 700, "f32", True),     # two k-steps: the prefix is half the row
    (96, 33001, 333, "f32", True),     # d padded to 128; ragged slices: full and partial prefix tiles
    (128, 70000, 517, "bf16", True),
    (256, 50001, 300, "f32", True),
    (512, 40000, 70, "bf16", True),    # two row tiles of queries per wave
    (256, 32768, 1, "f32", True),      # the smallest pruned cache, one query
    (128, 20000, 200, "f32", True),    # below 32,768 rows: the option changes nothing
    (1024, 900, 40, "f32", True),      # no DMA kernel at d = 1024: the option changes nothing
    (32, 40000, 200, "f32", True),     # one k-step: nothing to prune
    (128, 40000, 200, "f32", False),   # no float16 image: the option changes nothing
])
def test_prune_matches_oracle_and_full(d, N, B, store, image):
    say("pruned lookup", d, N, B, store, "image", image)
    st, zq = mixture_case(d, N, B, store, seed=d + N + B)
    ref = oracle.lookup_blocked(zq, st.z, st.r, st.label)
    c = build_cache(st, image=image)
    what = f"prune d={d} N={N} B={B} {store} image={image}"
    pr, sf, sp = same_as_full(c, gpu(zq), what)
    compare_lookup(pr, ref, what)
    check_band(pr, ref, what)
    say(what, "rechecked full", int(sf[L.STAT_RECHECKED]), "pruned", int(sp[L.STAT_RECHECKED]))
    if B >= 20:
        assert (ref.index >= 0).sum() > 0


def test_prune_prefix_geometry():
    """Pairs placed by where their distance lies: entirely past the prefix (a
    hit the prefix cannot see), entirely inside it, a prefix that alone fits
    the ball while the whole row does not, and pairs at relative 1e-6 and
    5e-6 inside and outside the ball boundary with the offset inside the
    prefix (band pairs the widened prefix ball must keep), among 40,000 far
    rows so the blocks around them are pruned."""
    say("pruned lookup: prefix geometry")
    rng = np.random.default_rng(11)
    d, N = 128, 40000
    z = (6.0 * rng.standard_normal((N, d))).astype(np.float32)
    r = np.full(N, 1.0, np.float32)
    lab = rng.integers(0, 5, N).astype(np.int32)
    picks = rng.choice(N, 12, replace=False)
    q = []
    tail = np.zeros(d)
    tail[40:] = rng.standard_normal(d - 40)
    tail /= np.linalg.norm(tail)
    head = np.zeros(d)
    head[:32] = rng.standard_normal(32)
    head /= np.linalg.norm(head)
    base = z[picks].astype(np.float64)
    q.append(base[0] + 0.7 * tail)                       # hit, offset past the prefix
    q.append(base[1] + 0.7 * head)                       # hit, offset inside the prefix
    q.append(base[2] + 0.6 * head + 0.9 * tail)          # prefix fits the ball, the row does not: miss
    for k, s in enumerate((1 - 1e-6, 1 + 1e-6, 1 - 5e-6, 1 + 5e-6)):
        q.append(base[3 + k] + s * head)                 # boundary band, offset in the prefix
    q.append(base[7] + 0.5 * head + 0.5 * tail)          # hit split between both parts
    q.append(6.0 * rng.standard_normal(d))               # far from everything
    zq = np.stack(q).astype(np.float32)
    st = oracle_cache(z, lab, r, d)
    ref = oracle.lookup(zq, st.z, st.r, st.label)
    c = build_cache(st)
    pr, sf, sp = same_as_full(c, gpu(zq), "prefix geometry")
    compare_lookup(pr, ref, "prefix geometry")
    check_band(pr, ref, "prefix geometry")
    got = host(pr.index)
    assert got[0] == picks[0] and got[1] == picks[1] and got[7] == picks[7], got.tolist()
    assert got[2] == -1 and got[8] == -1, got.tolist()
    assert ref.n_band[3:7].sum() >= 2, ref.n_band.tolist()


@pytest.mark.parametrize("N,B", [(33000, 64)])
def test_prune_outside_f16_range(N, B):
    """Rows and queries outside the float16 range pass the prefix filter
    against everything, as they pass the full one."""
    say("pruned lookup outside f16 range", N, B)
    rng = np.random.default_rng(N + B + 1)
    d = 128
    z = rng.standard_normal((N, d))
    z[::97] *= 4.0e4
    r = (0.05 * np.linalg.norm(z, axis=1)).astype(np.float32)
    z = z.astype(np.float32)
    st = oracle_cache(z, rng.integers(0, 9, N).astype(np.int32), r, d)
    pick = rng.integers(0, N, B)
    v = rng.standard_normal((B, d))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    zq = (st.z[pick].astype(np.float64) + (rng.uniform(0, 2, B) * st.r[pick])[:, None] * v).astype(np.float32)
    ref = oracle.lookup_blocked(zq, st.z, st.r, st.label)
    c = build_cache(st)
    pr, _, _ = same_as_full(c, gpu(zq), "prune outside f16 range")
    compare_lookup(pr, ref, "prune outside f16 range")
    assert (ref.index >= 0).sum() > B // 4


def test_prune_workload_blocks():
    """A 40,000-row sub-block of each d >= 64 workload (its own rows and
    query recipe): answers equal the oracle's and the full lookup's."""
    for name in ("tiny-d64-c10", "mix-d128-c100", "mix-d256-c200", "stream-d256-c200-bf16"):
        cfg = wlmod.CONFIGS[name]
        wl = wlmod.make_workload(cfg, seed=0, n_cache=40000)
        say("pruned lookup workload block", name)
        sig = oracle.spectral_norm(wl.W).sigma
        cert = oracle.certify(wl.z, wl.W, wl.b, sig, store=cfg.store_dtype)
        st = oracle_cache(wl.z, cert.label, cert.r, cfg.d, store=cfg.store_dtype)
        draws = wlmod.draw_queries(wl, 0, batch=1024)
        idx = wlmod.near_indices(draws, st.n)
        zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
        ref = oracle.lookup_blocked(zq, st.z, st.r, st.label)
        c = build_cache(st)
        pr, sf, sp = same_as_full(c, gpu(zq), name)
        compare_lookup(pr, ref, f"prune {name}")
        check_band(pr, ref, f"prune {name}")


def test_prune_invalid_uses():
    """The option is a lookup option: the filter dump and the indexed lookup
    reject it, and unknown option bits are invalid."""
    st, zq = mixture_case(64, 300, 8, "f32", seed=5)
    c = build_cache(st)
    lib = L.load()
    import ctypes
    cs = c.cstruct()
    out = torch.empty(8, dtype=torch.int32, device="cuda:0")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda:0")
    zq_t = gpu(zq)
    bad = L.F16 | 0x200
    st_ = lib.lipcache_lookup(ctypes.byref(cs), ctypes.c_void_p(zq_t.data_ptr()), 8, bad,
                              ctypes.c_void_p(out.data_ptr()), None, None, None, None,
                              ctypes.c_void_p(ws.data_ptr()), ws.numel(), None)
    assert st_ == L.EINVAL
    g = torch.empty(8 * 300, dtype=torch.float32, device="cuda:0")
    cand = torch.empty(8 * 300, dtype=torch.uint8, device="cuda:0")
    st_ = lib.lipcache_lookup_filter_dump(ctypes.byref(cs), ctypes.c_void_p(zq_t.data_ptr()), 8,
                                          L.F16 | L.LOOKUP_PRUNE, ctypes.c_void_p(g.data_ptr()),
                                          ctypes.c_void_p(cand.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                          ws.numel(), None)
    assert st_ == L.EINVAL
