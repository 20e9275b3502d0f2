"""The streaming workload: rounds of lookup -> certify -> write-back on a bf16 cache.

Each round composes its queries from the cache state agreed at the start of
the round, looks them up, certifies every query (rounded to bf16, the value a
miss is stored as) and appends the misses.

* ``test_stream_lockstep`` runs the whole protocol on both sides at a reduced
  size and compares every query of every round.  When the two sides differ
  only on queries the oracle flags (a pair within relative 1e-5 of a ball
  boundary), both append the oracle's miss set, so the states stay in
  lockstep; any other difference fails.
* ``test_stream_full_size_round`` runs the full workload (2,097,152 initial
  entries, 16 rounds of 65,536 queries, one test per round) with the same
  protocol: every query of every round is compared with the oracle
  (``oracle.lookup_partitioned`` through the mixture components; appended
  rows join the cluster of their nearest class mean), every hit is checked
  for validity and certified consistency, both sides append the oracle's
  miss set, and the appended rows (bf16 values, labels, radii) must equal
  the oracle's certify of the queries.  Every round also runs the pruned
  lookup (LIPCACHE_LOOKUP_PRUNE), whose answers must equal the full lookup's
  bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_13144_amd import api
from paper_2608_13144_amd import workload as wlmod
from gpu_helpers import DEV, check_hits_valid, compare_lookup, gpu, host, say

pytestmark = pytest.mark.gpu

NAME = "stream-d256-c200-bf16"


def _initial(cfg, n_cache, capacity):
    wl = wlmod.make_workload(cfg, seed=0, n_cache=n_cache)
    sig_o = oracle.spectral_norm(wl.W).sigma
    cert_o = oracle.certify(wl.z, wl.W, wl.b, sig_o, store="bf16")
    st = oracle.CacheState(d=cfg.d, capacity=capacity, store="bf16")
    oracle.insert(st, wl.z, cert_o.label, cert_o.r)
    W, b = gpu(wl.W), gpu(wl.b)
    sig = api.spectral_norm(W)
    assert abs(sig.sigma - sig_o) <= 1e-9 * sig_o
    cache = api.LipCache(cfg.d, capacity, store="bf16", device=DEV)
    cert = api.certify(gpu(wl.z), W, b, sig.sigma, store="bf16")
    cache.insert(gpu(wl.z), cert.label, cert.r)
    assert cache.n == st.n
    return wl, sig_o, st, W, b, sig.sigma, cache, cert_o.r > 0


def _check_appended(cache, n0, st, n0_o, what):
    """Rows appended this round: bf16 values bit-exact, labels exact, radii within 1e-5."""
    zs = host(cache.z[n0:cache.n].view(torch.int16)).view(np.uint16)
    want = (st.z[n0_o:].view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(zs, want), what
    assert np.array_equal(host(cache.label[n0:cache.n]), st.label[n0_o:]), what
    r = host(cache.r[n0:cache.n]).astype(np.float64)
    if r.size:
        rel = np.abs(r - st.r[n0_o:]) / st.r[n0_o:]
        assert rel.max() <= 1e-5, f"{what}: radius rel {rel.max()}"


def test_stream_lockstep():
    cfg = wlmod.CONFIGS[NAME]
    n_cache, B, rounds = 8192, 1024, 4
    cap = n_cache + rounds * B
    wl, sig_o, st, W, b, sig, cache, _ = _initial(cfg, n_cache, cap)
    adopted = 0
    for t in range(rounds):
        say("stream lockstep round", t, "n", st.n)
        draws = wlmod.draw_queries(wl, t, batch=B)
        idx = wlmod.near_indices(draws, st.n)
        zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
        ref = oracle.lookup_blocked(zq, st.z, st.r, st.label)
        res = cache.lookup(gpu(zq), precision="f16")
        compare_lookup(res, ref, f"stream round {t}")
        lab = host(res.label)
        differs = lab != ref.label
        if differs.any():            # only flagged queries can get here
            adopted += int(differs.sum())
            sel = gpu(ref.label)
        else:
            sel = res.label
        cq_o = oracle.certify(zq, wl.W, wl.b, sig_o, store="bf16")
        n0, n0_o = cache.n, st.n
        oracle.insert(st, zq, cq_o.label, cq_o.r, ref.label)
        cq = api.certify(gpu(zq), W, b, sig, store="bf16")
        got = cache.insert(gpu(zq), cq.label, cq.r, sel)
        assert got == st.n - n0_o and cache.n == st.n
        _check_appended(cache, n0, st, n0_o, f"round {t}")
        check_hits_valid(res, zq, oracle.CacheState(cfg.d, st.capacity, "bf16", st.z[:n0_o], st.r[:n0_o],
                                                    st.label[:n0_o], st.norm2[:n0_o]),
                         wl.W, wl.b, f"round {t}")
    say("stream lockstep: adopted oracle decisions on", adopted, "flagged queries; final n", st.n)
    assert st.n > n_cache + rounds * B // 2


def _nearest_mean(x, mu):
    """Cluster of appended rows for the oracle's partition: the nearest class
    mean (any assignment keeps lookup_partitioned exact)."""
    X = np.asarray(x, dtype=np.float64)
    d2 = (X * X).sum(1)[:, None] + (mu * mu).sum(1)[None, :] - 2.0 * X @ mu.T
    return np.argmin(d2, axis=1)


@pytest.fixture(scope="module")
def full_stream():
    cfg = wlmod.CONFIGS[NAME]
    wl, sig_o, st, W, b, sig, cache, keep = _initial(cfg, cfg.n_cache, cfg.capacity)
    state = dict(cfg=cfg, wl=wl, sig_o=sig_o, st=st, W=W, b=b, sig=sig, cache=cache,
                 assign=wl.z_class[keep].astype(np.int64), round=0, adopted=0)
    say("stream full size: initial n", st.n)
    yield state
    del state["cache"]
    torch.cuda.empty_cache()


@pytest.mark.slow
@pytest.mark.parametrize("t", range(16))
def test_stream_full_size_round(full_stream, t):
    """Round t of the full streaming workload (65,536 queries against 2.1M ->
    2.9M bf16 entries): every query compared with the oracle (through the
    mixture partition), every hit valid and certified-consistent, both sides
    append the oracle's miss set, and the appended rows (bf16 bits, labels,
    radii) equal the oracle's certify."""
    S = full_stream
    assert S["round"] == t, "rounds run in order"
    cfg, wl, st, cache = S["cfg"], S["wl"], S["st"], S["cache"]
    draws = wlmod.draw_queries(wl, t)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    n0, n0_o = cache.n, st.n
    before = oracle.CacheState(cfg.d, st.capacity, "bf16", st.z, st.r, st.label, st.norm2)
    res = cache.lookup(gpu(zq), precision="f16")
    ref = oracle.lookup_partitioned(zq, st.z, st.r, st.label, S["assign"], wl.mu)
    compare_lookup(res, ref, f"stream full round {t}")
    assert cache.lookup_prunes("f16")
    pr = cache.lookup(gpu(zq), precision="f16", prune=True)
    for f in ("label", "index", "dist2", "band"):
        a, b2 = getattr(res, f), getattr(pr, f)
        assert torch.equal(a.view(torch.uint8), b2.view(torch.uint8)), f"stream full round {t}: pruned {f}"
    sf, sp = host(res.stats), host(pr.stats)
    assert sf[0] == sp[0] and sf[2] == sp[2] and sf[3] == sp[3] and sp[1] <= sf[1], (sf, sp)
    nhit = check_hits_valid(res, zq, before, wl.W, wl.b, f"stream full round {t}")
    lab = host(res.label)
    differs = lab != ref.label          # only flagged queries can get here
    S["adopted"] += int(differs.sum())
    sel = gpu(ref.label) if differs.any() else res.label
    cq_o = oracle.certify(zq, wl.W, wl.b, S["sig_o"], store="bf16")
    oracle.insert(st, zq, cq_o.label, cq_o.r, ref.label)
    cq = api.certify(gpu(zq), S["W"], S["b"], S["sig"], store="bf16")
    got = cache.insert(gpu(zq), cq.label, cq.r, sel)
    assert got == st.n - n0_o and cache.n == st.n
    _check_appended(cache, n0, st, n0_o, f"full round {t}")
    S["assign"] = np.concatenate([S["assign"], _nearest_mean(st.z[n0_o:], wl.mu)])
    S["round"] = t + 1
    say("stream full round", t, "n", n0, "->", cache.n, "hits", nhit, "flagged", int(ref.flagged.sum()),
        "adopted so far", S["adopted"], "stats", host(res.stats).tolist())
    if t == cfg.rounds - 1:
        assert cache.n > cfg.n_cache + cfg.rounds * cfg.batch // 2
