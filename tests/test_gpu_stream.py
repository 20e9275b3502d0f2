"""The streaming workload: rounds of lookup -> certify -> write-back on a bf16 cache.

Each round composes its queries from the cache state agreed at the start of
the round, looks them up, certifies every query (rounded to bf16, the value a
miss is stored as) and appends the misses.

* ``test_stream_lockstep`` runs the whole protocol on both sides at a reduced
  size and compares every query of every round.  When the two sides differ
  only on queries the oracle flags (a pair within relative 1e-5 of a ball
  boundary), both append the oracle's miss set, so the states stay in
  lockstep; any other difference fails.
* ``test_stream_full_size`` runs the full workload (2,097,152 initial entries,
  16 rounds of 65,536 queries) on the device as bench.py does.  The oracle
  cannot afford 16 full rounds, so per round it checks a seeded sample of
  queries exactly, every hit for validity and certified consistency, and the
  appended rows (bf16 values, labels, radii) against its own certify of the
  queries; its state then appends the rows the device's miss set selects.
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
    return wl, sig_o, st, W, b, sig.sigma, cache


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
    wl, sig_o, st, W, b, sig, cache = _initial(cfg, n_cache, cap)
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


@pytest.mark.slow
def test_stream_full_size():
    cfg = wlmod.CONFIGS[NAME]
    sample = 256
    wl, sig_o, st, W, b, sig, cache = _initial(cfg, cfg.n_cache, cfg.capacity)
    say("stream full size: initial n", st.n)
    rng = np.random.default_rng(11)
    for t in range(cfg.rounds):
        draws = wlmod.draw_queries(wl, t)
        idx = wlmod.near_indices(draws, st.n)
        zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
        n0, n0_o = cache.n, st.n
        before = oracle.CacheState(cfg.d, st.capacity, "bf16", st.z, st.r, st.label, st.norm2)
        res, cq, got = cache.serve(gpu(zq), W, b, sig, precision="f16")
        rows = np.sort(rng.choice(cfg.batch, sample, replace=False))
        ref = oracle.lookup_blocked(zq[rows], before.z, before.r, before.label)
        compare_lookup(res, ref, f"stream full round {t}", rows=rows)
        nhit = check_hits_valid(res, zq, before, wl.W, wl.b, f"stream full round {t}")
        cq_o = oracle.certify(zq, wl.W, wl.b, sig_o, store="bf16")
        oracle.insert(st, zq, cq_o.label, cq_o.r, host(res.label))
        assert got == st.n - n0_o and cache.n == st.n
        _check_appended(cache, n0, st, n0_o, f"full round {t}")
        say("stream full round", t, "n", n0, "->", cache.n, "hits", nhit, "stats", host(res.stats).tolist())
    assert cache.n > cfg.n_cache + cfg.rounds * cfg.batch // 2
    del cache
    torch.cuda.empty_cache()
