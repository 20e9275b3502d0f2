"""The four single-batch workloads at full size, built and launched as bench.py does.

Per workload: sigma, labels and radii of all N cache candidates against the
oracle's certify; the cache built on the device from the device's own
certificates; one batch of queries composed from the oracle's cache state;
the lookup with both filters, and the pruned float16 lookup, compared with
the oracle on EVERY query of the batch (``oracle.lookup_partitioned``
through the workload's own mixture components, itself cross-checked against
``oracle.lookup_blocked`` on a seeded sample), and every hit checked for
validity and certified consistency.  The pruned lookup must also equal the
full float16 lookup bit for bit.  At the headline workload each lookup is
run twice and must give the same bytes.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_13144_amd import api
from paper_2608_13144_amd import workload as wlmod
from gpu_helpers import DEV, check_hits_valid, compare_lookup, gpu, host, oracle_cache, say

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

NAMES = ["tiny-d64-c10", "mix-d128-c10", "mix-d128-c100", "mix-d256-c200"]


def check_certify(cert_gpu, cert_o, W, what):
    """Labels exact and radii within relative 1e-5, except where the top-2 logits
    are closer than the float64 accumulation error could reach."""
    lab = host(cert_gpu.label)
    r = host(cert_gpu.r).astype(np.float64)
    # sum_k |W_ck z_k| <= max|W| * ||z||_1 bounds the terms of every logit
    scale = 2.0 * float(np.abs(W).max()) * np.abs(cert_o.stored.astype(np.float64)).sum(axis=1)
    near_tie = cert_o.margin <= 1e-9 * scale
    assert np.array_equal(lab[~near_tie], cert_o.label[~near_tie]), what
    ok = ~near_tie & (cert_o.r > 0)
    rel = np.abs(r[ok] - cert_o.r[ok]) / cert_o.r[ok]
    assert rel.max() <= 1e-5, f"{what}: radius rel {rel.max()}"
    assert np.array_equal(r[~near_tie] > 0, cert_o.r[~near_tie] > 0), what
    return int(near_tie.sum())


def full_batch_reference(zq, st, assign, mu, what, sample=512):
    """The oracle's answer for every query, through the mixture partition;
    on a seeded sample it must equal the blocked oracle's field by field."""
    ref = oracle.lookup_partitioned(zq, st.z, st.r, st.label, assign, mu)
    rows = np.sort(np.random.default_rng(7).choice(zq.shape[0], min(sample, zq.shape[0]), replace=False))
    chk = oracle.lookup_blocked(zq[rows], st.z, st.r, st.label)
    for f in ("label", "index", "dist2", "n_hits", "n_band", "flagged"):
        assert np.array_equal(getattr(chk, f), getattr(ref, f)[rows]), f"{what}: partitioned oracle {f}"
    return ref


@pytest.mark.parametrize("name", NAMES)
def test_workload_full_size(name):
    cfg = wlmod.CONFIGS[name]
    say("workload", name, "N", cfg.n_cache, "B", cfg.batch, "d", cfg.d, "C", cfg.C)
    wl = wlmod.make_workload(cfg, seed=0)
    N, B, d = cfg.n_cache, cfg.batch, cfg.d

    sig_o = oracle.spectral_norm(wl.W).sigma
    cert_o = oracle.certify(wl.z, wl.W, wl.b, sig_o, store=cfg.store_dtype)
    st = oracle_cache(wl.z, cert_o.label, cert_o.r, d, store=cfg.store_dtype)
    assign = wl.z_class[cert_o.r > 0]          # insert keeps the certified rows in order
    say(name, "oracle chain done, n", st.n)

    W, b, z = gpu(wl.W), gpu(wl.b), gpu(wl.z)
    sig = api.spectral_norm(W)
    assert sig.converged and abs(sig.sigma - sig_o) <= 1e-9 * sig_o, (sig.sigma, sig_o)
    cert = api.certify(z, W, b, sig.sigma, store=cfg.store_dtype)
    ties = check_certify(cert, cert_o, wl.W, name)
    cache = api.LipCache(d, N + B, store=cfg.store_dtype, device=DEV)
    cache.insert(z, cert.label, cert.r)
    assert cache.n == st.n
    if ties == 0:
        assert np.array_equal(host(cache.label[: cache.n]), st.label)

    draws = wlmod.draw_queries(wl, 0)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    ref = full_batch_reference(zq, st, assign, wl.mu, name)
    say(name, "oracle lookup of all", B, "queries done; flagged", int(ref.flagged.sum()))
    full = {}
    for precision, prune in (("f16", False), ("f32", False), ("f16", True)):
        what = f"{name}/{precision}{'/pruned' if prune else ''}"
        res = cache.lookup(gpu(zq), precision=precision, prune=prune)
        nflag = compare_lookup(res, ref, what)
        nhit = check_hits_valid(res, zq, st, wl.W, wl.b, what)
        stats = host(res.stats)
        assert stats[0] == nhit
        assert 0.2 < nhit / B < 0.32, nhit / B
        say(what, "hits", nhit, "flagged", nflag, "near-tie entries", ties, "stats", stats.tolist())
        if name == "mix-d256-c200":
            again = cache.lookup(gpu(zq), precision=precision, prune=prune)
            for f in ("label", "index", "dist2", "stats", "band"):
                a, b2 = getattr(res, f), getattr(again, f)
                assert torch.equal(a.view(torch.uint8), b2.view(torch.uint8)), f"{what}: run twice {f}"
        if prune:
            # the pruned lookup gives the full float16 lookup's answers, bit for bit
            f16 = full["f16"]
            for f in ("label", "index", "dist2", "band"):
                a, b2 = getattr(f16, f), getattr(res, f)
                assert torch.equal(a.view(torch.uint8), b2.view(torch.uint8)), f"{what}: {f} differs from full"
            s16 = host(f16.stats)
            assert stats[0] == s16[0] and stats[2] == s16[2] and stats[3] == s16[3], (stats, s16)
            assert stats[1] <= s16[1], (stats, s16)
        else:
            full[precision] = res

    del cache
    torch.cuda.empty_cache()
