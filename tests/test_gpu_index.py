"""The exact cluster index on the device (lipcache_index_build,
lipcache_lookup_indexed), against the brute-force oracle.

Index invariants, checked on the host in float64 from the device's arrays:
perm is a permutation, the offsets cover [0, n), sorted rows are the cache
rows perm[j] bit for bit, and every live row lies within its cluster's
bound: ||z_i - mu_c|| + r_i <= R_c (clusters without a live row have
R_c = -inf).

Two builds of one cache are identical bit for bit.

The indexed lookup returns the oracle's answers query by query and the
dense device lookup's outputs bit for bit (label, index, d^2, band flags,
hit and band counters), for both stores and filters, K from 1 to n,
rows appended after the build, dead rows, duplicated rows (empty
clusters), queries with more candidate clusters than a list takes, long
lists (items cut for 8-wave blocks), a ragged batch, non-finite queries,
wide features (d = 512, 1024), and the full-size mixture (every query of
the batch).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_13144_amd import api
from paper_2608_13144_amd import workload as wlmod
from gpu_helpers import DEV, build_cache, compare_lookup, gpu, host, oracle_cache, say

pytestmark = pytest.mark.gpu


def check_index(c, ix, what):
    n, K = c.n, ix.K
    assert ix.n_indexed == n and ix.sorted.n == n, what
    perm = host(ix.perm)
    off = host(ix.offsets)
    assert np.array_equal(np.sort(perm), np.arange(n)), f"{what}: perm"
    assert off[0] == 0 and off[K] == n and np.all(np.diff(off) >= 0), f"{what}: offsets"
    z = host(c.z[:n].view(torch.int16 if c.store == "bf16" else torch.int32))
    zs = host(ix.sorted.z[:n].view(torch.int16 if c.store == "bf16" else torch.int32))
    assert np.array_equal(zs, z[perm]), f"{what}: sorted rows"
    if c.zimg is not None:
        assert np.array_equal(host(ix.sorted.zimg[:n].view(torch.int16)),
                              host(c.zimg[:n].view(torch.int16))[perm]), f"{what}: image"
    r = host(c.r[:n])
    for name in ("r", "label", "norm2"):
        a = host(getattr(ix.sorted, name)[:n])
        b = host(getattr(c, name)[:n])[perm]
        assert np.array_equal(a.view(np.int32), b.view(np.int32)), f"{what}: {name}"
    zf = host(c.z[:n].float()).astype(np.float64)
    mu = host(ix.centers).astype(np.float64)
    R = host(ix.bound).astype(np.float64)
    for cl in range(K):
        rows = perm[off[cl]:off[cl + 1]]
        live = rows[r[rows] > 0]
        if live.size == 0:
            assert R[cl] == -np.inf, f"{what}: cluster {cl} has no live row but R = {R[cl]}"
            continue
        reach = np.sqrt(np.sum((zf[live] - mu[cl]) ** 2, axis=1)) + r[live].astype(np.float64)
        assert reach.max() <= R[cl], f"{what}: cluster {cl} bound {R[cl]} < reach {reach.max()}"


def same_as_dense(res_i, res_d, what):
    for f in ("label", "index", "band"):
        assert torch.equal(getattr(res_i, f), getattr(res_d, f)), f"{what}: {f}"
    assert torch.equal(res_i.dist2.view(torch.int32), res_d.dist2.view(torch.int32)), f"{what}: dist2"
    si, sd = host(res_i.stats), host(res_d.stats)
    for k in (0, 2, 3):
        assert si[k] == sd[k], f"{what}: stats[{k}] {si} vs {sd}"
    # the indexed scan filters a subset of the dense scan's pairs with the same arithmetic
    assert si[1] <= sd[1], f"{what}: re-checked {si[1]} > dense {sd[1]}"


def plan_pairs_bounds(ix, zq):
    """Pairs the plan must and may scan, from the host in float64.  Must:
    every cluster with ||q - mu_c|| < R_c is a candidate of q (soundness).
    May: the float16 cross term 2<q, mu> is within 2E of the exact one, E =
    k (||q||^2 + ||mu||^2) / 2 + e1 (||q|| + ||mu||) + e0 (k = 2u + u^2 +
    gamma (1 + u)^2, e1 = eta (1 + u) (1 + gamma) sqrt(d_pad), e0 = (1 +
    gamma) d_pad eta^2, u = 2^-11, eta = 2^-14), and the plan admits a
    cluster when the computed ||q - mu||^2 is below R^2 + 4E, so no cluster
    with an exact ||q - mu||^2 >= R^2 + 6E is ever a candidate.  A query with
    more than 256 candidates scans every indexed row."""
    mu = host(ix.centers).astype(np.float64)
    R = host(ix.bound).astype(np.float64)
    off = host(ix.offsets)
    size = np.diff(off)
    n = int(off[-1])
    Q = zq.astype(np.float64)
    D2 = ((Q[:, None, :] - mu[None, :, :]) ** 2).sum(-1)
    live = (R > 0)[None, :]
    d_pad = 32
    while d_pad < Q.shape[1]:
        d_pad *= 2
    u, eta = 2.0 ** -11, 2.0 ** -14
    gam = (d_pad + 2) * 2.0 ** -24 / (1 - (d_pad + 2) * 2.0 ** -24)
    k = 2 * u + u * u + gam * (1 + u) ** 2
    e1 = eta * (1 + u) * (1 + gam) * np.sqrt(d_pad)
    e0 = (1 + gam) * d_pad * eta * eta
    qn, cn = (Q * Q).sum(1)[:, None], (mu * mu).sum(1)[None, :]
    E = k * (qn + cn) / 2 + e1 * (np.sqrt(qn) + np.sqrt(cn)) + e0

    def pairs_of(cand):
        kk = cand.sum(1)
        per = np.where(kk > 256, n, (cand * size[None, :]).sum(1))
        return int(per.sum())
    return (pairs_of((D2 < (R * R)[None, :]) & live),
            pairs_of((D2 < (R * R)[None, :] * (1 + 1e-12) + 6.01 * E) & live))


@pytest.fixture(scope="module")
def tiny():
    wl = wlmod.make_workload("tiny-d64-c10", seed=0)
    sig = oracle.spectral_norm(wl.W).sigma
    out = {}
    for store in ("f32", "bf16"):
        cert = oracle.certify(wl.z, wl.W, wl.b, sig, store=store)
        st = oracle_cache(wl.z, cert.label, cert.r, 64, store=store)
        draws = wlmod.draw_queries(wl, 0, batch=1000)
        idx = wlmod.near_indices(draws, st.n)
        zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
        out[store] = (wl, st, zq, oracle.lookup_blocked(zq, st.z, st.r, st.label))
    return out


CASES = [("f32", "f16", True), ("f32", "f16", False), ("bf16", "f16", True), ("bf16", "f16", False),
         ("f32", "f32", True), ("bf16", "f32", True)]


@pytest.mark.parametrize("store,prec,image", CASES)
@pytest.mark.parametrize("K,iters", [(1, 0), (16, 3), (256, 4), (4096, 1)])
def test_indexed_matches_oracle_and_dense(tiny, store, prec, image, K, iters):
    wl, st, zq, ref = tiny[store]
    what = f"{store}/{prec}/image={image}/K={K}/it={iters}"
    say("index", what)
    c = build_cache(st, image=image)
    ix = c.build_index(K, iters)
    check_index(c, ix, what)
    q = gpu(zq)
    res_i, pairs = c.lookup_indexed(ix, q, precision=prec)
    compare_lookup(res_i, ref, what)
    res_d = c.lookup(q, precision=prec)
    same_as_dense(res_i, res_d, what)
    assert 0 < pairs <= zq.shape[0] * st.n
    lo, hi = plan_pairs_bounds(ix, zq)
    assert lo <= pairs <= hi, (what, lo, pairs, hi)
    say("index", what, "pairs", pairs, "of", zq.shape[0] * st.n, "exact plan", lo)


@pytest.mark.parametrize("store,prec", [("f32", "f16"), ("bf16", "f16"), ("f32", "f32")])
@pytest.mark.parametrize("K", [1, 4])
def test_long_lists(tiny, store, prec, K):
    """8,192 queries against 1 or 4 clusters: the lists average 512 queries
    or more, so the items are cut again for 8-wave blocks of 512 queries and
    longer row chunks.  Same answers as the oracle and the dense lookup, and
    the plan's pair bounds."""
    wl, st, _, _ = tiny[store]
    what = f"long lists {store}/{prec}/K={K}"
    say("index", what)
    draws = wlmod.draw_queries(wl, 1, batch=8192)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    ref = oracle.lookup_blocked(zq, st.z, st.r, st.label)
    c = build_cache(st)
    ix = c.build_index(K, 2)
    q = gpu(zq)
    res_i, pairs = c.lookup_indexed(ix, q, precision=prec)
    compare_lookup(res_i, ref, what)
    same_as_dense(res_i, c.lookup(q, precision=prec), what)
    lo, hi = plan_pairs_bounds(ix, zq)
    assert lo <= pairs <= hi, (what, lo, pairs, hi)
    say("index", what, "pairs", pairs, "of", zq.shape[0] * st.n)


@pytest.mark.parametrize("K,iters", [(4, 3), (64, 2)])
def test_build_is_deterministic(tiny, K, iters):
    """Two builds of one cache give the same index bit for bit: each Lloyd
    update sums a cluster's sampled rows in sample order (K = 4 samples every
    other row of the 4,096; K = 64 takes them all)."""
    wl, st, zq, ref = tiny["f32"]
    say("index determinism", K, iters)
    c = build_cache(st)
    a = c.build_index(K, iters)
    b = c.build_index(K, iters)
    for name in ("perm", "offsets"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    for name in ("centers", "bound"):
        assert torch.equal(getattr(a, name).view(torch.int32), getattr(b, name).view(torch.int32)), name
    check_index(c, a, f"determinism K={K}")


@pytest.mark.parametrize("store,image", [("f32", True), ("bf16", True), ("f32", False), ("bf16", False)])
def test_build_assigns_nearest_centres(tiny, store, image):
    """The final assignment puts every row in a cluster whose centre is the
    nearest one up to the rounding of the matrix-core distances: bf16 rows and
    centres (an f32 store with its image, a bf16 store) give
    d^2(assigned) <= d^2(nearest) + 2^-6 (||x||^2 + max ||mu||^2); float32 (an
    f32 store without image) 2^-14 of the same."""
    wl, st, zq, ref = tiny[store]
    say("index assignment", store, "image", image)
    c = build_cache(st, image=image)
    ix = c.build_index(16, 2)
    perm, off = host(ix.perm), host(ix.offsets)
    assign = np.empty(c.n, dtype=np.int64)
    for cl in range(ix.K):
        assign[perm[off[cl]:off[cl + 1]]] = cl
    x = host(c.z[:c.n].float()).astype(np.float64)
    mu = host(ix.centers).astype(np.float64)
    d2 = ((x[:, None, :] - mu[None, :, :]) ** 2).sum(-1)
    gap = d2[np.arange(c.n), assign] - d2.min(axis=1)
    scale = (x ** 2).sum(1) + (mu ** 2).sum(1).max()
    rel = 2.0 ** -6 if image or store == "bf16" else 2.0 ** -14
    assert np.all(gap <= rel * scale), float((gap / scale).max())
    say("assignment gap / scale max", float((gap / scale).max()), "rows not at the nearest", int(np.sum(gap > 0)))


def test_every_pair_rechecked_once_when_queues_fill():
    """Every radius huge, so every pair is a hit and every cluster a
    candidate: the indexed scan covers exactly the dense scan's pairs with the
    same filter arithmetic, so both re-check the same number of pairs.  With
    256 clusters of about 64 rows and 512 queries, each of the 2,048 waves of
    the scan meets 4,096 passing pairs: its LDS queue fills (the rest are
    re-checked at once) and the global queue (4 B + 65,536 slots) overflows
    (the late waves settle their own queues) -- no pair may be lost or
    counted twice on any of these paths."""
    cfg = wlmod.WorkloadConfig("allhit-d64", d=64, C=10, n_cache=16384, batch=512, sigma=0.5)
    wl = wlmod.make_workload(cfg, seed=5)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig)
    r = np.full(cert.r.shape, 1000.0, dtype=np.float32)
    st = oracle_cache(wl.z, cert.label, r, cfg.d)
    draws = wlmod.draw_queries(wl, 0, batch=cfg.batch)
    idx = wlmod.near_indices(draws, st.n)
    # queries near the data (composed with the certified radii), so every
    # cluster is a candidate of every query
    zq = wlmod.compose_queries(draws, st.z[idx], cert.r[idx])
    say("index all-hit queues")
    c = build_cache(st)
    ix = c.build_index(256, 2)
    check_index(c, ix, "all-hit")
    q = gpu(zq)
    res_i, pairs = c.lookup_indexed(ix, q)
    res_d = c.lookup(q)
    same_as_dense(res_i, res_d, "all-hit")
    si, sd = host(res_i.stats), host(res_d.stats)
    assert pairs == zq.shape[0] * st.n
    assert si[1] == sd[1] == zq.shape[0] * st.n, (si, sd)
    compare_lookup(res_i, oracle.lookup_blocked(zq, st.z, st.r, st.label), "all-hit")


def test_rows_appended_after_build(tiny):
    wl, st, zq, ref = tiny["f32"]
    say("index appended rows")
    c = build_cache(st, capacity=st.n + zq.shape[0])
    ix = c.build_index(64, 3)
    q = gpu(zq)
    sig = oracle.spectral_norm(wl.W).sigma
    cq = oracle.certify(zq, wl.W, wl.b, sig)
    c.insert(q, gpu(cq.label), gpu(cq.r))
    st2 = oracle_cache(np.concatenate([st.z, zq]), np.concatenate([st.label, cq.label]),
                       np.concatenate([st.r, cq.r]), 64)
    draws = wlmod.draw_queries(wl, 1, batch=777)
    idx = wlmod.near_indices(draws, st2.n)
    zq2 = wlmod.compose_queries(draws, st2.z[idx], st2.r[idx])
    ref2 = oracle.lookup_blocked(zq2, st2.z, st2.r, st2.label)
    res_i, pairs = c.lookup_indexed(ix, gpu(zq2))
    compare_lookup(res_i, ref2, "appended")
    same_as_dense(res_i, c.lookup(gpu(zq2)), "appended")
    assert host(res_i.index).max() >= st.n, "some hits should land in the appended rows"
    assert pairs >= zq2.shape[0] * zq.shape[0]


def test_dead_rows_and_duplicates(tiny):
    wl, st, zq, ref = tiny["f32"]
    say("index dead rows and duplicates")
    # every row twice (duplicates give empty clusters), one class dead
    z = np.repeat(st.z, 2, axis=0)
    lab = np.repeat(st.label, 2)
    r = np.repeat(st.r, 2)
    r = np.where(lab == 2, np.float32(0.0), r)
    st2 = oracle_cache(z, lab, r, 64)
    c = build_cache(st2)
    ix = c.build_index(1024, 2)
    check_index(c, ix, "dup")
    off = host(ix.offsets)
    say("empty clusters", int(np.sum(np.diff(off) == 0)), "dead", int(np.sum(host(ix.bound) == -np.inf)))
    ref2 = oracle.lookup_blocked(zq, st2.z, st2.r, st2.label)
    res_i, _ = c.lookup_indexed(ix, gpu(zq))
    compare_lookup(res_i, ref2, "dup")
    same_as_dense(res_i, c.lookup(gpu(zq)), "dup")


def test_queries_with_many_candidates(tiny):
    """Entries of one class get radius 15 and the index has 512 clusters:
    queries near that class have more than 256 candidate clusters and are
    scanned against every indexed row; the rest go through cluster lists."""
    wl, st, zq, ref = tiny["f32"]
    say("index many candidates")
    r = np.where(st.label == 0, np.float32(15.0), st.r).astype(np.float32)
    st2 = oracle_cache(st.z, st.label, r, 64)
    c = build_cache(st2)
    ix = c.build_index(512, 2)
    check_index(c, ix, "many")
    ref2 = oracle.lookup_blocked(zq, st2.z, st2.r, st2.label)
    res_i, pairs = c.lookup_indexed(ix, gpu(zq))
    compare_lookup(res_i, ref2, "many")
    same_as_dense(res_i, c.lookup(gpu(zq)), "many")
    say("many candidates: pairs", pairs, "of", zq.shape[0] * st.n)


def test_edge_batches(tiny):
    wl, st, zq, ref = tiny["bf16"]
    say("index edge batches")
    c = build_cache(st)
    ix = c.build_index(32, 2)
    res, pairs = c.lookup_indexed(ix, gpu(zq[:0]))
    assert pairs == 0 and host(res.stats)[0] == 0
    bad = zq[:70].copy()
    bad[3, 5] = np.nan
    bad[9, 0] = np.inf
    bad[11] = 0.0
    res_i, _ = c.lookup_indexed(ix, gpu(bad))
    res_d = c.lookup(gpu(bad))
    same_as_dense(res_i, res_d, "non-finite")
    lab = host(res_i.label)
    assert lab[3] == oracle.MISS and lab[9] == oracle.MISS
    one, _ = c.lookup_indexed(ix, gpu(zq[:1]))
    assert host(one.label)[0] == ref.label[0] or ref.flagged[0]


@pytest.mark.parametrize("store", ["f32", "bf16"])
@pytest.mark.parametrize("d", [512, 1024])
def test_wide_features(store, d):
    """d > 256: the Lloyd update takes two or four features per thread, the
    reorder several vectors per lane, and at d = 1024 the bf16 lookup scans
    the work list with the register-staged kernel.  K = 2 samples every
    other row of the 2,048; K = 16 takes them all."""
    cfg = wlmod.WorkloadConfig(f"wide-d{d}", d=d, C=10, n_cache=2048, batch=512, sigma=0.5)
    wl = wlmod.make_workload(cfg, seed=3)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig, store=store)
    st = oracle_cache(wl.z, cert.label, cert.r, d, store=store)
    draws = wlmod.draw_queries(wl, 0, batch=cfg.batch)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    ref = oracle.lookup_blocked(zq, st.z, st.r, st.label)
    c = build_cache(st)
    q = gpu(zq)
    for K in (2, 16):
        what = f"wide d={d} {store} K={K}"
        say("index", what)
        ix = c.build_index(K, 3)
        check_index(c, ix, what)
        res_i, pairs = c.lookup_indexed(ix, q)
        compare_lookup(res_i, ref, what)
        same_as_dense(res_i, c.lookup(q), what)
        assert 0 < pairs <= zq.shape[0] * st.n


@pytest.mark.slow
def test_full_size_mixture():
    cfg = wlmod.CONFIGS["mix-d256-c200"]
    say("index full size", cfg.name, "N", cfg.n_cache, "B", cfg.batch)
    wl = wlmod.make_workload(cfg, seed=0)
    sig_o = oracle.spectral_norm(wl.W).sigma
    cert_o = oracle.certify(wl.z, wl.W, wl.b, sig_o, store=cfg.store_dtype)
    st = oracle_cache(wl.z, cert_o.label, cert_o.r, cfg.d, store=cfg.store_dtype)
    draws = wlmod.draw_queries(wl, 0)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    c = build_cache(st)
    ix = c.build_index(1024, 4)
    torch.cuda.synchronize()
    say("index built")
    check_index(c, ix, "full")
    q = gpu(zq)
    res_i, pairs = c.lookup_indexed(ix, q)
    res_d = c.lookup(q)
    same_as_dense(res_i, res_d, "full")
    keep = cert_o.r > 0
    ref = oracle.lookup_partitioned(zq, st.z, st.r, st.label, wl.z_class[keep], wl.mu)
    compare_lookup(res_i, ref, "full batch")
    say("index full size pairs", pairs, "fraction", pairs / (zq.shape[0] * st.n))
    assert pairs < 0.5 * zq.shape[0] * st.n
