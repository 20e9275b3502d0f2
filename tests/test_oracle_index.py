"""Pins of the cluster-pruned lookup (the exact sublinear index, Sec. 4.4).

* on every partition (random, by class, one cluster, singletons) and for
  any centres, the pruned lookup returns brute force's label, index, d^2
  and hit count (the triangle inequality argument);
* singletons: the candidacy test ||q - z_i|| < 0 + r_i is the hit test
  itself, so the pairs tested equal the total number of hits (a dropped
  + r_i gives no pair, a doubled one too many);
* one cluster: every row of a live cluster is tested for the queries it
  can reach, never more than B n pairs;
* dead rows (r = 0) raise no bound: a cluster of dead rows is never tested;
* the partition by mixture component prunes most pairs.

``lookup_partitioned`` (every field of ``lookup``, for full-size batches):
equal to ``lookup`` on random partitions, by component with any centres,
and at the outer edge of the boundary band around singleton clusters;
equal to ``lookup_blocked`` on a mixture of 20,000 rows; three planted
mistakes (bounds without the band, multi-cluster queries skipped, flipped
cross term) are each caught.
"""
import numpy as np
import pytest

import oracle
from paper_2608_13144_amd import workload as wlmod


@pytest.fixture(scope="module")
def tiny():
    wl = wlmod.make_workload("tiny-d64-c10", seed=0, n_cache=1024)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig)
    st = oracle.CacheState(d=64, capacity=wl.z.shape[0])
    oracle.insert(st, wl.z, cert.label, cert.r)
    draws = wlmod.draw_queries(wl, 0, batch=96)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    assert st.n == wl.z.shape[0]
    return st, zq, oracle.lookup(zq, st.z, st.r, st.label), wl.z_class


def same_answers(a, ref):
    assert np.array_equal(a.label, ref.label)
    assert np.array_equal(a.index, ref.index)
    assert np.array_equal(a.dist2, ref.dist2)
    assert np.array_equal(a.n_hits, ref.n_hits)


@pytest.mark.parametrize("K", [1, 7, 64])
def test_random_partitions_are_exact(tiny, K):
    st, zq, ref, _ = tiny
    assign = np.random.default_rng(K).integers(0, K, st.n)
    res, pairs = oracle.cluster_pruned_lookup(zq, st.z, st.r, st.label, assign)
    same_answers(res, ref)
    assert pairs <= zq.shape[0] * st.n


def test_any_centres_are_exact(tiny):
    st, zq, ref, _ = tiny
    assign = np.arange(st.n) % 16
    centres = np.random.default_rng(3).standard_normal((16, st.d)) * 3.0
    res, _ = oracle.cluster_pruned_lookup(zq, st.z, st.r, st.label, assign, centres=centres)
    same_answers(res, ref)


def test_singletons_test_exactly_the_hits(tiny):
    st, zq, ref, _ = tiny
    res, pairs = oracle.cluster_pruned_lookup(zq, st.z, st.r, st.label, np.arange(st.n))
    same_answers(res, ref)
    assert ref.n_hits.sum() > 20
    assert pairs == int(ref.n_hits.sum())


def test_component_partition_prunes(tiny):
    st, zq, ref, comp = tiny
    res, pairs = oracle.cluster_pruned_lookup(zq, st.z, st.r, st.label, comp)
    same_answers(res, ref)
    assert pairs < 0.5 * zq.shape[0] * st.n


def test_dead_rows_raise_no_bound(tiny):
    st, zq, ref, _ = tiny
    r = st.r.copy()
    dead = st.label == 3
    r[dead] = 0.0
    assign = np.where(dead, 0, 1 + st.label)
    res, pairs = oracle.cluster_pruned_lookup(zq, st.z, r, st.label, assign)
    same_answers(res, oracle.lookup(zq, st.z, r, st.label))
    res2, pairs2 = oracle.cluster_pruned_lookup(zq, st.z[~dead], r[~dead], st.label[~dead], assign[~dead])
    assert pairs == pairs2


# ---------------------------------------------------------------- lookup_partitioned
def same_everything(a, ref):
    same_answers(a, ref)
    assert np.array_equal(a.n_band, ref.n_band)
    assert np.array_equal(a.flagged, ref.flagged)


@pytest.mark.parametrize("K", [1, 7, 64])
def test_partitioned_equals_lookup_on_random_partitions(tiny, K):
    st, zq, ref, _ = tiny
    assign = np.random.default_rng(K).integers(0, K, st.n)
    centres = np.stack([st.z[assign == c].astype(np.float64).mean(axis=0) if np.any(assign == c)
                        else np.zeros(st.d) for c in range(K)])
    same_everything(oracle.lookup_partitioned(zq, st.z, st.r, st.label, assign, centres), ref)


def test_partitioned_equals_lookup_by_component_and_any_centres(tiny):
    st, zq, ref, comp = tiny
    K = int(comp.max()) + 1
    centres = np.stack([st.z[comp == c].astype(np.float64).mean(axis=0) for c in range(K)])
    same_everything(oracle.lookup_partitioned(zq, st.z, st.r, st.label, comp, centres), ref)
    far = np.random.default_rng(3).standard_normal((K, st.d)) * 3.0
    same_everything(oracle.lookup_partitioned(zq, st.z, st.r, st.label, comp, far), ref)


def _band_edge_case():
    """Singleton clusters centred on their rows: R_c = (1 + band) r_c.
    Queries at D = (1 +- 0.5e-5) r (band pairs, one a hit), at (1 + 3e-5) r
    (outside the band) and duplicates at distance 0 of a dead row."""
    rng = np.random.default_rng(9)
    d = 32
    z = rng.standard_normal((6, d)).astype(np.float32)
    r = np.array([0.5, 0.7, 0.9, 1.1, 0.0, 0.4], np.float32)
    lab = np.arange(6, dtype=np.int32)
    v = rng.standard_normal((8, d))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    pick = np.array([0, 1, 2, 3, 0, 5, 1, 2])
    f = np.array([1 + 0.5e-5, 1 - 0.5e-5, 1 + 3e-5, 0.5, 1 + 0.9e-5, 1 - 0.9e-5, 2.0, 1 + 0.2e-5])
    zq = (z[pick].astype(np.float64) + (f * r[pick])[:, None] * v).astype(np.float32)
    zq = np.concatenate([zq, z[4:5]])  # exactly on the dead row
    ref = oracle.lookup(zq, z, r, lab)
    assert ref.n_band.sum() >= 4 and ref.flagged.sum() >= 3
    return zq, z, r, lab, ref


def test_partitioned_keeps_band_pairs_of_pruned_clusters():
    zq, z, r, lab, ref = _band_edge_case()
    assign = np.arange(z.shape[0])
    same_everything(oracle.lookup_partitioned(zq, z, r, lab, assign, z.astype(np.float64)), ref)


def _mutant(old, new):
    """lookup_partitioned with one planted mistake (a source-level edit)."""
    import inspect
    from oracle import lipcache_oracle as base
    src = inspect.getsource(base.lookup_partitioned)
    assert src.count(old) == 1, old
    ns = dict(vars(base))
    exec(src.replace(old, new), ns)
    return ns["lookup_partitioned"]


PARTITION_MUTANTS = {
    # bounds without the band's width: band pairs just outside a pruned ball are lost
    "no band in R_c": ("R[c] = np.max(dz + (1.0 + band_rel) * r64[live])", "R[c] = np.max(dz + r64[live])"),
    # a query whose hits may lie in several clusters is never searched
    "multi-cluster queries skipped": ("for qi in np.flatnonzero(count > 1):", "for qi in np.flatnonzero(count > K):"),
    # sign of the cross term in ||q - mu||^2
    "flipped expansion": ("d2 = scale - 2.0 * (Q[s0:s1] @ mu.T)", "d2 = scale + 2.0 * (Q[s0:s1] @ mu.T)"),
}


@pytest.mark.parametrize("name", sorted(PARTITION_MUTANTS))
def test_partitioned_planted_mistake_is_caught(tiny, name):
    fn = _mutant(*PARTITION_MUTANTS[name])
    caught = False
    zq, z, r, lab, ref = _band_edge_case()
    try:
        same_everything(fn(zq, z, r, lab, np.arange(z.shape[0]), z.astype(np.float64)), ref)
    except AssertionError:
        caught = True
    st, zq2, ref2, comp = tiny
    for K in (7, 64):
        assign = np.random.default_rng(K).integers(0, K, st.n)
        centres = np.stack([st.z[assign == c].astype(np.float64).mean(axis=0) for c in range(K)])
        try:
            same_everything(fn(zq2, st.z, st.r, st.label, assign, centres), ref2)
        except AssertionError:
            caught = True
    assert caught, name


def test_partitioned_full_size_shape_prunes():
    """On a mixture partitioned by component, every query searches one
    cluster, and the answers equal lookup_blocked's on the whole batch."""
    cfg = wlmod.WorkloadConfig("part-d64", d=64, C=20, n_cache=20000, batch=600, sigma=0.5)
    wl = wlmod.make_workload(cfg, seed=4)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig)
    draws = wlmod.draw_queries(wl, 0)
    idx = wlmod.near_indices(draws, wl.z.shape[0])
    zq = wlmod.compose_queries(draws, wl.z[idx], cert.r[idx])
    ref = oracle.lookup_blocked(zq, wl.z, cert.r, cert.label)
    res = oracle.lookup_partitioned(zq, wl.z, cert.r, cert.label, wl.z_class, wl.mu)
    same_everything(res, ref)
    assert (ref.index >= 0).sum() > 100
