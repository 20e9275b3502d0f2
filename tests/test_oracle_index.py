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
