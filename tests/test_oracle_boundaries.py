"""Pins of the reuse-boundary radii and the certified-consistency count (Sec. 6).

* scaled certified radii (factor <= 1) never break consistency (every hit
  lies inside the certified ball, Lemma 5.1), hit sets shrink monotonically
  with the factor, and factor 0 gives no hit;
* a global threshold tau reuses exactly the brute-force nearest entry when
  it lies within tau;
* the inter-class empirical radius on hand-placed classes equals half the
  distance between class means (closed form), +inf with a single class;
* on the tiny workload the empirical boundaries hit more but are not
  consistent, as the paper reports for its datasets.
"""
import numpy as np
import pytest

import oracle
from paper_2608_13144_amd import workload as wlmod


@pytest.fixture(scope="module")
def tiny():
    wl = wlmod.make_workload("tiny-d64-c10", seed=0)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig)
    st = oracle.CacheState(d=64, capacity=wl.z.shape[0])
    oracle.insert(st, wl.z, cert.label, cert.r)
    draws = wlmod.draw_queries(wl, 0, batch=192)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    head = np.argmax(oracle.logits_of(zq, wl.W, wl.b), axis=1)
    return wl, st, zq, head


def test_scaled_radii_keep_consistency_and_shrink(tiny):
    wl, st, zq, head = tiny
    prev = None
    for f in (1.0, 0.75, 0.5, 0.25, 0.0):
        r = oracle.boundary_radius(st, "scaled", f)
        res = oracle.lookup_blocked(zq, st.z, r, st.label)
        hits, cons = oracle.consistency(res.label, head)
        assert hits == cons, f"factor {f}: a certified hit returned another label"
        hit_set = res.index >= 0
        if prev is not None:
            assert not np.any(hit_set & ~prev), "hits must shrink with the factor"
        prev = hit_set
        if f == 1.0:
            assert np.array_equal(r, st.r)
            assert hits > 50
    assert not prev.any()


def test_global_threshold_is_the_nearest_entry(tiny):
    wl, st, zq, head = tiny
    d2 = ((zq[:, None, :].astype(np.float64) - st.z[None, :, :].astype(np.float64)) ** 2).sum(-1)
    nn = np.argmin(d2, axis=1)
    tau = float(np.quantile(np.sqrt(d2.min(axis=1)), 0.5))
    res = oracle.lookup_blocked(zq, st.z, oracle.boundary_radius(st, "global", tau), st.label)
    within = d2[np.arange(zq.shape[0]), nn] < tau * tau
    assert np.array_equal(res.index >= 0, within)
    assert np.array_equal(res.index[within], nn[within])


def test_interclass_closed_form():
    z = np.zeros((6, 32), np.float32)
    z[:, 0] = [0, 2, 10, 12, 1, 40]
    z[5, 1] = 30.0
    st = oracle.CacheState(d=32, capacity=8)
    oracle.insert(st, z, np.array([0, 0, 1, 1, 0, 2], np.int32), np.ones(6, np.float32))
    r = oracle.boundary_radius(st, "interclass", 1.0)
    # means: class 0 at x = 1, class 1 at x = 11, class 2 at (40, 30): nearest pairs 0-1 (10) and 2-1 (sqrt(29^2+30^2))
    assert np.allclose(r[[0, 1, 4]], 5.0) and np.allclose(r[[2, 3]], 5.0)
    assert np.isclose(r[5], 0.5 * np.hypot(29.0, 30.0), rtol=1e-6)
    assert np.allclose(oracle.boundary_radius(st, "interclass", 0.5)[:5], 2.5)
    one = oracle.CacheState(d=32, capacity=2)
    oracle.insert(one, z[:2], np.zeros(2, np.int32), np.ones(2, np.float32))
    assert np.all(np.isinf(oracle.boundary_radius(one, "interclass", 1.0)))


def test_consistency_counts():
    assert oracle.consistency([3, -1, 2, 2, -1], [3, 1, 1, 2, -1]) == (3, 2)
    assert oracle.consistency([], []) == (0, 0)


def test_empirical_boundaries_hit_more_but_break_consistency(tiny):
    wl, st, zq, head = tiny
    cert_hits, _ = oracle.consistency(oracle.lookup_blocked(zq, st.z, st.r, st.label).label, head)
    r = oracle.boundary_radius(st, "interclass", 1.0)
    hits, cons = oracle.consistency(oracle.lookup_blocked(zq, st.z, r, st.label).label, head)
    assert hits > cert_hits and cons < hits
