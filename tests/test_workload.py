"""The seeded input generator: determinism and the distributions it promises."""
import math

import numpy as np

from paper_2608_13144_amd import workload as wlmod


def test_same_seed_same_bytes():
    a = wlmod.make_workload("tiny-d64-c10", seed=0)
    b = wlmod.make_workload("tiny-d64-c10", seed=0)
    for x, y in [(a.W, b.W), (a.b, b.b), (a.z, b.z), (a.mu, b.mu)]:
        assert x.tobytes() == y.tobytes()
    qa, qb = wlmod.draw_queries(a, 3), wlmod.draw_queries(b, 3)
    for x, y in [(qa.fresh, qb.fresh), (qa.direction, qb.direction), (qa.perm, qb.perm)]:
        assert x.tobytes() == y.tobytes()
    c = wlmod.make_workload("tiny-d64-c10", seed=1)
    assert a.z.tobytes() != c.z.tobytes()


def test_shapes_and_distributions():
    cfg = wlmod.CONFIGS["mix-d128-c100"]
    wl = wlmod.make_workload(cfg, seed=0, n_cache=20000)
    assert wl.W.shape == (100, 128) and wl.W.dtype == np.float32
    assert abs(wl.W.std() - 1 / math.sqrt(128)) < 0.02 / math.sqrt(128) * 10
    assert abs(wl.b.std() - 0.1) < 0.03
    assert abs(wl.mu.std() - 2.0) < 0.05
    resid = wl.z.astype(np.float64) - wl.mu[wl.z_class]
    assert abs(resid.std() - 0.7) < 0.01
    counts = np.bincount(wl.z_class, minlength=100)
    assert counts.min() > 100
    tiny = wlmod.make_workload("tiny-d64-c10", seed=0)
    assert np.all(tiny.b == 0)


def test_chunked_draw_matches_single_draw():
    cfg = wlmod.WorkloadConfig("t", d=8, C=3, n_cache=5, batch=4, sigma=0.5)
    wl = wlmod.make_workload(cfg, seed=11)
    rng = np.random.default_rng(11)
    W = (rng.standard_normal((3, 8)) / math.sqrt(8)).astype(np.float32)
    mu = rng.standard_normal((3, 8)) * 2.0
    k = rng.integers(0, 3, size=5)
    z = (mu[k] + 0.5 * rng.standard_normal((5, 8))).astype(np.float32)
    assert np.array_equal(W, wl.W) and np.array_equal(z, wl.z)


def test_compose_places_queries_at_u_r():
    wl = wlmod.make_workload("tiny-d64-c10", seed=0, n_cache=100)
    dr = wlmod.draw_queries(wl, 0, batch=64)
    r = np.linspace(0.1, 1.0, 100).astype(np.float32)
    idx = wlmod.near_indices(dr, 100)
    q = wlmod.compose_queries(dr, wl.z[idx], r[idx])
    assert q.shape == (64, 64) and q.dtype == np.float32
    inv = np.argsort(dr.perm)
    near = q[inv[: dr.n_near]]
    dist = np.linalg.norm(near.astype(np.float64) - wl.z[idx].astype(np.float64), axis=1)
    assert np.allclose(dist, dr.u * r[idx], rtol=1e-5, atol=1e-6)
    assert np.array_equal(q[inv[dr.n_near:]], dr.fresh)
