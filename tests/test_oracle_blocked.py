"""``oracle.lookup_blocked`` (BLAS prefilter + direct re-check) against ``oracle.lookup``.

``lookup`` is the plain definition of Eq. (13)-(15), pinned in ``pins.py``;
the blocked form only skips pairs that a rigorous bound proves to be neither
hits nor band pairs, so every field must agree bit for bit.  The cases stress
the prefilter: pairs at relative 1e-6 .. 1e-12 of the ball boundary, large
feature norms (the slack scales with them), duplicates, non-positive radii,
a NaN query, bfloat16 stored values and an empty cache.
"""
import inspect

import numpy as np
import pytest

import oracle
from oracle import lipcache_oracle as base
from paper_2608_13144_amd import workload as wlmod

FIELDS = ("label", "index", "dist2", "n_hits", "n_band", "flagged")


def same(a, b):
    return all(getattr(a, f).tobytes() == getattr(b, f).tobytes() for f in FIELDS)


def adversarial(d, n=600, B=300, offset=6.0, seed=0, store="f32"):
    """Entries with large norms and queries on, just inside and just outside balls."""
    rng = np.random.default_rng(seed)
    z = (offset + rng.standard_normal((n, d))).astype(np.float32)
    z = oracle.stored_values(z, store)
    z[7] = z[3]                                   # duplicate entry: lower index wins
    r = rng.uniform(0.2, 2.0, n).astype(np.float32)
    r[11] = 0.0                                   # never hit
    r[12] = -1.0
    lab = rng.integers(0, 10, n).astype(np.int32)
    pick = rng.integers(0, n, B)
    v = rng.standard_normal((B, d))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    rel = rng.choice([1 - 1e-6, 1 + 1e-6, 1 - 1e-9, 1 + 1e-9, 1 - 1e-12, 1 + 1e-12, 1 + 0.9e-5, 1 - 0.9e-5,
                      1 + 1.1e-5, 0.5, 1.0, 1.5, 0.0], B)
    q = (z[pick].astype(np.float64) + (rel * r[pick].astype(np.float64))[:, None] * v).astype(np.float32)
    q[5] = np.nan
    q[6] = z[3]                                   # at the duplicated centre
    q[8] = z[11]                                  # at a centre with r = 0
    q[9] = z[12]                                  # at a centre with r < 0
    return q, z, r, lab


@pytest.mark.parametrize("d,store", [(32, "f32"), (128, "f32"), (256, "bf16")])
def test_blocked_equals_definition_near_boundaries(d, store):
    q, z, r, lab = adversarial(d, store=store)
    a = oracle.lookup(q, z, r, lab)
    b = oracle.lookup_blocked(q, z, r, lab, q_chunk=64, n_chunk=128)
    assert same(a, b)
    assert a.n_band.sum() > 10 and a.flagged.any() and (a.index >= 0).sum() > 50
    assert a.index[6] == 3 and a.label[5] == oracle.MISS


def test_blocked_equals_definition_on_tiny_workload():
    wl = wlmod.make_workload("tiny-d64-c10", seed=0)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig)
    st = oracle.CacheState(d=64, capacity=wl.z.shape[0])
    oracle.insert(st, wl.z, cert.label, cert.r)
    draws = wlmod.draw_queries(wl, 0, batch=256)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    a = oracle.lookup(zq, st.z, st.r, st.label)
    b = oracle.lookup_blocked(zq, st.z, st.r, st.label, n_chunk=1000)
    assert same(a, b)
    assert 0.15 < (a.index >= 0).mean() < 0.4


@pytest.mark.parametrize("name", ["mix-d128-c10", "mix-d128-c100", "mix-d256-c200", "stream-d256-c200-bf16"])
def test_blocked_equals_definition_on_workload_sub_blocks(name):
    cfg = wlmod.CONFIGS[name]
    wl = wlmod.make_workload(cfg, seed=0, n_cache=3000)
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig, store=cfg.store_dtype)
    st = oracle.CacheState(d=cfg.d, capacity=3000, store=cfg.store_dtype)
    oracle.insert(st, wl.z, cert.label, cert.r)
    draws = wlmod.draw_queries(wl, 0, batch=160)
    idx = wlmod.near_indices(draws, st.n)
    zq = wlmod.compose_queries(draws, st.z[idx], st.r[idx])
    a = oracle.lookup(zq, st.z, st.r, st.label)
    b = oracle.lookup_blocked(zq, st.z, st.r, st.label, q_chunk=48, n_chunk=700)
    assert same(a, b)
    assert (a.index >= 0).sum() > 20


def test_blocked_empty_inputs():
    z = np.zeros((0, 32), np.float32)
    q = np.ones((3, 32), np.float32)
    out = oracle.lookup_blocked(q, z, np.zeros(0, np.float32), np.zeros(0, np.int32))
    assert np.all(out.label == oracle.MISS) and np.all(np.isinf(out.dist2))
    out = oracle.lookup_blocked(np.zeros((0, 32), np.float32), np.ones((4, 32), np.float32),
                                np.ones(4, np.float32), np.zeros(4, np.int32))
    assert out.label.size == 0


def _mutated_blocked(old, new):
    """A copy of lookup_blocked with one expression replaced (planted on the CPU)."""
    src = inspect.getsource(base.lookup_blocked)
    assert old in src
    ns = dict(vars(base))
    exec(compile(src.replace(old, new), "<mutant>", "exec"), ns)
    return ns["lookup_blocked"]


@pytest.mark.parametrize("mutant", ["negative_slack", "no_live_mask", "sign"])
def test_blocked_mutants_are_caught(monkeypatch, mutant):
    """A prefilter that drops true hits or admits dead entries breaks the equality above."""
    q, z, r, lab = adversarial(128)
    a = oracle.lookup(q, z, r, lab)
    if mutant == "negative_slack":
        monkeypatch.setattr(base, "prefilter_rel", lambda d: -1e-3)
        fn = base.lookup_blocked
    elif mutant == "no_live_mask":
        fn = _mutated_blocked("b[~live[ns:ne]] = np.inf", "pass")
    else:
        fn = _mutated_blocked("G -= b[None, :]", "G += b[None, :]")
    assert not same(a, fn(q, z, r, lab))
