"""Plant plausible mistakes in a copy of the CPU oracle and check a pin fails.

This shows the pins are strong enough: a dropped sqrt 2, a wrong sign, a
transposed operand, a non-strict hit test, nearest-entry instead of
nearest-hit, truncating bfloat16 conversion, ... are each caught by at least
one check in ``pins.py``.  The mistakes are planted in the oracle, on the CPU.
"""
import types

import numpy as np
import pytest

import oracle
import pins
from oracle import lipcache_oracle as base


def _copy(**over):
    ns = types.SimpleNamespace(**{k: getattr(oracle, k) for k in dir(oracle) if not k.startswith("__")})
    for k, v in over.items():
        setattr(ns, k, v)
    return ns


def _certify_with(radius=None, margin=None, logits=None, tie_high=False):
    def certify(z, W, b, sigma, store="f32", radius_mode="conservative"):
        out = base.certify(z, W, b, sigma, store, radius_mode)
        s = out.logits if logits is None else logits(out.stored, W, b)
        if tie_high:
            lab = s.shape[1] - 1 - np.argmax(s[:, ::-1], axis=1)
        else:
            lab = np.argmax(s, axis=1)
        rows = np.arange(s.shape[0])
        top1 = s[rows, lab]
        oth = s.copy()
        oth[rows, lab] = -np.inf
        top2 = oth.max(axis=1)
        m = (top1 - top2) if margin is None else margin(s, top1, top2)
        r64 = m / (sigma * base.SQRT2) if radius is None else radius(m, sigma)
        if radius_mode == "tight":
            r64 = out.r64
        return base.Certified(lab.astype(np.int32), r64.astype(np.float32), r64, m,
                              out.norm2, out.stored, s)
    return certify


def _spectral_fro(W, max_iters=20000, rel_tol=1e-13, seed=0):
    A = np.asarray(W, np.float64)
    s = float(np.linalg.norm(A))
    if s == 0:
        raise base.DegenerateHead("zero")
    return base.SpectralNorm(s, 1, max_iters > 1)


def _spectral_max_row(W, max_iters=20000, rel_tol=1e-13, seed=0):
    A = np.asarray(W, np.float64)
    s = float(np.max(np.linalg.norm(A, axis=1)))
    if s == 0:
        raise base.DegenerateHead("zero")
    return base.SpectralNorm(s, 1, max_iters > 1)


def _spectral_few_iters(W, max_iters=20000, rel_tol=1e-13, seed=0):
    return base.spectral_norm(W, max_iters=min(max_iters, 3), rel_tol=rel_tol, seed=seed)


def _lookup_variant(nonstrict=False, nearest_entry=False, ignore_sign=False, tie_high=False):
    def lookup(zq, cache_z, cache_r, cache_label, band_rel=base.BAND_REL):
        Q = np.asarray(zq, np.float64)
        Z = np.asarray(cache_z, np.float64)
        r = np.asarray(cache_r, np.float32).astype(np.float64)
        lab = np.asarray(cache_label, np.int32)
        B = Q.shape[0]
        L = np.full(B, base.MISS, np.int32)
        I = np.full(B, -1, np.int64)
        D = np.full(B, np.inf)
        for q in range(B):
            if Z.shape[0] == 0:
                continue
            d2 = np.sum((Z - Q[q]) ** 2, axis=1)
            live = np.ones_like(r, bool) if ignore_sign else r > 0
            hit = live & ((d2 <= r * r) if nonstrict else (d2 < r * r))
            if nearest_entry:
                i = int(np.argmin(d2))
                if hit[i]:
                    L[q], I[q], D[q] = lab[i], i, d2[i]
                continue
            if hit.any():
                best = d2[hit].min()
                cand = np.flatnonzero(hit & (d2 == best))
                i = int(cand[-1] if tie_high else cand[0])
                L[q], I[q], D[q] = lab[i], i, d2[i]
        z0 = np.zeros(B, np.int64)
        return base.LookupResult(L, I, D, z0, z0, np.zeros(B, bool))
    return lookup


def _bf16_truncate(x):
    a = np.ascontiguousarray(np.asarray(x, np.float32))
    return (a.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32).reshape(a.shape)


def _insert_variant(keep_nonpositive=False, ignore_selector=False, reverse=False):
    def insert(state, z_src, label_src, r_src, selector=None):
        zs = np.asarray(z_src, np.float32)
        rs = np.asarray(r_src, np.float32)
        ls = np.asarray(label_src, np.int32)
        take = np.ones(rs.shape, bool) if keep_nonpositive else rs > 0
        if selector is not None and not ignore_selector:
            take &= np.asarray(selector) == base.MISS
        idx = np.flatnonzero(take)
        if reverse:
            idx = idx[::-1]
        if state.n + idx.size > state.capacity:
            raise base.CapacityError("full")
        st = base.stored_values(zs[idx], state.store)
        state.z = np.concatenate([state.z, st])
        state.r = np.concatenate([state.r, rs[idx]])
        state.label = np.concatenate([state.label, ls[idx]])
        state.norm2 = np.concatenate([state.norm2, np.sum(st.astype(np.float64) ** 2, axis=1)])
        return int(idx.size)
    return insert


MUTANTS = {
    "radius without sqrt2": dict(certify=_certify_with(radius=lambda m, s: m / s)),
    "radius times sigma": dict(certify=_certify_with(radius=lambda m, s: m * s / base.SQRT2)),
    "margin sign flipped": dict(certify=_certify_with(margin=lambda s, t1, t2: t2 - t1)),
    "margin against the smallest logit": dict(
        certify=_certify_with(margin=lambda s, t1, t2: t1 - s.min(axis=1))),
    "bias dropped": dict(certify=_certify_with(
        logits=lambda z, W, b: base.logits_of(z, W, None))),
    "head transposed": dict(certify=_certify_with(
        logits=lambda z, W, b: base.logits_of(z, np.asarray(W).T, b))),
    "argmax ties to highest index": dict(certify=_certify_with(tie_high=True)),
    "spectral norm = Frobenius": dict(spectral_norm=_spectral_fro),
    "spectral norm = largest row norm": dict(spectral_norm=_spectral_max_row),
    "power iteration stopped early": dict(spectral_norm=_spectral_few_iters),
    "hit test not strict": dict(lookup=_lookup_variant(nonstrict=True)),
    "nearest entry instead of nearest hit": dict(lookup=_lookup_variant(nearest_entry=True)),
    "negative radii accepted": dict(lookup=_lookup_variant(ignore_sign=True)),
    "distance ties to highest index": dict(lookup=_lookup_variant(tie_high=True)),
    "bf16 by truncation": dict(bf16_round=_bf16_truncate),
    "insert keeps r <= 0": dict(insert=_insert_variant(keep_nonpositive=True)),
    "insert ignores selector": dict(insert=_insert_variant(ignore_selector=True)),
    "insert reverses order": dict(insert=_insert_variant(reverse=True)),
}


def _some_pin_fails(ns) -> bool:
    for pin in pins.ALL_PINS:
        try:
            pin(ns)
        except Exception:
            return True
    return False


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    over = dict(MUTANTS[name])
    if "bf16_round" in over:
        trunc = over["bf16_round"]

        def stored_values(z, store):
            z32 = np.asarray(z, np.float32)
            return z32.copy() if store == "f32" else trunc(z32)
        over.setdefault("stored_values", stored_values)
    assert _some_pin_fails(_copy(**over)), f"no pin catches: {name}"


def test_unmutated_oracle_passes_every_pin():
    assert not _some_pin_fails(_copy())
