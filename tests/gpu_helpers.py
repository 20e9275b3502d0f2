"""Helpers shared by the GPU test modules (device transfers, cache set-up, comparison)."""
import sys

import numpy as np
import torch

import oracle
from paper_2608_13144_amd import api

DEV = "cuda:0"


def say(*a):
    print("[gpu-test]", *a, file=sys.stderr, flush=True)


def gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def build_cache(state: "oracle.CacheState", capacity=None, store=None, image=True):
    """GPU cache holding the same rows as an oracle state (inserted through the HIP path)."""
    store = store or state.store
    cap = capacity or max(state.n, 1)
    c = api.LipCache(state.d, cap, store=store, device=DEV, image=image)
    if state.n:
        got = c.insert(gpu(state.z.astype(np.float32)), gpu(state.label), gpu(state.r))
        assert got == state.n
    return c


def oracle_cache(z, label, r, d, store="f32", capacity=None):
    st = oracle.CacheState(d=d, capacity=capacity or max(len(r), 1), store=store)
    oracle.insert(st, z, label, r)
    return st


def compare_lookup(res_gpu, ref, what, rows=None):
    """GPU answers (at ``rows`` of the batch, default all) against the oracle's for those rows."""
    lab = host(res_gpu.label)
    idx = host(res_gpu.index)
    d2 = host(res_gpu.dist2)
    if rows is not None:
        lab, idx, d2 = lab[rows], idx[rows], d2[rows]
    ok = ~ref.flagged
    nflag = int(ref.flagged.sum())
    bad_lab = np.flatnonzero(ok & (lab != ref.label))
    bad_idx = np.flatnonzero(ok & (idx != ref.index))
    assert bad_lab.size == 0, f"{what}: label mismatch at {bad_lab[:10]} gpu={lab[bad_lab[:10]]} ref={ref.label[bad_lab[:10]]}"
    assert bad_idx.size == 0, f"{what}: index mismatch at {bad_idx[:10]}"
    hit = ok & (ref.index >= 0)
    if hit.any():
        rel = np.abs(d2[hit].astype(np.float64) - ref.dist2[hit]) / np.maximum(ref.dist2[hit], 1e-300)
        assert rel.max() <= 1e-5, f"{what}: dist2 rel err {rel.max()}"
    assert np.all(np.isinf(d2[ok & (ref.index < 0)]))
    return nflag


def check_hits_valid(res_gpu, zq, state, W, b, what, band_rel=1e-5):
    """Properties of every hit in the batch, at any size.

    Each returned index is a live entry whose ball holds the query (D^2 < r^2
    in float64 on the stored values, or a pair in the boundary band), the
    label is that entry's payload, the distance is the pair's, and - the
    certified-consistency property of the radius (Lemma 5.1) - the head's
    argmax at the query equals the returned label.
    """
    lab = host(res_gpu.label)
    idx = host(res_gpu.index)
    d2 = host(res_gpu.dist2)
    hit = idx >= 0
    assert np.array_equal(hit, lab >= 0), what
    if not hit.any():
        return 0
    qi = np.flatnonzero(hit)
    e = idx[qi]
    assert e.max() < state.n, what
    Q = zq[qi].astype(np.float64)
    D2 = np.sum((state.z[e].astype(np.float64) - Q) ** 2, axis=1)
    r = state.r[e].astype(np.float64)
    inside = D2 < r * r
    band = np.abs(np.sqrt(D2) - r) <= band_rel * r
    assert np.all(inside | band), f"{what}: {int((~inside & ~band).sum())} hits outside their ball"
    assert np.array_equal(lab[qi], state.label[e]), what
    rel = np.abs(d2[qi].astype(np.float64) - D2) / np.maximum(D2, 1e-300)
    assert rel.max() <= 1e-5, f"{what}: dist2 rel {rel.max()}"
    s = oracle.logits_of(zq[qi], W, b)
    assert np.array_equal(np.argmax(s, axis=1).astype(np.int32), lab[qi]), f"{what}: certified consistency"
    return int(qi.size)
