"""lipcache_lookup_noalloc captured into a HIP graph and replayed.

The allocation-free lookup is meant for callers that cannot allocate, code
under graph capture among them: every launch of a lookup reads its sizes
from the host, allocates nothing and clears its own workspace with its own
kernels (no memset or copy nodes).  Here one lookup is captured (torch's
graph API drives the capture on its stream), then replayed three times on
new queries written into the captured input buffer, with eager lookups and
synchronisations between the replays.  Each replay must give the eager
lipcache_lookup's answers on the same queries bit for bit (label, index,
d^2 bits, band flags and counters), and the first replay the oracle's.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import build_cache, compare_lookup, gpu, host, oracle_cache, say
from paper_2608_13144_amd import api

pytestmark = pytest.mark.gpu


def _mixture(d, N, B, store, seed, rounds, C=7):
    """A Gaussian-mixture cache and `rounds` batches of B queries: half near
    a ball (u r_i from a random entry, u ~ U(0, 2)), half fresh draws."""
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((C, d)) / math.sqrt(d)).astype(np.float32)
    mu = 2.0 * rng.standard_normal((C, d))
    z = (mu[rng.integers(0, C, N)] + 0.5 * rng.standard_normal((N, d))).astype(np.float32)
    sig = oracle.spectral_norm(W).sigma
    cert = oracle.certify(z, W, None, sig, store=store)
    st = oracle_cache(z, cert.label, cert.r, d, store=store)
    batches = []
    for _ in range(rounds):
        pick = rng.integers(0, st.n, B)
        v = rng.standard_normal((B, d))
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        zq = (st.z[pick].astype(np.float64) + (rng.uniform(0, 2, B) * st.r[pick])[:, None] * v).astype(np.float32)
        zq[1::2] = (mu[rng.integers(0, C, zq[1::2].shape[0])] + 0.5 * rng.standard_normal(zq[1::2].shape)).astype(
            np.float32)
        batches.append(zq)
    return st, batches


def _fields(res):
    return (res.label, res.index, res.dist2, res.stats, res.band)


@pytest.mark.parametrize("d,N,B,store,precision,prune", [
    (128, 5000, 517, "f32", "f16", False),
    (128, 5000, 517, "f32", "f32", False),
    (256, 3001, 300, "bf16", "f16", False),
    (256, 40000, 300, "f32", "f16", True),     # the pruned path (n >= 32768)
])
def test_noalloc_lookup_graph_replays(d, N, B, store, precision, prune):
    what = f"graph d={d} N={N} B={B} {store}/{precision} prune={prune}"
    say(what)
    st, batches = _mixture(d, N, B, store, seed=d + N + B, rounds=3)
    c = build_cache(st)
    if prune:
        assert c.lookup_prunes(precision)
    dev = torch.device("cuda:0")
    zq_static = gpu(batches[0]).clone()
    out = api.LookupResult(torch.empty(B, dtype=torch.int32, device=dev),
                           torch.empty(B, dtype=torch.int64, device=dev),
                           torch.empty(B, dtype=torch.float32, device=dev),
                           torch.zeros(4, dtype=torch.int64, device=dev),
                           torch.empty(B, dtype=torch.uint8, device=dev))
    # one eager call on a side stream first (the library looks its static
    # workspace up on a device's first call), as graph capture expects
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        c.lookup_noalloc(zq_static, precision=precision, out=out, prune=prune)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        c.lookup_noalloc(zq_static, precision=precision, out=out, prune=prune)
    torch.cuda.synchronize()
    for rnd, zq in enumerate(batches):
        zq_static.copy_(gpu(zq))
        ref = c.lookup(gpu(zq), precision=precision, prune=prune)   # eager, its own workspace and outputs
        torch.cuda.synchronize()
        for f in _fields(out):
            f.fill_(7)       # the replay must write every output
        graph.replay()
        torch.cuda.synchronize()
        for a, b, name in zip(_fields(out), _fields(ref), ("label", "index", "dist2", "stats", "band")):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"{what} replay {rnd}: {name} differs"
        if rnd == 0:
            compare_lookup(out, oracle.lookup_blocked(zq, st.z, st.r, st.label), f"{what} replay 0")
        say(what, "replay", rnd, "hits", int((host(out.label) >= 0).sum()), "stats", host(out.stats).tolist())
    del graph
