"""The synchronous calls from several host threads at once.

lipcache_spectral_norm, lipcache_insert and lipcache_lookup_indexed read a
few bytes back to the host through slots of one pinned buffer that the
library shares between calls.  Here eight threads, each on its own stream
(default priority), run them concurrently many times; every result must
equal the one the same call gives when run alone.
"""
import math
import threading

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import build_cache, gpu, host, oracle_cache, say
from paper_2608_13144_amd import api

pytestmark = pytest.mark.gpu

THREADS = 8
REPS = 12


def _head(seed, C, d):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((C, d)) / math.sqrt(d)).astype(np.float32)


def test_concurrent_synchronous_calls():
    say("synchronous calls from", THREADS, "threads")
    d, N, B, C = 64, 6000, 256, 7
    rng = np.random.default_rng(3)
    mu = 2.0 * rng.standard_normal((C, d))
    z = (mu[rng.integers(0, C, N)] + 0.5 * rng.standard_normal((N, d))).astype(np.float32)
    W0 = _head(1, C, d)
    sig = oracle.spectral_norm(W0).sigma
    cert = oracle.certify(z, W0, None, sig)
    st = oracle_cache(z, cert.label, cert.r, d)
    zq = (st.z[rng.integers(0, st.n, B)] + 0.05 * rng.standard_normal((B, d))).astype(np.float32)

    # per-thread inputs and the answers each call gives alone
    heads = [gpu(_head(100 + t, 10 + t, 48 + 16 * (t % 3))) for t in range(THREADS)]
    sigma_alone = [api.spectral_norm(W).sigma for W in heads]
    caches = [build_cache(st, capacity=st.n + 2 * B) for _ in range(THREADS)]
    n0 = caches[0].n
    lab = torch.full((B,), -1, dtype=torch.int32, device="cuda:0")
    sel = lab.clone()
    sel[::3] = 0        # a third of the rows are "hits" and are not appended
    r = gpu(np.full(B, 0.5, np.float32))
    zq_t = gpu(zq)
    got_alone = caches[0].insert(zq_t, lab, r, sel)
    caches[0].n = n0
    # every cache holds the same rows and index builds are deterministic, so
    # every thread's indexed lookup must give the lone call's answers
    indexes = [c.build_index(16, 2) for c in caches]
    ref, pairs_alone = caches[0].lookup_indexed(indexes[0], zq_t)
    ref = [host(x).copy() for x in (ref.label, ref.index, ref.dist2)]
    torch.cuda.synchronize()

    errors = []

    def work(t):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                c = caches[t]
                for _ in range(REPS):
                    sg = api.spectral_norm(heads[t]).sigma
                    if sg != sigma_alone[t]:
                        errors.append(f"thread {t}: sigma {sg} vs {sigma_alone[t]}")
                    got = c.insert(zq_t, lab, r, sel)
                    c.n = n0
                    if got != got_alone:
                        errors.append(f"thread {t}: inserted {got} vs {got_alone}")
                    res, pairs = c.lookup_indexed(indexes[t], zq_t)
                    if pairs != pairs_alone:
                        errors.append(f"thread {t}: pairs {pairs} vs {pairs_alone}")
                    for a, b, f in zip((res.label, res.index, res.dist2), ref, ("label", "index", "dist2")):
                        if not np.array_equal(a.cpu().numpy(), b):
                            errors.append(f"thread {t}: indexed lookup {f} differs")
                s.synchronize()
        except Exception as e:  # reported below, on the test's thread
            errors.append(f"thread {t}: {e!r}")

    threads = [threading.Thread(target=work, args=(t,)) for t in range(THREADS)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not any(th.is_alive() for th in threads), "a thread did not finish"
    torch.cuda.synchronize()
    assert not errors, errors[:5]
    say("threads done: sigma, insert and indexed lookup agree with the lone calls")
