"""Checks that pin the CPU oracle to facts other than its own code.

Each ``pin_*`` takes an oracle-like namespace (the real ``oracle`` module, or a
deliberately broken copy in the mutation tests) and raises AssertionError
when the oracle disagrees with what the paper and the mathematics fix:

* sigma_max(W) against a one-sided Jacobi SVD written here, numpy's SVD and
  closed forms (diagonal, rank one, two rows, scaled orthonormal rows);
* the radius against the antipodal two-class head, whose conservative ball is
  exactly the distance to the decision boundary (Eq. (21) is tight there);
* Lemma 5.1 (Sec. 5.2): uniform samples inside every ball and the worst-case
  directions at (1 - 1e-9) r keep the head's argmax;
* Remark 5.1: r_{i,j} equals the distance to the hyperplane f_y = f_j found by
  bisection, and r* >= r;
* lookup (Eq. (13)-(15)) against hand cases with exact binary values and
  pure-Python brute force on tiny inputs;
* insert against order, selection and capacity rules, and bfloat16 rounding
  against hand values and torch's conversion.

Nothing here imports the HIP path.
"""
from __future__ import annotations

import math

import numpy as np

MISS = -1


# ------------------------------------------------------------ independent helpers
def jacobi_singular_values(A, tol: float = 1e-15, max_sweeps: int = 60) -> np.ndarray:
    """Singular values by one-sided (Hestenes) Jacobi rotations, descending."""
    U = np.array(A, dtype=np.float64)
    if U.shape[1] > U.shape[0]:
        U = U.T.copy()
    n = U.shape[1]
    for _ in range(max_sweeps):
        worst = 0.0
        for p in range(n - 1):
            for q in range(p + 1, n):
                a = float(U[:, p] @ U[:, p])
                b = float(U[:, q] @ U[:, q])
                g = float(U[:, p] @ U[:, q])
                if a == 0.0 or b == 0.0:
                    continue
                rel = abs(g) / math.sqrt(a * b)
                worst = max(worst, rel)
                if rel <= tol:
                    continue
                zeta = (b - a) / (2.0 * g)
                t = math.copysign(1.0, zeta) / (abs(zeta) + math.sqrt(1.0 + zeta * zeta))
                c = 1.0 / math.sqrt(1.0 + t * t)
                s = c * t
                up = U[:, p].copy()
                U[:, p] = c * up - s * U[:, q]
                U[:, q] = s * up + c * U[:, q]
        if worst <= tol:
            break
    return np.sort(np.sqrt(np.sum(U * U, axis=0)))[::-1]


def brute_lookup(Q, Z, r, lab):
    """Pure-Python loops: nearest entry among those with ||q - z|| < r."""
    out = []
    for q in Q:
        best = None
        for i, (z, ri) in enumerate(zip(Z, r)):
            d2 = 0.0
            for a, b in zip(q, z):
                d2 += (float(a) - float(b)) ** 2
            if float(ri) > 0.0 and math.sqrt(d2) < float(ri):
                if best is None or d2 < best[0]:
                    best = (d2, i)
        out.append((MISS, -1) if best is None else (int(lab[best[1]]), best[1]))
    return out


def argmax_head(W, b, x):
    s = np.asarray(W, np.float64) @ np.asarray(x, np.float64)
    if b is not None:
        s = s + np.asarray(b, np.float64)
    return int(np.argmax(s))


def uniform_in_ball(rng, centre, radius, count):
    d = centre.shape[0]
    v = rng.standard_normal((count, d))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    rad = radius * rng.random(count) ** (1.0 / d)
    return centre[None, :] + rad[:, None] * v


def boundary_distance_by_bisection(W, b, z, y, j, direction, hi):
    """Distance along ``direction`` from z to where logit y stops beating logit j."""
    def gap(t):
        x = z + t * direction
        s = np.asarray(W, np.float64) @ x + (0 if b is None else np.asarray(b, np.float64))
        return s[y] - s[j]
    lo_t, hi_t = 0.0, hi
    assert gap(lo_t) > 0 and gap(hi_t) < 0
    for _ in range(200):
        mid = 0.5 * (lo_t + hi_t)
        if gap(mid) > 0:
            lo_t = mid
        else:
            hi_t = mid
    return 0.5 * (lo_t + hi_t)


# ----------------------------------------------------------------------- pins
def pin_spectral_closed_forms(orc):
    # diagonal: sigma = max |s|
    W = np.diag([0.5, -3.25, 2.0]).astype(np.float32)
    assert abs(orc.spectral_norm(W).sigma - 3.25) <= 1e-12 * 3.25
    # rank one a b^T: sigma = ||a|| ||b||
    rng = np.random.default_rng(1)
    a = rng.standard_normal(7).astype(np.float32)
    bb = rng.standard_normal(12).astype(np.float32)
    W = np.outer(a, bb).astype(np.float32)
    ref = float(np.linalg.norm(W.astype(np.float64), "fro"))   # rank one: Frobenius = spectral
    assert abs(orc.spectral_norm(W).sigma - ref) <= 1e-12 * ref
    # two rows: sigma^2 = (g11+g22)/2 + sqrt(((g11-g22)/2)^2 + g12^2), G = W W^T
    W = rng.standard_normal((2, 9)).astype(np.float32)
    A = W.astype(np.float64)
    g11, g22, g12 = A[0] @ A[0], A[1] @ A[1], A[0] @ A[1]
    ref = math.sqrt((g11 + g22) / 2 + math.sqrt(((g11 - g22) / 2) ** 2 + g12 ** 2))
    assert abs(orc.spectral_norm(W).sigma - ref) <= 1e-12 * ref
    # c Q with orthonormal rows: sigma = |c|
    Qm, _ = np.linalg.qr(rng.standard_normal((16, 5)))
    W = 1.75 * Qm.T
    assert abs(orc.spectral_norm(W).sigma - 1.75) <= 1e-12
    # the antipodal head [[1,0..],[-1,0..]] has sigma = sqrt 2
    W = np.zeros((2, 4), np.float32)
    W[0, 0], W[1, 0] = 1.0, -1.0
    assert abs(orc.spectral_norm(W).sigma - math.sqrt(2.0)) <= 1e-13
    # W = 0 is degenerate: Alg. 1 stops
    try:
        orc.spectral_norm(np.zeros((3, 4), np.float32))
    except ValueError:
        pass
    else:
        raise AssertionError("zero head must be reported as degenerate")
    # one iteration cannot report convergence
    W = rng.standard_normal((6, 8)).astype(np.float32)
    assert not orc.spectral_norm(W, max_iters=1).converged


def pin_spectral_vs_jacobi(orc):
    rng = np.random.default_rng(2)
    for C, d in [(2, 2), (3, 5), (10, 16), (16, 16), (16, 7), (5, 1)]:
        W = (rng.standard_normal((C, d)) / math.sqrt(d)).astype(np.float32)
        sj = jacobi_singular_values(W)[0]
        sn = float(np.linalg.svd(W.astype(np.float64), compute_uv=False)[0])
        assert abs(sj - sn) <= 1e-12 * sn, (C, d, sj, sn)
        res = orc.spectral_norm(W)
        assert res.converged
        assert abs(res.sigma - sj) <= 1e-10 * sj, (C, d, res.sigma, sj)


def pin_jacobi_itself():
    """The Jacobi helper on closed forms (so the pin is not pinned to itself)."""
    s = jacobi_singular_values(np.diag([1.0, -4.0, 2.5]))
    assert np.allclose(s, [4.0, 2.5, 1.0], rtol=0, atol=1e-14)
    a, b = np.array([1.0, 2.0, 2.0]), np.array([3.0, 4.0])
    s = jacobi_singular_values(np.outer(a, b))
    assert abs(s[0] - 15.0) <= 1e-13 and abs(s[1]) <= 1e-13


def pin_certify_hand(orc):
    # W = I, b = 0, sigma = 1: logits = z; label = argmax; m = top1 - top2; r = m / sqrt 2
    W = np.eye(3, 4, dtype=np.float32)
    z = np.array([[3.0, 1.0, 2.0, 9.0],      # label 0, m = 1
                  [2.0, 2.0, 1.0, 0.0],      # tie -> lowest index 0, m = 0 -> r = 0
                  [-1.0, 0.5, -4.0, 0.0]],   # label 1, m = 1.5
                 dtype=np.float32)
    out = orc.certify(z, W, None, 1.0)
    assert list(out.label) == [0, 0, 1]
    assert np.allclose(out.margin, [1.0, 0.0, 1.5], rtol=0, atol=0)
    assert np.allclose(out.r64, [1.0 / math.sqrt(2), 0.0, 1.5 / math.sqrt(2)], rtol=1e-15, atol=0)
    assert out.r[1] <= 0.0
    assert np.allclose(out.norm2, [95.0, 9.0, 17.25], rtol=0, atol=0)
    # the bias shifts logits: b = (0, 3, 0) moves row 0 to label 1, m = 1
    out = orc.certify(z, W, np.array([0.0, 3.0, 0.0], np.float32), 1.0)
    assert list(out.label) == [1, 1, 1] and out.margin[0] == 1.0
    # sigma scales the radius inversely
    out2 = orc.certify(z, W, None, 4.0)
    assert np.allclose(out2.r64[0], 1.0 / (4.0 * math.sqrt(2)), rtol=1e-15)


def pin_certify_two_class_closed_form(orc):
    rng = np.random.default_rng(3)
    d = 32
    W = rng.standard_normal((2, d)).astype(np.float32)
    b = rng.standard_normal(2).astype(np.float32)
    z = rng.standard_normal((50, d)).astype(np.float32)
    out = orc.certify(z, W, b, 2.0)
    A = W.astype(np.float64)
    m = np.abs(z.astype(np.float64) @ (A[0] - A[1]) + float(b[0]) - float(b[1]))
    assert np.allclose(out.margin, m, rtol=1e-12, atol=1e-12)
    lab = (z.astype(np.float64) @ (A[1] - A[0]) + float(b[1]) - float(b[0]) > 0).astype(int)
    assert np.array_equal(out.label, lab)


def pin_certify_antipodal_tightness(orc):
    """W = [[1,0,...],[-1,0,...]]: sigma = sqrt 2 and r = |x| is the boundary distance."""
    d = 64
    W = np.zeros((2, d), np.float32)
    W[0, 0], W[1, 0] = 1.0, -1.0
    sigma = orc.spectral_norm(W).sigma
    xs = np.array([0.75, 1.5, 3.0, 0.125], np.float64)
    z = np.zeros((xs.size, d), np.float32)
    z[:, 0] = xs
    z[:, 5] = 0.25       # coordinates off the head's row space do not matter
    out = orc.certify(z, W, None, sigma)
    assert np.all(out.label == 0)
    assert np.allclose(out.r64, xs, rtol=1e-13, atol=0)
    for x, r in zip(xs, out.r64):
        inside = np.zeros(d)
        inside[0] = x - (1 - 1e-9) * r
        outside = np.zeros(d)
        outside[0] = x - (1 + 1e-9) * r
        assert argmax_head(W, None, inside) == 0
        assert argmax_head(W, None, outside) == 1


def pin_certify_lemma(orc):
    """Lemma 5.1: inside every conservative ball the head's argmax is y_i."""
    rng = np.random.default_rng(4)
    for C, d, scale in [(3, 8, 1.0), (10, 32, 2.0), (7, 16, 0.3), (6, 6, 1.0)]:
        W = (rng.standard_normal((C, d)) / math.sqrt(d)).astype(np.float32)
        b = (0.1 * rng.standard_normal(C)).astype(np.float32)
        z = (scale * rng.standard_normal((40, d))).astype(np.float32)
        sigma = orc.spectral_norm(W).sigma
        out = orc.certify(z, W, b, sigma)
        A = W.astype(np.float64)
        for i in range(z.shape[0]):
            y, r = int(out.label[i]), float(out.r64[i])
            if out.margin[i] < 1e-6:
                continue
            centre = z[i].astype(np.float64)
            assert argmax_head(W, b, centre) == y
            for x in uniform_in_ball(rng, centre, r, 64):
                assert argmax_head(W, b, x) == y
            for j in range(C):
                if j == y:
                    continue
                v = A[j] - A[y]
                v /= np.linalg.norm(v)
                assert argmax_head(W, b, centre + (1 - 1e-9) * r * v) == y
        # the radius cannot be the trivial one
        assert np.all(out.r64[out.margin > 0] > 0)


def pin_certify_tight(orc):
    """Remark 5.1: r_{i,j} is the hyperplane distance, r* >= r, and r* is reached."""
    rng = np.random.default_rng(5)
    C, d = 5, 12
    W = (rng.standard_normal((C, d)) / math.sqrt(d)).astype(np.float32)
    b = (0.1 * rng.standard_normal(C)).astype(np.float32)
    z = rng.standard_normal((12, d)).astype(np.float32)
    sigma = orc.spectral_norm(W).sigma
    cons = orc.certify(z, W, b, sigma)
    tight = orc.certify(z, W, b, sigma, radius_mode="tight")
    assert np.array_equal(cons.label, tight.label)
    assert np.all(tight.r64 >= cons.r64 * (1 - 1e-12))
    A = W.astype(np.float64)
    for i in range(z.shape[0]):
        y = int(tight.label[i])
        centre = z[i].astype(np.float64)
        dists = []
        for j in range(C):
            if j == y:
                continue
            v = A[j] - A[y]
            v /= np.linalg.norm(v)
            dists.append(boundary_distance_by_bisection(W, b, centre, y, j, v, hi=1e3))
        assert abs(min(dists) - tight.r64[i]) <= 1e-9 * max(1.0, tight.r64[i])
    # equal rows put no finite constraint on that pair
    W2 = np.stack([W[0], W[1], W[1]]).astype(np.float32)
    b2 = np.array([0.0, 0.0, -1.0], np.float32)
    zz = (5.0 * A[1] / np.linalg.norm(A[1]))[None, :].astype(np.float32)
    t2 = orc.certify(zz, W2, b2, orc.spectral_norm(W2).sigma, radius_mode="tight")
    assert int(t2.label[0]) == 1
    assert np.isfinite(t2.r64[0])


def _lookup_basic(orc, Q, Z, r, lab):
    res = orc.lookup(np.asarray(Q, np.float32), np.asarray(Z, np.float32),
                     np.asarray(r, np.float32), np.asarray(lab, np.int32))
    return list(zip(res.label.tolist(), res.index.tolist())), res


def pin_lookup_hand(orc):
    d = 32
    e1 = np.zeros(d)
    e1[0] = 1.0
    Z = np.zeros((1, d))
    # entry 0 at the origin with r = 1: D = r exactly is a miss (strict, Eq. (13))
    got, res = _lookup_basic(orc, [e1, 0.75 * e1], Z, [1.0], [7])
    assert got == [(MISS, -1), (7, 0)]
    assert res.dist2[1] == 0.5625
    # nearest hit, not nearest entry (Eq. (14)): A at distance 1 with r = 0.5 is
    # not a hit; B at distance 2 with r = 3 is.
    Z = np.stack([e1 * 1.0, e1 * -2.0])
    got, _ = _lookup_basic(orc, [np.zeros(d)], Z, [0.5, 3.0], [1, 2])
    assert got == [(2, 1)]
    # among hits the nearest wins
    Z = np.stack([e1 * 1.0, e1 * -0.5, e1 * 0.25])
    got, _ = _lookup_basic(orc, [np.zeros(d)], Z, [4.0, 4.0, 0.125], [1, 2, 3])
    assert got == [(2, 1)]
    # duplicate entries: the lower index wins
    Z = np.stack([e1, e1, e1 * 0.5, e1 * 0.5])
    got, _ = _lookup_basic(orc, [e1 * 0.5], Z, [1.0, 1.0, 1.0, 1.0], [4, 5, 6, 7])
    assert got == [(6, 2)]
    # a non-positive radius is never a hit
    got, _ = _lookup_basic(orc, [np.zeros(d)], np.zeros((2, d)), [0.0, -1.0], [1, 2])
    assert got == [(MISS, -1)]
    # empty cache: every query misses
    got, _ = _lookup_basic(orc, [np.zeros(d), e1], np.zeros((0, d)), [], [])
    assert got == [(MISS, -1), (MISS, -1)]
    # a NaN query misses
    q = np.zeros(d)
    q[3] = np.nan
    got, _ = _lookup_basic(orc, [q], np.zeros((1, d)), [10.0], [1])
    assert got == [(MISS, -1)]


def pin_lookup_bruteforce(orc):
    rng = np.random.default_rng(6)
    for trial in range(4):
        d, N, B = 4, 24, 20
        Z = rng.standard_normal((N, d)).astype(np.float32)
        r = (0.9 * rng.random(N)).astype(np.float32)
        r[rng.random(N) < 0.1] = 0.0
        lab = rng.integers(0, 5, N).astype(np.int32)
        Q = (Z[rng.integers(0, N, B)] + 0.4 * rng.standard_normal((B, d))).astype(np.float32)
        got, res = _lookup_basic(orc, Q, Z, r, lab)
        assert got == brute_lookup(Q, Z, r, lab), trial
        for k, (l, i) in enumerate(got):
            if i >= 0:
                ref = sum((float(a) - float(b)) ** 2 for a, b in zip(Q[k], Z[i]))
                assert abs(res.dist2[k] - ref) <= 1e-15 * max(ref, 1.0)


def pin_lookup_band(orc):
    """Band bookkeeping: a pair at D = r (1 + 1e-7) is in the band and flags its query."""
    d = 32
    e1 = np.zeros(d)
    e1[0] = 1.0
    Z = np.zeros((2, d))
    Z[1] = 10.0 * e1
    res = orc.lookup(np.stack([1.0000001 * e1, 0.5 * e1, 5.0 * e1]).astype(np.float32),
                     Z.astype(np.float32), np.array([1.0, 1.0], np.float32),
                     np.array([3, 4], np.int32))
    assert res.n_band.tolist() == [1, 0, 0]
    assert res.flagged.tolist() == [True, False, False]


def pin_lookup_certified_consistency(orc, workload_module):
    """Every hit returns the head's own argmax at the query (Lemma 5.1, proxy payload)."""
    wl = workload_module.make_workload("tiny-d64-c10", seed=0, n_cache=1024)
    sigma = orc.spectral_norm(wl.W).sigma
    cert = orc.certify(wl.z, wl.W, wl.b, sigma)
    keep = cert.r > 0
    Zc, rc, lc = cert.stored[keep], cert.r[keep], cert.label[keep]
    draws = workload_module.draw_queries(wl, 0, batch=256)
    idx = workload_module.near_indices(draws, Zc.shape[0])
    zq = workload_module.compose_queries(draws, Zc[idx], rc[idx])
    res = orc.lookup(zq, Zc, rc, lc)
    hits = res.index >= 0
    assert hits.sum() > 20
    s = zq.astype(np.float64) @ wl.W.astype(np.float64).T + wl.b.astype(np.float64)
    assert np.array_equal(np.argmax(s, axis=1)[hits], res.label[hits])


def pin_bf16(orc):
    one = np.float32(1.0)
    vals = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -15, -(1 + 3 * 2 ** -8),
                     2 ** -8, 65504.0, 0.0, -0.0, 1 - 2 ** -9], np.float32)
    want = np.array([1.0, 1 + 2 ** -6, 1 + 2 ** -7, -(1 + 2 ** -6),
                     2 ** -8, 65536.0, 0.0, -0.0, 1.0], np.float32)
    got = orc.bf16_round(vals)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (got, want)
    assert one == 1.0
    import torch
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(orc.bf16_round(x).view(np.uint32), ref.view(np.uint32))


def pin_insert(orc):
    d = 32
    rng = np.random.default_rng(8)
    st = orc.CacheState(d=d, capacity=10)
    z = rng.standard_normal((6, d)).astype(np.float32)
    r = np.array([0.5, 0.0, 1.0, -2.0, 0.25, 3.0], np.float32)
    lab = np.arange(6, dtype=np.int32)
    sel = np.array([MISS, MISS, 4, MISS, MISS, MISS], np.int32)
    k = orc.insert(st, z, lab, r, sel)
    # rows 0, 4, 5 (row 1: r = 0, row 2: hit, row 3: r < 0), ascending order
    assert k == 3 and st.n == 3
    assert st.label.tolist() == [0, 4, 5]
    assert np.array_equal(st.z, z[[0, 4, 5]])
    assert np.allclose(st.norm2, np.sum(z[[0, 4, 5]].astype(np.float64) ** 2, axis=1), rtol=1e-15)
    # all-or-nothing capacity: 8 more rows do not fit into 7 free slots
    z2 = rng.standard_normal((8, d)).astype(np.float32)
    try:
        orc.insert(st, z2, np.zeros(8, np.int32), np.ones(8, np.float32))
    except ValueError:
        pass
    else:
        raise AssertionError("capacity overflow must fail")
    assert st.n == 3
    # a bfloat16 cache stores rounded values and their norms
    sb = orc.CacheState(d=d, capacity=4, store="bf16")
    zz = np.full((1, d), 1 + 3 * 2 ** -8, np.float32)
    orc.insert(sb, zz, np.zeros(1, np.int32), np.ones(1, np.float32))
    assert np.all(sb.z == np.float32(1 + 2 ** -6))
    assert sb.norm2[0] == d * (1 + 2 ** -6) ** 2


ALL_PINS = [
    pin_spectral_closed_forms,
    pin_spectral_vs_jacobi,
    pin_certify_hand,
    pin_certify_two_class_closed_form,
    pin_certify_antipodal_tightness,
    pin_certify_lemma,
    pin_certify_tight,
    pin_lookup_hand,
    pin_lookup_bruteforce,
    pin_lookup_band,
    pin_bf16,
    pin_insert,
]
