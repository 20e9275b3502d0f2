"""Plain, slow, fp64 CPU oracle of LipCache's certified cache path.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  The product path
(the HIP library and its Python binding) never calls it and shares no code
with it: nothing here is imported by, or imports, ``paper_2608_13144_amd``.

Every function writes out the paper's definition on the exact values the
device path consumes (float32 inputs, or their bfloat16-rounded values for a
bfloat16 cache), with float64 as the stand-in for exact arithmetic:

  * ``spectral_norm``  - sigma_max(W), the Lipschitz bound of the affine head
                         (Sec. 5.1, Eq. (18)-(19)); computed by power iteration
                         as construction step "compute sigma_max(W)" of Alg. 1.
  * ``certify``        - logits s = W z + b (Sec. 4.1, Eq. (5)), label = argmax
                         (Eq. (6)), margin m = s_y - max_{j != y} s_j (Eq. (20)),
                         conservative radius r = m / (sigma_max(W) sqrt 2)
                         (Eq. (21)); optional tight radius
                         r* = min_j (s_y - s_j) / ||W_y - W_j|| (Remark 5.1, Eq. (29)).
  * ``lookup``         - hit set H = {i : ||z - z_i|| < r_i} (Eq. (13)), nearest
                         hit i* (Eq. (14)), payload or miss (Eq. (15)).
  * ``lookup_blocked`` - the same answers with a float32 BLAS prefilter of
                         rigorous slack and the same float64 distances for
                         the survivors (for large test batches); pinned
                         bit-for-bit against ``lookup``.
  * ``insert``         - write-back of missed samples (Sec. 4.4, Alg. 2).
  * ``construct``      - offline construction of the feature store (Sec. 4.3,
                         Alg. 1): eligibility, budgets and the selection
                         strategies (radius-prioritised de-duplication,
                         caller priority / random, K-center).
  * ``cluster_pruned_lookup`` - ``lookup`` through a partition of the rows,
                         pruning clusters by the triangle inequality (the
                         exact sublinear index of Sec. 4.4); pinned equal to
                         ``lookup`` on every partition.
  * ``lookup_partitioned`` - every field of ``lookup`` (band counts and flags
                         too) through a partition, for full-size batches;
                         pinned equal to ``lookup`` on every partition and
                         at the band's edges.
  * ``boundary_radius``, ``consistency`` - the reuse boundaries compared in
                         Sec. 6 (scaled certified radius, global threshold,
                         inter-class empirical radius) and the
                         certified-consistency count.
  * ``bf16_round``     - round-to-nearest-even float32 -> bfloat16 (storage).

Pins: every function is checked in ``tests/`` against closed forms, brute
force on tiny inputs, Jacobi SVD, Lemma 5.1 and hand cases; see the tests.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

MISS = -1
BAND_REL = 1e-5          # relative width of the ball-boundary band
SQRT2 = float(np.sqrt(np.float64(2.0)))


class DegenerateHead(ValueError):
    """sigma_max(W) <= 0: Alg. 1 reports a degenerate head and stops."""


class CapacityError(ValueError):
    """Appending would exceed the cache budget; nothing is appended."""


# ---------------------------------------------------------------- bfloat16
def bf16_round(x) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), as float32.

    bfloat16 keeps the upper 16 bits of the float32 pattern; the discarded
    lower half decides the rounding: above half -> up, below -> down, exactly
    half -> towards the even upper half.  NaN stays NaN.
    """
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    bits = a.view(np.uint32).astype(np.uint64)
    upper = bits >> np.uint64(16)
    lower = bits & np.uint64(0xFFFF)
    half = np.uint64(0x8000)
    round_up = (lower > half) | ((lower == half) & ((upper & np.uint64(1)) == np.uint64(1)))
    upper = upper + round_up.astype(np.uint64)
    out = (upper << np.uint64(16)).astype(np.uint32).view(np.float32).copy()
    nan = np.isnan(a)
    out[nan] = a[nan]
    return out.reshape(a.shape)


def to_f32_toward_zero(x) -> np.ndarray:
    """float64 -> float32 rounded toward zero, so a stored radius never exceeds
    the certificate it comes from (Lemma 5.1 holds for any r' <= r)."""
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    over = np.abs(f.astype(np.float64)) > np.abs(x)
    f[over] = np.nextafter(f[over], np.float32(0.0))
    return f


def stored_values(z, store: str) -> np.ndarray:
    """The values a cache of dtype ``store`` ("f32" or "bf16") holds for z."""
    z32 = np.asarray(z, dtype=np.float32)
    if store == "f32":
        return z32.copy()
    if store == "bf16":
        return bf16_round(z32)
    raise ValueError(f"unknown store dtype {store!r}")


# ---------------------------------------------------------- spectral norm
@dataclass
class SpectralNorm:
    sigma: float
    iterations: int
    converged: bool


def spectral_norm(W, max_iters: int = 20000, rel_tol: float = 1e-13,
                  seed: int = 0) -> SpectralNorm:
    """sigma_max(W) by power iteration on W^T W, in float64.

    Alg. 1 computes sigma_max(W) before certifying any candidate; the head is
    sigma_max(W)-Lipschitz (Eq. (18)).  Start from a seeded Gaussian unit
    vector v.  Each iteration: u = W v, sigma_k = ||u|| (= ||W v|| with
    ||v|| = 1), w = W^T u, v = w / ||w||.  Converged once
    |sigma_k - sigma_{k-1}| <= rel_tol * sigma_k holds on two consecutive
    iterations.  Raises DegenerateHead when sigma <= 0 (Alg. 1: report and
    stop).
    """
    A = np.asarray(W, dtype=np.float64)
    if A.ndim != 2 or A.shape[0] < 1 or A.shape[1] < 1:
        raise ValueError("W must be a non-empty C x d matrix")
    rng = np.random.default_rng(seed)
    v = rng.standard_normal(A.shape[1])
    v /= np.linalg.norm(v)
    prev = None
    stable = 0
    sigma = 0.0
    for it in range(1, max_iters + 1):
        u = A @ v
        sigma = float(np.linalg.norm(u))
        w = A.T @ u
        nw = float(np.linalg.norm(w))
        if nw == 0.0 or sigma <= 0.0:
            raise DegenerateHead("sigma_max(W) <= 0: degenerate classification head")
        v = w / nw
        if prev is not None and abs(sigma - prev) <= rel_tol * sigma:
            stable += 1
            if stable >= 2:
                return SpectralNorm(sigma, it, True)
        else:
            stable = 0
        prev = sigma
    return SpectralNorm(sigma, max_iters, False)


# ----------------------------------------------------------------- certify
@dataclass
class Certified:
    label: np.ndarray      # int32, argmax of the logits (lowest index on ties)
    r: np.ndarray          # float32 radius, the float64 value rounded toward zero
    r64: np.ndarray        # float64 radius before rounding
    margin: np.ndarray     # float64 top-1 minus top-2 logit
    norm2: np.ndarray      # float64 squared norm of the stored feature
    stored: np.ndarray     # float32 values certified (bf16-rounded for a bf16 store)
    logits: np.ndarray     # float64 (N, C)


def logits_of(z, W, b=None) -> np.ndarray:
    """s(z) = W z + b for every row z (Eq. (5)), in float64."""
    Z = np.asarray(z, dtype=np.float64)
    A = np.asarray(W, dtype=np.float64)
    s = Z @ A.T
    if b is not None:
        s = s + np.asarray(b, dtype=np.float64)[None, :]
    return s


def certify(z, W, b, sigma: float, store: str = "f32",
            radius_mode: str = "conservative") -> Certified:
    """Label, margin and certified radius of every row of z.

    label y = argmax_c s_c (Eq. (6); lowest index on ties),
    margin m = s_y - max_{j != y} s_j (Eq. (20)),
    conservative radius r = m / (sigma sqrt 2) (Eq. (21)), or with
    ``radius_mode="tight"`` r* = min_{j != y} (s_y - s_j) / ||W_y - W_j||
    (Remark 5.1, Eq. (29)), where a competitor with W_y = W_j sets no finite
    constraint.  A radius <= 0 marks a candidate that construction discards
    (Alg. 1).  For a bfloat16 store the rounded feature is certified.
    """
    A = np.asarray(W, dtype=np.float32)
    C = A.shape[0]
    if C < 2:
        raise ValueError("the margin needs at least two classes")
    if not sigma > 0.0:
        raise DegenerateHead("sigma_max(W) <= 0")
    zs = stored_values(z, store)
    s = logits_of(zs, A, b)
    n = s.shape[0]
    label = np.argmax(s, axis=1) if n else np.zeros(0, dtype=np.int64)
    rows = np.arange(n)
    top1 = s[rows, label]
    others = s.copy()
    others[rows, label] = -np.inf
    top2 = others.max(axis=1) if n else np.zeros(0)
    margin = top1 - top2
    if radius_mode == "conservative":
        r64 = margin / (float(sigma) * SQRT2)
    elif radius_mode == "tight":
        A64 = A.astype(np.float64)
        r64 = np.empty(n)
        for i in range(n):
            y = label[i]
            best = np.inf
            for j in range(C):
                if j == y:
                    continue
                den = float(np.linalg.norm(A64[y] - A64[j]))
                if den == 0.0:
                    continue
                best = min(best, (top1[i] - s[i, j]) / den)
            r64[i] = best
    else:
        raise ValueError(f"unknown radius mode {radius_mode!r}")
    r = to_f32_toward_zero(r64)
    norm2 = np.sum(zs.astype(np.float64) ** 2, axis=1)
    return Certified(label.astype(np.int32), r, r64, margin, norm2, zs, s)


# ------------------------------------------------------------------ lookup
@dataclass
class LookupResult:
    label: np.ndarray       # int32 payload of i*, MISS on a miss
    index: np.ndarray       # int64 i*, -1 on a miss
    dist2: np.ndarray       # float64 ||z - z_i*||^2, +inf on a miss
    n_hits: np.ndarray      # int64 |H|
    n_band: np.ndarray      # int64 pairs with |D - r| <= BAND_REL * r
    flagged: np.ndarray     # bool: a band pair could change this query's answer


def lookup(zq, cache_z, cache_r, cache_label, band_rel: float = BAND_REL) -> LookupResult:
    """Certified lookup of every query against every cache entry (Eq. (13)-(15)).

    For query z: D_i^2 = sum_k (z_k - z_{i,k})^2 in float64 over the stored
    entry values; H = {i : D_i < r_i}, evaluated as D_i^2 < r_i^2 with r_i > 0
    (r_i^2 of a float32 r_i is exact in float64); a miss if H is empty, else
    i* = the hit of least D_i, lowest index among equal distances, and the
    answer is (label[i*], i*, D_{i*}^2).

    The boundary band is the set of pairs with |D_i - r_i| <= band_rel * r_i.
    A query is flagged when such a pair could change its answer: it has a
    band pair and either no hit outside the band, or a band pair no farther
    than (1 + band_rel) times its nearest non-band hit, or its two nearest
    hits lie within band_rel of each other.
    """
    Q = np.asarray(zq, dtype=np.float64)
    Z = np.asarray(cache_z)
    r = np.asarray(cache_r, dtype=np.float32).astype(np.float64)
    lab = np.asarray(cache_label, dtype=np.int32)
    B = Q.shape[0]
    out_label = np.full(B, MISS, dtype=np.int32)
    out_index = np.full(B, -1, dtype=np.int64)
    out_d2 = np.full(B, np.inf)
    n_hits = np.zeros(B, dtype=np.int64)
    n_band = np.zeros(B, dtype=np.int64)
    flagged = np.zeros(B, dtype=bool)
    if Z.shape[0] == 0:
        return LookupResult(out_label, out_index, out_d2, n_hits, n_band, flagged)
    r2 = r * r
    live = r > 0
    for qi in range(B):
        D2 = _dist2_to_all(Z, Q[qi])
        hit = live & (D2 < r2)
        D = np.sqrt(D2)
        band = live & (np.abs(D - r) <= band_rel * r)
        n_hits[qi] = int(hit.sum())
        n_band[qi] = int(band.sum())
        if n_hits[qi]:
            hd = D2[hit]
            best = hd.min()
            i_star = int(np.flatnonzero(hit & (D2 == best))[0])
            out_index[qi] = i_star
            out_label[qi] = lab[i_star]
            out_d2[qi] = D2[i_star]
        if n_band[qi]:
            solid = hit & ~band
            if not solid.any():
                flagged[qi] = True
            else:
                d_solid = np.sqrt(D2[solid].min())
                if np.any(D[band] <= (1.0 + band_rel) * d_solid):
                    flagged[qi] = True
        if n_hits[qi] >= 2:
            hd = np.sort(np.sqrt(D2[hit]))
            if hd[1] - hd[0] <= band_rel * max(hd[1], 1e-300):
                flagged[qi] = True
    return LookupResult(out_label, out_index, out_d2, n_hits, n_band, flagged)


def _dist2_to_all(Z, q, chunk: int = 1 << 15) -> np.ndarray:
    """D_i^2 = sum_k (q_k - z_{i,k})^2 in float64 for every row of Z (rows in chunks)."""
    out = np.empty(Z.shape[0])
    for s in range(0, Z.shape[0], chunk):
        e = min(Z.shape[0], s + chunk)
        out[s:e] = np.sum((Z[s:e].astype(np.float64) - q) ** 2, axis=1)
    return out


def lookup_rows(zq, cache_z, cache_r, cache_label, rows, band_rel: float = BAND_REL) -> LookupResult:
    """``lookup`` on the selected query rows only (sampled checks at full size)."""
    Q = np.asarray(zq)[np.asarray(rows, dtype=np.int64)]
    return lookup(Q, cache_z, cache_r, cache_label, band_rel)


def prefilter_rel(d: int) -> float:
    """Relative slack of the float32 matrix-product prefilter of ``lookup_blocked``.

    With float32 products and sums (any order), the expansion
    ||q||^2 + ||z||^2 - 2 q.z differs from the exact squared distance by at
    most about 2 (d + 3) 2^-24 (||q||^2 + ||z||^2): the dot product and the
    entry norm each contribute gamma_d, the few remaining roundings 6 u.  The
    slack is four times that.
    """
    return 8.0 * (d + 8) * 2.0 ** -24


def lookup_blocked(zq, cache_z, cache_r, cache_label, band_rel: float = BAND_REL,
                   q_chunk: int = 256, n_chunk: int = 1 << 16) -> LookupResult:
    """``lookup`` with a matrix-product prefilter; the same result.

    For each (query, entry) block the squared distance is first estimated
    from the expansion ||q||^2 + ||z_i||^2 - 2 q.z_i (one float32 BLAS product
    per block): a pair whose estimate, less prefilter_rel(d) (||q||^2 +
    ||z_i||^2), still exceeds (1 + band_rel)^2 r_i^2 can be neither a hit nor
    a band pair (an entry with r_i <= 0 never is), so only the survivors get
    the direct float64 sum_k (q_k - z_{i,k})^2 of ``lookup`` (the same
    expression, row by row), and the answer, band count and flag follow from
    them exactly as in ``lookup``.
    """
    Q = np.asarray(zq, dtype=np.float64)
    Q32 = np.asarray(zq, dtype=np.float32)
    Z = np.asarray(cache_z)
    r = np.asarray(cache_r, dtype=np.float32).astype(np.float64)
    lab = np.asarray(cache_label, dtype=np.int32)
    B, N = Q.shape[0], Z.shape[0]
    out_label = np.full(B, MISS, dtype=np.int32)
    out_index = np.full(B, -1, dtype=np.int64)
    out_d2 = np.full(B, np.inf)
    n_hits = np.zeros(B, dtype=np.int64)
    n_band = np.zeros(B, dtype=np.int64)
    flagged = np.zeros(B, dtype=bool)
    if N == 0 or B == 0:
        return LookupResult(out_label, out_index, out_d2, n_hits, n_band, flagged)
    r2 = r * r
    live = r > 0
    reach = (1.0 + band_rel) ** 2 * r2
    c = prefilter_rel(Q.shape[1])
    # estimate <= reach with estimate = (1 - c)(||q||^2 + ||z||^2) - 2 q.z,
    # rearranged as q.z >= a_q + b_i (the roundings this adds are inside c)
    a = ((1.0 - c) * np.sum(Q * Q, axis=1) / 2.0).astype(np.float32)
    pairs_q, pairs_e = [], []
    for ns in range(0, N, n_chunk):
        ne = min(N, ns + n_chunk)
        Zc = np.asarray(Z[ns:ne], dtype=np.float32)
        nz = np.sum(Zc * Zc, axis=1, dtype=np.float64)
        b = ((1.0 - c) * nz - reach[ns:ne]) / 2.0
        b[~live[ns:ne]] = np.inf          # entries that are never hit
        b = b.astype(np.float32)
        for qs in range(0, B, q_chunk):
            qe = min(B, qs + q_chunk)
            G = Q32[qs:qe] @ Zc.T
            G -= b[None, :]
            qi, ei = np.nonzero(G >= a[qs:qe, None])
            pairs_q.append(qi + qs)
            pairs_e.append(ei + ns)
    pq = np.concatenate(pairs_q)
    pe = np.concatenate(pairs_e)
    order = np.lexsort((pe, pq))          # by query, then ascending entry index
    pq, pe = pq[order], pe[order]
    starts = np.searchsorted(pq, np.arange(B + 1))
    for qi in range(B):
        idx = pe[starts[qi]:starts[qi + 1]]
        if idx.size == 0:
            continue
        D2 = np.sum((Z[idx].astype(np.float64) - Q[qi]) ** 2, axis=1)
        rr, rr2 = r[idx], r2[idx]
        hit = D2 < rr2
        D = np.sqrt(D2)
        band = np.abs(D - rr) <= band_rel * rr
        n_hits[qi] = int(hit.sum())
        n_band[qi] = int(band.sum())
        if n_hits[qi]:
            best = D2[hit].min()
            i_star = int(idx[np.flatnonzero(hit & (D2 == best))[0]])
            out_index[qi] = i_star
            out_label[qi] = lab[i_star]
            out_d2[qi] = best
        if n_band[qi]:
            solid = hit & ~band
            if not solid.any():
                flagged[qi] = True
            else:
                d_solid = np.sqrt(D2[solid].min())
                if np.any(D[band] <= (1.0 + band_rel) * d_solid):
                    flagged[qi] = True
        if n_hits[qi] >= 2:
            hd = np.sort(np.sqrt(D2[hit]))
            if hd[1] - hd[0] <= band_rel * max(hd[1], 1e-300):
                flagged[qi] = True
    return LookupResult(out_label, out_index, out_d2, n_hits, n_band, flagged)


# ------------------------------------------------------------------ insert
@dataclass
class CacheState:
    """Feature cache C = {(z_i, y~_i, r_i)} (Sec. 4.1) with a budget (capacity)."""

    d: int
    capacity: int
    store: str = "f32"
    z: np.ndarray = None          # (n, d) float32 stored values
    r: np.ndarray = None          # (n,) float32
    label: np.ndarray = None      # (n,) int32
    norm2: np.ndarray = None      # (n,) float64 squared norm of the stored values

    def __post_init__(self):
        if self.z is None:
            self.z = np.zeros((0, self.d), dtype=np.float32)
            self.r = np.zeros(0, dtype=np.float32)
            self.label = np.zeros(0, dtype=np.int32)
            self.norm2 = np.zeros(0, dtype=np.float64)

    @property
    def n(self) -> int:
        return int(self.r.shape[0])


def insert(state: CacheState, z_src, label_src, r_src, selector=None) -> int:
    """Append selected rows in ascending row order (write-back, Sec. 4.4, Alg. 2).

    Row j is taken when ``selector`` is None or ``selector[j] == MISS``, and
    its radius is positive (a non-positive radius is never cached, Alg. 1).
    The stored feature is the row cast to the store dtype (bfloat16 rounding to
    nearest even for a bfloat16 cache); its squared norm is recomputed from the
    stored values.  All-or-nothing: raises CapacityError, appending nothing,
    when the selected rows do not fit.  Returns the number of rows appended.
    """
    zs = np.asarray(z_src, dtype=np.float32)
    rs = np.asarray(r_src, dtype=np.float32)
    ls = np.asarray(label_src, dtype=np.int32)
    take = rs > 0
    if selector is not None:
        take &= np.asarray(selector) == MISS
    idx = np.flatnonzero(take)
    if state.n + idx.size > state.capacity:
        raise CapacityError(f"{state.n} + {idx.size} rows exceed capacity {state.capacity}")
    stored = stored_values(zs[idx], state.store) if idx.size else np.zeros((0, state.d), np.float32)
    state.z = np.concatenate([state.z, stored], axis=0)
    state.r = np.concatenate([state.r, rs[idx]])
    state.label = np.concatenate([state.label, ls[idx]])
    state.norm2 = np.concatenate([state.norm2, np.sum(stored.astype(np.float64) ** 2, axis=1)])
    return int(idx.size)


# ------------------------------------------------------------ construction
SELECT_STRATEGIES = ("radius_dedup", "priority", "kcenter")


def construct(state: CacheState, z, label, r, strategy: str = "radius_dedup", budget_total=None,
              budget_per_class: int = 0, priority=None, guard_label=None, n_classes=None) -> np.ndarray:
    """Offline construction of the feature store (Alg. 1): select and append.

    Eligible candidates have r_i > 0 and, when ``guard_label`` is given (the
    cache-centre label-consistency flag of Alg. 1), guard_label_i == label_i;
    with the priority strategy a NaN priority is not eligible, and with a
    per-class budget and ``n_classes`` given, neither is a label outside
    [0, n_classes).
    At most ``budget_total`` entries are appended (default: the free
    capacity; more than the free capacity raises CapacityError) and, when
    ``budget_per_class`` > 0, at most that many per payload label.  Distances
    are float64 over the stored values (bfloat16-rounded for a bf16 store).

    * ``radius_dedup`` - visit eligible candidates by decreasing r (ties:
      lower index); skip one whose class is full; skip a duplicate, i.e. a
      candidate strictly inside the ball ||z_i - z_j|| < r_j of an entry
      already in the cache (present before the call or appended earlier);
      append the rest until the total budget is used.
    * ``priority`` - the same visit, by decreasing ``priority`` (e.g. random
      keys: the random strategy), without the duplicate test.
    * ``kcenter`` - farthest-first traversal: start at the eligible candidate
      of largest r (ties: lower index), then repeatedly append the eligible,
      not yet chosen candidate (of a class that is not full) whose distance to
      the nearest chosen candidate is largest (ties: lower index).  With a
      per-class budget each class is traversed on its own (distances to its
      own chosen candidates), classes in ascending label order.  Entries
      present before the call are not used.

    Returns the selected candidate indices in the order they were appended.
    """
    if strategy not in SELECT_STRATEGIES:
        raise ValueError(f"unknown strategy {strategy!r}")
    zs = stored_values(np.asarray(z, dtype=np.float32), state.store)
    lab = np.asarray(label, dtype=np.int32)
    rr = np.asarray(r, dtype=np.float32)
    n = zs.shape[0]
    free = state.capacity - state.n
    budget = free if budget_total is None else int(budget_total)
    if budget < 0 or budget > free:
        raise CapacityError(f"budget {budget} exceeds the free capacity {free}")
    eligible = rr > 0
    if guard_label is not None:
        eligible &= np.asarray(guard_label, dtype=np.int32) == lab
    if strategy == "priority":
        eligible &= ~np.isnan(np.asarray(priority, dtype=np.float32))
    if budget_per_class > 0 and n_classes is not None:
        eligible &= (lab >= 0) & (lab < n_classes)
    counts: dict[int, int] = {}

    def class_open(c: int) -> bool:
        return budget_per_class <= 0 or counts.get(c, 0) < budget_per_class

    chosen: list[int] = []
    if strategy in ("radius_dedup", "priority"):
        key = rr if strategy == "radius_dedup" else np.asarray(priority, dtype=np.float32)
        idx = np.flatnonzero(eligible)
        order = idx[np.lexsort((idx, -key[idx].astype(np.float64)))]
        cz = state.z.astype(np.float64)
        cr2 = state.r.astype(np.float64) ** 2
        clive = state.r > 0
        for i in order:
            if len(chosen) >= budget:
                break
            c = int(lab[i])
            if not class_open(c):
                continue
            if strategy == "radius_dedup" and cz.shape[0]:
                d2 = np.sum((cz - zs[i].astype(np.float64)) ** 2, axis=1)
                if np.any(clive & (d2 < cr2)):
                    continue
            chosen.append(int(i))
            counts[c] = counts.get(c, 0) + 1
            if strategy == "radius_dedup":
                cz = np.concatenate([cz, zs[i:i + 1].astype(np.float64)])
                cr2 = np.concatenate([cr2, [float(rr[i]) ** 2]])
                clive = np.concatenate([clive, [True]])
    else:
        groups = [np.flatnonzero(eligible)]
        if budget_per_class > 0:
            groups = [np.flatnonzero(eligible & (lab == c)) for c in np.unique(lab[eligible])]
        for g in groups:
            if len(chosen) >= budget or g.size == 0:
                continue
            first = g[np.lexsort((g, -rr[g].astype(np.float64)))[0]]
            picked = [int(first)]
            mind = np.sum((zs[g].astype(np.float64) - zs[first].astype(np.float64)) ** 2, axis=1)
            taken = np.zeros(g.size, dtype=bool)
            taken[np.flatnonzero(g == first)[0]] = True
            limit = budget - len(chosen)
            if budget_per_class > 0:
                limit = min(limit, budget_per_class)
            while len(picked) < limit and not taken.all():
                cand = np.where(taken, -1.0, mind)
                j = int(np.flatnonzero(cand == cand.max())[0])   # lowest index among the farthest
                picked.append(int(g[j]))
                taken[j] = True
                mind = np.minimum(mind, np.sum((zs[g].astype(np.float64) - zs[g[j]].astype(np.float64)) ** 2,
                                               axis=1))
            chosen.extend(picked)
    sel = np.asarray(chosen, dtype=np.int64)
    if sel.size:
        state.z = np.concatenate([state.z, zs[sel]], axis=0)
        state.r = np.concatenate([state.r, rr[sel]])
        state.label = np.concatenate([state.label, lab[sel]])
        state.norm2 = np.concatenate([state.norm2, np.sum(zs[sel].astype(np.float64) ** 2, axis=1)])
    return sel


# ------------------------------------------------- reuse boundaries, metric
BOUNDARY_MODES = ("scaled", "global", "interclass")


def boundary_radius(state: CacheState, mode: str, factor: float) -> np.ndarray:
    """Per-entry reuse radii for the boundary comparisons of Sec. 6 (float32).

    * ``scaled``     - factor * r_i: radius tightening for factor <= 1, which
                       keeps every hit inside its certified ball.
    * ``global``     - factor for every entry: one global nearest-neighbour
                       threshold tau (the nearest entry within tau is reused).
    * ``interclass`` - an empirical radius from inter-class distance
                       statistics: factor * 1/2 * min_{c != y_i} ||mu_{y_i} -
                       mu_c||, where mu_c is the mean of the cached features
                       of label c (float64); +inf when no other label is
                       cached.
    Entries with r_i <= 0 keep radius 0 (never hit).
    """
    r = state.r.astype(np.float64)
    live = state.r > 0
    if mode == "scaled":
        out = factor * r
    elif mode == "global":
        out = np.full(state.n, float(factor))
    elif mode == "interclass":
        lab = state.label
        classes = np.unique(lab[live])
        z = state.z.astype(np.float64)
        mu = {int(c): z[live & (lab == c)].mean(axis=0) for c in classes}
        half = {}
        for c in classes:
            others = [np.linalg.norm(mu[int(c)] - mu[int(o)]) for o in classes if o != c]
            half[int(c)] = 0.5 * min(others) if others else np.inf
        out = np.array([factor * half.get(int(l), 0.0) for l in lab])
    else:
        raise ValueError(f"unknown boundary mode {mode!r}")
    out = np.where(live, out, 0.0)
    return out.astype(np.float32)


def cluster_pruned_lookup(zq, cache_z, cache_r, cache_label, assign, centres=None):
    """``lookup`` through a partition of the cache rows (the exact sublinear
    index the paper points to in Sec. 4.4 for large caches).

    ``assign[i]`` is the cluster of row i; the centre mu_c of a cluster is
    ``centres[c]`` when given, else the float64 mean of its rows.  Its bound
    is R_c = max over its live rows (r_i > 0) of ||z_i - mu_c|| + r_i; by the
    triangle inequality a query z with ||z - mu_c|| >= R_c lies outside every
    ball of the cluster, so only the rows of clusters with ||z - mu_c|| < R_c
    are tested.  Returns (``LookupResult`` with indices into the whole cache,
    number of (query, row) pairs tested).  The label, index, d^2 and hit
    count equal ``lookup``'s for every partition; the band counts cover the
    tested rows only.
    """
    Q = np.asarray(zq, dtype=np.float64)
    Z = np.asarray(cache_z)
    Z64 = Z.astype(np.float64)
    r = np.asarray(cache_r, dtype=np.float32).astype(np.float64)
    lab = np.asarray(cache_label, dtype=np.int32)
    a = np.asarray(assign, dtype=np.int64)
    K = int(a.max()) + 1 if a.size else 0
    members = [np.flatnonzero(a == c) for c in range(K)]
    mu = np.zeros((K, Z.shape[1]))
    R = np.full(K, -np.inf)
    for c, rows in enumerate(members):
        if centres is not None:
            mu[c] = np.asarray(centres[c], dtype=np.float64)
        elif rows.size:
            mu[c] = Z64[rows].mean(axis=0)
        live = rows[r[rows] > 0]
        if live.size:
            R[c] = np.max(np.sqrt(np.sum((Z64[live] - mu[c]) ** 2, axis=1)) + r[live])
    B = Q.shape[0]
    parts = []
    pairs = 0
    for qi in range(B):
        dc = np.sqrt(np.sum((mu - Q[qi]) ** 2, axis=1))
        cand = [members[c] for c in range(K) if dc[c] < R[c]]
        rows = np.sort(np.concatenate(cand)) if cand else np.zeros(0, np.int64)
        pairs += rows.size
        res = lookup(Q[qi:qi + 1], Z[rows], r[rows].astype(np.float32), lab[rows])
        if res.index[0] >= 0:
            res.index[0] = rows[res.index[0]]
        parts.append(res)
    cat = lambda f: np.concatenate([getattr(p, f) for p in parts]) if parts else np.zeros(0)  # noqa: E731
    out = LookupResult(cat("label").astype(np.int32), cat("index").astype(np.int64), cat("dist2"),
                       cat("n_hits").astype(np.int64), cat("n_band").astype(np.int64), cat("flagged").astype(bool))
    return out, pairs


def lookup_partitioned(zq, cache_z, cache_r, cache_label, assign, centres, band_rel: float = BAND_REL,
                       widen: float = 1e-6) -> LookupResult:
    """``lookup`` for full-size batches, through a partition of the rows: the
    same ``LookupResult`` as ``lookup``, every field (band counts and flags
    included).

    Row i belongs to cluster ``assign[i]`` with centre ``centres[c]``.  A
    row of cluster c with ||q - mu_c|| >= R_c = max over its live rows of
    ||z_i - mu_c|| + (1 + band_rel) r_i lies at D = ||q - z_i|| >= ||q -
    mu_c|| - ||z_i - mu_c|| >= (1 + band_rel) r_i from the query (triangle
    inequality): neither a hit (D < r_i, Eq. (13)) nor a band pair (|D - r_i|
    <= band_rel r_i) unless D sits exactly on the band's outer edge.  So only
    clusters with ||q - mu_c|| < R_c (1 + widen) + widen are searched; the
    widening covers that edge and the float64 rounding of these norms.  Every
    hit and band pair of q lies in its searched clusters, and so do its
    answer, hit count, band count and flag (all defined by those pairs
    alone).  A query with one searched cluster gets ``lookup_blocked`` on
    that cluster's rows; one with several gets ``lookup`` on their union.
    """
    Q = np.asarray(zq, dtype=np.float64)
    Z = np.asarray(cache_z)
    r = np.asarray(cache_r, dtype=np.float32)
    lab = np.asarray(cache_label, dtype=np.int32)
    a = np.asarray(assign, dtype=np.int64)
    mu = np.asarray(centres, dtype=np.float64)
    B, K = Q.shape[0], mu.shape[0]
    out = LookupResult(np.full(B, MISS, dtype=np.int32), np.full(B, -1, dtype=np.int64), np.full(B, np.inf),
                       np.zeros(B, dtype=np.int64), np.zeros(B, dtype=np.int64), np.zeros(B, dtype=bool))
    if B == 0 or Z.shape[0] == 0:
        return out
    order = np.argsort(a, kind="stable")              # rows of each cluster in ascending order
    starts = np.searchsorted(a[order], np.arange(K + 1))
    R = np.full(K, -np.inf)
    r64 = r.astype(np.float64)
    for c in range(K):
        rows = order[starts[c]:starts[c + 1]]
        live = rows[r[rows] > 0]
        if live.size:
            dz = np.sqrt(np.sum((Z[live].astype(np.float64) - mu[c]) ** 2, axis=1))
            R[c] = np.max(dz + (1.0 + band_rel) * r64[live])
    reach = R * (1.0 + widen) + widen
    # ||q - mu_c||^2 from the float64 expansion, less a bound on its rounding
    # error (4 (d + 4) 2^-53 (||q||^2 + ||mu_c||^2)): a superset of the
    # clusters with ||q - mu_c|| < reach
    nq = np.sum(Q * Q, axis=1)
    nm = np.sum(mu * mu, axis=1)
    tol = 4.0 * (Q.shape[1] + 4) * 2.0 ** -53
    searched = np.empty((B, K), dtype=bool)
    for s0 in range(0, B, 8192):
        s1 = min(B, s0 + 8192)
        scale = nq[s0:s1, None] + nm[None, :]
        d2 = scale - 2.0 * (Q[s0:s1] @ mu.T)
        searched[s0:s1] = (d2 - tol * scale < (reach * reach)[None, :]) & (R > -np.inf)[None, :]
    count = searched.sum(axis=1)

    def put(qidx, res, rows):
        out.label[qidx] = res.label
        out.index[qidx] = np.where(res.index >= 0, rows[np.maximum(res.index, 0)], -1)
        out.dist2[qidx] = res.dist2
        out.n_hits[qidx] = res.n_hits
        out.n_band[qidx] = res.n_band
        out.flagged[qidx] = res.flagged

    only = np.where(count == 1, np.argmax(searched, axis=1), -1)
    for c in range(K):
        qidx = np.flatnonzero(only == c)
        rows = order[starts[c]:starts[c + 1]]
        if qidx.size and rows.size:
            put(qidx, lookup_blocked(Q[qidx], Z[rows], r[rows], lab[rows], band_rel), rows)
    for qi in np.flatnonzero(count > 1):
        rows = np.sort(np.concatenate([order[starts[c]:starts[c + 1]] for c in np.flatnonzero(searched[qi])]))
        put(np.array([qi]), lookup(Q[qi:qi + 1], Z[rows], r[rows], lab[rows], band_rel), rows)
    return out


def consistency(lookup_label, head_label):
    """Certified-consistency bookkeeping (Sec. 6): among the hits (lookup
    label != MISS), how many return the head's own argmax at the query.
    Returns (hits, consistent)."""
    lk = np.asarray(lookup_label, dtype=np.int64)
    hd = np.asarray(head_label, dtype=np.int64)
    hit = lk != MISS
    return int(hit.sum()), int((hit & (lk == hd)).sum())
