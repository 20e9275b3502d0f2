"""Seeded synthetic inputs for the certified cache path.

The paper evaluates on image datasets encoded by a trained guard network
(Sec. 6.1); neither is available, so the feature space itself is synthesised:
Gaussian-mixture features with a Gaussian linear head, scaled up from the
paper's operating point (d = 64, C = 10, 200 entries per class; Sec. 6.1,
Sec. 6.5) to cache sizes of 4K .. 4M entries.

This module draws random numbers and lays them out; it contains none of the
method's arithmetic (no logits, margins, radii, distances or hit tests).  The
only place where a method output enters is ``compose_queries``, which takes the
certified radii as an *argument* to place "near-ball" queries at u * r_i from a
cache centre.  Both the HIP path and the CPU oracle consume these arrays.

Draw order for one configuration (``numpy.random.default_rng(seed)``, PCG64):

  1. ``W = standard_normal((C, d)) / sqrt(d)``            -> float32
  2. ``b = standard_normal(C) * bias_std``  (only drawn if bias_std > 0)
  3. ``mu = standard_normal((C, d)) * mu_std``            (float64, kept)
  4. cache candidates: ``k = integers(0, C, N)``, then
     ``z = mu[k] + sigma * standard_normal((N, d))``     -> float32
     (drawn in row chunks; the stream is consumed in the same order)
  5. queries of round t use their own stream
     ``default_rng(SeedSequence([seed, 1 + t]))``:
       fresh half:  ``k = integers(0, C, n_fresh)``,
                    ``x = mu[k] + sigma * standard_normal((n_fresh, d))`` -> float32
       near half:   ``pick = random(n_near)`` (index = floor(pick * n_live)),
                    ``v = standard_normal((n_near, d))`` normalised to unit length,
                    ``u = uniform(0, 2, n_near)``
       ``perm = permutation(B)``
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "WorkloadConfig",
    "CONFIGS",
    "Workload",
    "QueryDraws",
    "make_workload",
    "draw_queries",
    "compose_queries",
]


@dataclass(frozen=True)
class WorkloadConfig:
    """Shape and distribution of one synthetic workload."""

    name: str
    d: int                 # feature dimension
    C: int                 # number of classes (rows of W)
    n_cache: int           # cache candidates drawn (initial cache size)
    batch: int             # queries per round
    sigma: float           # within-class standard deviation
    mu_std: float = 2.0    # class means ~ N(0, mu_std^2 I)
    bias_std: float = 0.0  # head bias ~ N(0, bias_std^2); 0 => b = 0, not drawn
    store_dtype: str = "f32"
    rounds: int = 1
    capacity: int = 0      # 0 => n_cache + rounds * batch

    @property
    def cache_capacity(self) -> int:
        return self.capacity or (self.n_cache + self.rounds * self.batch)


# The five workloads.  Variances in the recipes are read as variances:
# W ~ N(0, 1/d) has std 1/sqrt(d); mu ~ N(0, 4 I) has std 2; b ~ N(0, 0.01)
# has std 0.1.  "0.5 N(0, I)" and "sigma = 0.7/0.8" are standard deviations.
CONFIGS: dict[str, WorkloadConfig] = {
    c.name: c
    for c in (
        WorkloadConfig("tiny-d64-c10", d=64, C=10, n_cache=4096, batch=1024, sigma=0.5),
        WorkloadConfig("mix-d128-c10", d=128, C=10, n_cache=65536, batch=8192, sigma=0.5),
        WorkloadConfig("mix-d128-c100", d=128, C=100, n_cache=262144, batch=16384,
                       sigma=0.7, bias_std=0.1),
        WorkloadConfig("mix-d256-c200", d=256, C=200, n_cache=1048576, batch=32768, sigma=0.8),
        WorkloadConfig("stream-d256-c200-bf16", d=256, C=200, n_cache=2097152, batch=65536,
                       sigma=0.8, store_dtype="bf16", rounds=16, capacity=4194304),
    )
}


@dataclass
class Workload:
    """Head and cache candidates of one configuration (float32 unless noted)."""

    config: WorkloadConfig
    seed: int
    W: np.ndarray            # (C, d) float32
    b: np.ndarray            # (C,) float32
    mu: np.ndarray           # (C, d) float64 class means (needed for fresh queries)
    z: np.ndarray            # (N, d) float32 cache candidates
    z_class: np.ndarray      # (N,) int32 mixture component of each candidate


@dataclass
class QueryDraws:
    """Random draws for one round of queries; positions depend on radii later."""

    fresh: np.ndarray        # (n_fresh, d) float32
    pick: np.ndarray         # (n_near,) float64 in [0, 1)
    direction: np.ndarray    # (n_near, d) float64 unit vectors
    u: np.ndarray            # (n_near,) float64 in [0, 2)
    perm: np.ndarray         # (B,) int64 permutation of [near; fresh]
    extra: dict = field(default_factory=dict)

    @property
    def n_near(self) -> int:
        return int(self.pick.shape[0])

    @property
    def batch(self) -> int:
        return int(self.perm.shape[0])


def _normal_rows(rng: np.random.Generator, rows: int, d: int, chunk: int = 1 << 16):
    """Yield (start, block) of standard normals, consuming the stream in row order."""
    for s in range(0, rows, chunk):
        e = min(rows, s + chunk)
        yield s, rng.standard_normal((e - s, d))


def make_workload(config: WorkloadConfig | str, seed: int = 0,
                  n_cache: int | None = None) -> Workload:
    """Draw the head and the cache candidates of ``config`` (steps 1-4 above).

    ``n_cache`` overrides the number of candidates (for scaled-down tests);
    the draw order is unchanged, so a smaller N is a prefix of the full draw
    of W, b and mu but not of z.
    """
    cfg = CONFIGS[config] if isinstance(config, str) else config
    C, d = cfg.C, cfg.d
    N = cfg.n_cache if n_cache is None else int(n_cache)
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((C, d)) / math.sqrt(d)).astype(np.float32)
    if cfg.bias_std > 0:
        b = (rng.standard_normal(C) * cfg.bias_std).astype(np.float32)
    else:
        b = np.zeros(C, dtype=np.float32)
    mu = rng.standard_normal((C, d)) * cfg.mu_std
    k = rng.integers(0, C, size=N)
    z = np.empty((N, d), dtype=np.float32)
    for s, g in _normal_rows(rng, N, d):
        e = s + g.shape[0]
        z[s:e] = (mu[k[s:e]] + cfg.sigma * g).astype(np.float32)
    return Workload(cfg, seed, W, b, mu, z, k.astype(np.int32))


def draw_queries(wl: Workload, round_index: int = 0, batch: int | None = None) -> QueryDraws:
    """Draw one round of queries (step 5): half near-ball, half fresh mixture draws."""
    cfg = wl.config
    B = cfg.batch if batch is None else int(batch)
    d = cfg.d
    rng = np.random.default_rng(np.random.SeedSequence([wl.seed, 1 + round_index]))
    n_near = B // 2
    n_fresh = B - n_near
    k = rng.integers(0, cfg.C, size=n_fresh)
    fresh = np.empty((n_fresh, d), dtype=np.float32)
    for s, g in _normal_rows(rng, n_fresh, d):
        e = s + g.shape[0]
        fresh[s:e] = (wl.mu[k[s:e]] + cfg.sigma * g).astype(np.float32)
    pick = rng.random(n_near)
    direction = rng.standard_normal((n_near, d))
    direction /= np.linalg.norm(direction, axis=1, keepdims=True)
    u = rng.uniform(0.0, 2.0, size=n_near)
    perm = rng.permutation(B)
    return QueryDraws(fresh=fresh, pick=pick, direction=direction, u=u, perm=perm)


def near_indices(draws: QueryDraws, n_live: int) -> np.ndarray:
    """Cache rows that the near-ball queries are placed around."""
    if n_live <= 0:
        return np.zeros(0, dtype=np.int64)
    return np.minimum((draws.pick * n_live).astype(np.int64), n_live - 1)


def compose_queries(draws: QueryDraws, centres: np.ndarray, radii: np.ndarray) -> np.ndarray:
    """Place the near-ball queries and return the shuffled (B, d) float32 batch.

    ``centres`` are the stored cache features of the rows ``near_indices``
    selects (as float32/float64 values) and ``radii`` their float32 radii,
    both already gathered, shape (n_near, d) and (n_near,).  Each near query
    is ``centre + u * r * direction`` formed in float64 and rounded to float32.
    With an empty cache the near half falls back to the first fresh draws.
    """
    n_near = draws.n_near
    if n_near and centres.shape[0] == 0:
        near = np.resize(draws.fresh, (n_near, draws.fresh.shape[1])).astype(np.float32)
    else:
        c = np.asarray(centres, dtype=np.float64)
        rr = np.asarray(radii, dtype=np.float64)
        near = (c + (draws.u * rr)[:, None] * draws.direction).astype(np.float32)
    allq = np.concatenate([near, draws.fresh], axis=0)
    return np.ascontiguousarray(allq[draws.perm])
