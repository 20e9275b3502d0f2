"""CPU oracle of the certified cache path (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline
leg import this package; the product path never does.
"""
from .lipcache_oracle import *  # noqa: F401,F403
from .lipcache_oracle import (MISS, BAND_REL, DegenerateHead, CapacityError,  # noqa: F401
                              bf16_round, stored_values, spectral_norm, certify,
                              logits_of, lookup, lookup_rows, lookup_blocked, insert, to_f32_toward_zero,
                              CacheState, construct, SELECT_STRATEGIES,
                              boundary_radius, consistency, BOUNDARY_MODES,
                              cluster_pruned_lookup, lookup_partitioned)
