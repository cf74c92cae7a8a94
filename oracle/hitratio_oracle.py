"""Plain reference models for the chunk-pool hit-ratio study.

TEST INFRASTRUCTURE ONLY (like lazy_oracle): only the tests call it; it shares no code with the library's pool.

- ``hit_ratio_advantage``: the paper's analytic model (Sec. 2, "Hit-ratio impact under limited cache capacity",
  eq. hit-ratio-analysis): with Zipf(alpha) document popularity, a position-agnostic cache of C entries holds the
  top C documents and a position-aware one about the top floor(C / D); the advantage is the ratio of the two
  popularity masses, sum_{i <= C} i^-alpha / sum_{i <= floor(C/D)} i^-alpha.
- ``zipf_mass``: the hit ratio of a static cache of the top C of N documents (H_agnostic of the same passage).
- ``lru``: a textbook least-recently-used cache written with an ordered dict, returning the hit / eviction
  sequence of a key trace.

Pins (tests/test_hitsim.py): the analytic model reproduces the paper's printed 2.86x and the alpha = 0 and alpha = 1
closed forms; ``lru`` reproduces hand-derived eviction sequences (tests/golden/lru_traces.json, chosen so that FIFO
or MRU replacement gives different ones) and, on long independent Zipf traces, Che's approximation of the LRU hit
ratio, below the static top-C bound ``zipf_mass``, which a sampled static cache matches.
"""
from __future__ import annotations

from collections import OrderedDict

import numpy as np


def zipf_mass(c: int, n: int, alpha: float) -> float:
    i = np.arange(1, n + 1, dtype=np.float64) ** (-alpha)
    return float(i[: min(c, n)].sum() / i.sum())


def hit_ratio_advantage(c: int, d: int, alpha: float) -> float:
    top = np.arange(1, c + 1, dtype=np.float64) ** (-alpha)
    k = c // d
    return float(top.sum() / top[:k].sum())


def lru(keys, capacity: int):
    """Hit flags and evicted keys (None where nothing was evicted) of an LRU cache of ``capacity`` entries."""
    cache: OrderedDict = OrderedDict()
    hits, evicted = [], []
    for k in keys:
        if k in cache:
            cache.move_to_end(k)
            hits.append(True)
            evicted.append(None)
            continue
        hits.append(False)
        if len(cache) >= capacity:
            old, _ = cache.popitem(last=False)
            evicted.append(old)
        else:
            evicted.append(None)
        cache[k] = True
    return hits, evicted
