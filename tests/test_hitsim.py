"""CPU tests of the position-agnostic chunk pool (native LRU) and the hit-ratio simulation, against a textbook LRU
and the paper's analytic hit-ratio model (Sec. 2, eq. hit-ratio-analysis)."""
import math

import numpy as np
import pytest

from oracle import hitratio_oracle as H
from paper_2606_04302_amd import hitsim


def test_analytic_advantage_matches_the_paper_and_closed_forms():
    # the paper prints a 2.86x advantage at D = 20 positions and C = 100 entries for a moderately skewed Zipf
    # distribution; alpha = 0.853 is the skew that reproduces it
    assert round(H.hit_ratio_advantage(100, 20, 0.853), 2) == 2.86
    # alpha = 0: every document equally popular, the advantage is C / floor(C / D)
    assert H.hit_ratio_advantage(100, 20, 0.0) == pytest.approx(20.0, abs=1e-12)
    assert H.hit_ratio_advantage(100, 30, 0.0) == pytest.approx(100 / 3, abs=1e-12)
    # more skew, smaller advantage (the top documents dominate both caches)
    assert H.hit_ratio_advantage(100, 20, 2.0) < H.hit_ratio_advantage(100, 20, 1.0) < 20.0
    # harmonic closed form of the static hit ratio at alpha = 1
    assert H.zipf_mass(10, 100, 1.0) == pytest.approx(sum(1 / i for i in range(1, 11)) /
                                                      sum(1 / i for i in range(1, 101)), rel=1e-12)


@pytest.mark.parametrize("capacity", [1, 3, 17])
def test_native_pool_is_exactly_lru(capacity):
    rng = np.random.default_rng(capacity)
    keys = rng.integers(0, 40, size=3000).tolist()
    hits, evicted = H.lru(keys, capacity)
    pool = hitsim.Pool(capacity)
    slots = {}
    for k, h, e in zip(keys, hits, evicted):
        slot, hit, ev = pool.acquire(k)
        assert hit == h and ev == e
        assert 0 <= slot < capacity
        if hit:
            assert slots[k] == slot          # a resident key keeps its slot
        slots[k] = slot
        if e is not None:
            slots.pop(e, None)
    lookups, nh, nev, resident = pool.stats()
    assert lookups == len(keys) and nh == sum(hits) and nev == sum(e is not None for e in evicted)
    assert resident == min(capacity, len(set(keys)))
    assert len(set(slots.values())) == len(slots)  # no two resident keys share a slot


def test_pool_rejects_bad_capacity_and_large_keys_work():
    with pytest.raises(ValueError):
        hitsim.Pool(0)
    pool = hitsim.Pool(2)
    big = (1 << 64) - 1
    assert pool.acquire(big)[1] is False and pool.acquire(big)[1] is True


def test_simulation_properties():
    docs = hitsim.zipf_trace(2000, 1.1, 1500, 10, seed=3)
    distinct = len(np.unique(docs))
    # a pool that never evicts misses only the first use of each document
    assert hitsim.hit_ratio(docs, distinct, "agnostic") == pytest.approx(1 - distinct / docs.size, abs=1e-12)
    # with one prompt position the two keyings coincide
    one = docs[:, :1]
    assert hitsim.hit_ratio(one, 50, "aware") == hitsim.hit_ratio(one, 50, "agnostic")
    # same trace, same entries: the position-agnostic pool hits more often
    for c in (20, 100, 400):
        assert hitsim.hit_ratio(docs, c, "agnostic") > hitsim.hit_ratio(docs, c, "aware")
