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


# ---------------------------------------------------------------------------------------------------------------
# Pins of the oracle's LRU that do not involve the native pool: hand-derived eviction sequences, and the long-run hit
# ratio of an LRU cache under independent Zipf requests.
import json
import os
from collections import deque

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lru_traces.json")


def _fifo(keys, capacity):
    """First-in first-out replacement (hits do not refresh an entry): only used to show the fixtures discriminate."""
    order, cache, hits, evicted = deque(), set(), [], []
    for k in keys:
        if k in cache:
            hits.append(True)
            evicted.append(None)
            continue
        hits.append(False)
        if len(cache) >= capacity:
            old = order.popleft()
            cache.remove(old)
            evicted.append(old)
        else:
            evicted.append(None)
        cache.add(k)
        order.append(k)
    return hits, evicted


def _mru(keys, capacity):
    """Most-recently-used replacement: only used to show the fixtures discriminate."""
    cache, last, hits, evicted = set(), None, [], []
    for k in keys:
        if k in cache:
            hits.append(True)
            evicted.append(None)
        else:
            hits.append(False)
            if len(cache) >= capacity:
                cache.remove(last)
                evicted.append(last)
            else:
                evicted.append(None)
            cache.add(k)
        last = k
    return hits, evicted


def test_oracle_lru_matches_hand_derived_traces():
    traces = json.load(open(GOLDEN))["traces"]
    for t in traces:
        hits, evicted = H.lru(t["keys"], t["capacity"])
        assert hits == t["lru_hits"] and evicted == t["lru_evicted"], t["derivation"]
        # the hand-derived FIFO / MRU columns agree with plain implementations of those rules ...
        assert list(_fifo(t["keys"], t["capacity"])) == [t["fifo_hits"], t["fifo_evicted"]]
        assert list(_mru(t["keys"], t["capacity"])) == [t["mru_hits"], t["mru_evicted"]]
    # ... and differ from LRU on the capacity-2 and capacity-3 traces, so either mistake in lru() fails above
    for t in traces[:2]:
        assert (t["fifo_hits"], t["fifo_evicted"]) != (t["lru_hits"], t["lru_evicted"])
        assert (t["mru_hits"], t["mru_evicted"]) != (t["lru_hits"], t["lru_evicted"])


def _che_lru_hit_ratio(p, capacity):
    """Che's approximation of an LRU cache's hit ratio under independent requests with popularity p (Che, Tung and
    Wang, IEEE JSAC 2002): the characteristic time T solves sum_i (1 - exp(-p_i T)) = C, and the hit ratio is
    sum_i p_i (1 - exp(-p_i T)).  Accurate to a few 1e-3 for caches of tens of entries or more."""
    from scipy.optimize import brentq

    t = brentq(lambda x: np.sum(1.0 - np.exp(-p * x)) - capacity, 1e-9, 1e12)
    return float(np.sum(p * (1.0 - np.exp(-p * t))))


@pytest.mark.parametrize("alpha,capacity", [(0.8, 100), (1.0, 50)])
def test_lru_long_trace_follows_che_approximation_and_static_bound(alpha, capacity):
    """eq. hit-ratio-analysis rests on the static top-C hit ratio (zipf_mass); an LRU pool under independent Zipf
    requests runs below it, at the hit ratio Che's approximation gives.  FIFO replacement runs ~0.03-0.05 lower
    still, outside the tolerance."""
    n, warm, total = 2000, 20000, 200000
    rng = np.random.default_rng(int(alpha * 100) + capacity)
    p = np.arange(1, n + 1, dtype=np.float64) ** (-alpha)
    p /= p.sum()
    keys = rng.choice(n, size=total, p=p).tolist()
    che = _che_lru_hit_ratio(p, capacity)
    hits, _ = H.lru(keys, capacity)
    lru_ratio = float(np.mean(hits[warm:]))
    assert abs(lru_ratio - che) < 0.006, (lru_ratio, che)
    fifo_ratio = float(np.mean(_fifo(keys, capacity)[0][warm:]))
    assert che - fifo_ratio > 0.02, (fifo_ratio, che)
    # a static cache of the C most popular documents hits at zipf_mass (sampling error only) and beats LRU
    static = float(np.mean(np.asarray(keys[warm:]) < capacity))
    assert abs(static - H.zipf_mass(capacity, n, alpha)) < 0.006
    assert lru_ratio < static
    # the native pool follows the same curve
    pool = hitsim.Pool(capacity)
    native = [pool.acquire(k)[1] for k in keys]
    assert abs(float(np.mean(native[warm:])) - che) < 0.006
