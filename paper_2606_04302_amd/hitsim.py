"""Hit-ratio simulation of a position-agnostic vs a position-aware chunk pool (Sec. 2 "Hit-ratio impact under
limited cache capacity"; the paper's Table 1 measures the same quantity on its traces, which are not used here).

Synthetic traces: N documents with Zipf(alpha) popularity; each query retrieves K distinct documents (drawn without
replacement by popularity) in a random order, so a document appears in any of D = K prompt positions.  Both pools
are the library's native LRU pool (lazy_pool_*) with the same number of entries: the position-agnostic pool keys a
chunk by its document (one stored copy serves every position, as position-free storage allows), the position-aware
pool by (document, position) (a positionally encoded copy per position).  The hit ratio is hits / lookups over all
K lookups of every query.

    python -m paper_2606_04302_amd.hitsim [--docs 100000] [--queries 20000] [--k 10]
"""
from __future__ import annotations

import argparse
import ctypes

import numpy as np

from . import ops


def zipf_trace(n_docs: int, alpha: float, n_queries: int, k: int, seed: int = 0):
    """doc ids [n_queries, k] (0 = most popular) in prompt order."""
    rng = np.random.default_rng(seed)
    p = np.arange(1, n_docs + 1, dtype=np.float64) ** (-alpha)
    p /= p.sum()
    docs = np.empty((n_queries, k), dtype=np.int64)
    for q in range(n_queries):
        pick = rng.choice(n_docs, size=k, replace=False, p=p)
        rng.shuffle(pick)
        docs[q] = pick
    return docs


class Pool:
    """ctypes handle of a native LRU chunk pool."""

    def __init__(self, capacity: int):
        self.h = ops.lib().lazy_pool_create(int(capacity))
        if not self.h:
            raise ValueError(f"lazy_pool_create({capacity}) failed")

    def acquire(self, key: int):
        slot, hit, ev, evk = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_uint64()
        ops._check(ops.lib().lazy_pool_acquire(self.h, ctypes.c_uint64(key), ctypes.byref(slot), ctypes.byref(hit),
                                               ctypes.byref(evk), ctypes.byref(ev)), "lazy_pool_acquire")
        return slot.value, bool(hit.value), (evk.value if ev.value else None)

    def stats(self):
        lk, ht, ev = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        res = ctypes.c_int32()
        ops._check(ops.lib().lazy_pool_stats(self.h, ctypes.byref(lk), ctypes.byref(ht), ctypes.byref(ev),
                                             ctypes.byref(res)), "lazy_pool_stats")
        return lk.value, ht.value, ev.value, res.value

    def close(self):
        if self.h:
            ops.lib().lazy_pool_destroy(self.h)
            self.h = None

    def __del__(self):
        self.close()


def keys_of(docs: np.ndarray, mode: str) -> np.ndarray:
    """Pool keys of a trace: the document (position-agnostic) or (document, prompt position) (position-aware)."""
    k = docs.shape[1]
    if mode == "agnostic":
        return docs.reshape(-1)
    if mode == "aware":
        return (docs * k + np.arange(k)[None, :]).reshape(-1)
    raise ValueError(mode)


def hit_ratio(docs: np.ndarray, capacity: int, mode: str) -> float:
    pool = Pool(capacity)
    for key in keys_of(docs, mode):
        pool.acquire(int(key))
    lookups, hits, _, _ = pool.stats()
    pool.close()
    return hits / lookups


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--docs", type=int, default=100_000)
    ap.add_argument("--queries", type=int, default=20_000)
    ap.add_argument("--k", type=int, default=10)
    ap.add_argument("--doc-tokens", type=int, default=512)
    ap.add_argument("--kv-bytes-per-token", type=int, default=131072, help="Llama-3-8B: 32 layers x 8 heads x 128 x 2 x 2 B")
    args = ap.parse_args()
    doc_bytes = args.doc_tokens * args.kv_bytes_per_token
    print(f"{'budget':>8} {'alpha':>6} {'entries':>8} {'agnostic':>9} {'aware':>9} {'ratio':>7}")
    for alpha in (1.1, 1.5, 2.1):
        docs = zipf_trace(args.docs, alpha, args.queries, args.k, seed=int(alpha * 10))
        for gb in (1, 5, 10, 50):
            entries = max(1, int(gb * 2**30 // doc_bytes))
            a = hit_ratio(docs, entries, "agnostic")
            b = hit_ratio(docs, entries, "aware")
            print(f"{gb:>6}GB {alpha:>6.1f} {entries:>8d} {100 * a:>8.2f}% {100 * b:>8.2f}% {a / b if b else float('inf'):>7.2f}")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
