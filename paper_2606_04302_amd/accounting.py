"""Algorithmic work of one attention launch, used for roofline fractions.

Useful FLOPs follow the paper's count for the two attention GEMMs (Sec. 3.2: 4 M N D FLOPs per query/key tile pair,
multiply and add counted separately), restricted to (query, key) pairs the causal rule leaves visible:
``4 * D * Hq * visible_pairs``.  Rotation work is overhead and never counted as useful.

Algorithmic bytes are what one launch must move at least once: K and V of every key of every request for one KV
head layout (each request reads its own table, so shared chunks count once per request that uses them: the
"logical" bytes), plus Q in and O out.  Unique pool bytes (each physical chunk once) are reported separately.
"""
from __future__ import annotations

import numpy as np


def visible_pairs(q_start, q_pos0, chunks, chunk_start, causal: bool = True) -> int:
    total = 0
    for r in range(len(q_start) - 1):
        lq = int(q_start[r + 1]) - int(q_start[r])
        if lq == 0:
            continue
        qpos = int(q_pos0[r]) + np.arange(lq, dtype=np.int64)
        for i in range(int(chunk_start[r]), int(chunk_start[r + 1])):
            n = int(chunks[i]["len"])
            p0 = int(chunks[i]["pos_offset"])
            if causal:
                total += int(np.clip(qpos - p0 + 1, 0, n).sum())
            else:
                total += n * lq
    return total


def useful_flops(w) -> int:
    return 4 * w.head_dim * w.num_q_heads * visible_pairs(w.q_start, w.q_pos0, w.chunks, w.chunk_start, w.causal)


def logical_kv_bytes(w, elem_bytes: int = 2) -> int:
    """K and V read once per (request, KV head): sum over requests of L_r * Hkv * D * 2 tensors."""
    return int(w.kv_lens.sum()) * w.num_kv_heads * w.head_dim * 2 * elem_bytes


def unique_kv_bytes(w, elem_bytes: int = 2) -> int:
    """Each distinct stored chunk counted once, at the largest length any request uses."""
    seen = {}
    for rec in w.chunks:
        key = (int(rec["k_offset"]), int(rec["v_offset"]))
        seen[key] = max(seen.get(key, 0), int(rec["len"]))
    return sum(seen.values()) * w.num_kv_heads * w.head_dim * 2 * elem_bytes


def qo_bytes(w, elem_bytes: int = 2) -> int:
    return 2 * w.total_q * w.num_q_heads * w.head_dim * elem_bytes


def algorithmic_bytes(w, elem_bytes: int = 2) -> int:
    return logical_kv_bytes(w, elem_bytes) + qo_bytes(w, elem_bytes)


def materialize_bytes(w, elem_bytes: int = 2) -> int:
    """Rotate-and-copy of K: every request's keys read once and written once."""
    return 2 * int(w.kv_lens.sum()) * w.num_kv_heads * w.head_dim * elem_bytes
