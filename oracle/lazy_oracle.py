"""Plain fp64 CPU oracle for LazyAttention's hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this module: only the tests, the package smoke
check and the benchmark's CPU-baseline leg call it.  It shares no code with the HIP library (no kernels, headers,
tables or helpers); both sides only take the same seeded inputs.

What it computes.  LazyAttention is exact: deferring RoPE into the kernel gives the same attention as rotating the
cached keys at their assigned positions and running ordinary attention (Sec. 1, where the method is stated to be
mathematically identical to re-encoding duplicated KV caches; Sec. 3.1 "Deferred encoding").  So the oracle is that
plain definition, written out without tiling, online softmax or any reordering:

1. RoPE frequencies theta_t = base^(-2t/D), t < D/2 (original RoPE, Sec. 3.1 "RoPE attention"), or a given table.
2. Every key of every chunk record is rotated explicitly at its position pos_offset + j with the half-split pairing
   of Sec. 3.2 "Prefilling": k1' = k1 cos(phi) - k2 sin(phi), k2' = k1 sin(phi) + k2 cos(phi), phi = pos * theta_t,
   where (k1, k2) are the two halves of the head dimension.  This is the materialised, re-encoded copy.
3. Every query token is rotated the same way at its own position (Sec. 3.1, f(Q, m)).
4. Scores q'.k' / sqrt(D) (Eqn. standard attention), query head h reads KV head floor(h / G) (Sec. 3.5, GQA).
   A key is visible to a query iff (not causal) or pos_key <= pos_query.
5. Full-row softmax with max subtraction; o = sum(w v) / sum(w); lse = m + ln(sum(w)).  A query that sees no key
   gets o = 0 and lse = -inf.

Key stores come in two conventions (``key_positions``).  "nope": keys are stored without any rotation and key j of a
record is encoded at pos_offset + j (step 2).  "local": the paper's own convention (Sec. 3.2 "Prefilling": each
document's cache keeps local positions indexed from 0, and reuse at offset Delta applies one fixed rotation to the
whole document): the stored key j is already encoded at position j, and re-encoding it at pos_offset + j is the
single rotation R(pos_offset) of the stored vector (the relative-rotation Fact, R(a) R(b) = R(a + b)).

Score-space positions (``pairing="alibi"``, Sec. 3.5 "Score-space positional methods"): nothing is rotated; the
scaled score of a query at m and a key at n gets the bias slope_h * (n - m) (ALiBi), with slope_h = 2^(-8 (h+1) / Hq)
unless a table is given.  The positions come from the chunk table exactly as for RoPE.

Decode is the same computation with one query token per request.  ``merge_partials`` is the plain definition of
combining softmax statistics computed over disjoint key sets.  Parity for all of this is pinned by the CPU tests
(textbook RoPE attention at contiguous positions, the relative-rotation Fact of Sec. 3.2, the rotate-the-query
Example of Sec. 3.1, closed forms and brute force on tiny inputs).
"""
from __future__ import annotations

import math

import numpy as np


def rope_frequencies(head_dim: int, base: float, inv_freq=None) -> np.ndarray:
    """theta_t = base^(-2t/D) for t = 0..D/2-1 in fp64; a given table (RoPE variants, Sec. 3.5) is used verbatim."""
    if inv_freq is not None:
        theta = np.asarray(inv_freq, dtype=np.float64)
        assert theta.shape == (head_dim // 2,)
        return theta
    t = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(np.float64(base), -2.0 * t / head_dim)


def rotate(x: np.ndarray, positions: np.ndarray, theta: np.ndarray, pairing: str = "half") -> np.ndarray:
    """Rotary encoding R(p) of the last axis.  Pair t is rotated by p * theta_t: (x_t, x_{t+D/2}) for the half-split
    pairing of Sec. 3.2 "Prefilling" (the K1/K2 halves), (x_{2t}, x_{2t+1}) for the interleaved pairing used by
    Llama (Sec. 3.5 "RoPE-family variants").

    x: [..., n, D] (any leading axes), positions: [n].  Returns fp64.
    """
    x = np.asarray(x, dtype=np.float64)
    half = x.shape[-1] // 2
    phi = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]  # [n, D/2]
    c, s = np.cos(phi), np.sin(phi)
    if pairing == "half":
        x1, x2 = x[..., :half], x[..., half:]
        return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)
    if pairing == "interleaved":
        x1, x2 = x[..., 0::2], x[..., 1::2]
        y = np.empty_like(x)
        y[..., 0::2] = x1 * c - x2 * s
        y[..., 1::2] = x1 * s + x2 * c
        return y
    raise ValueError(f"unknown pairing {pairing!r}")


def request_kv(pool_k, pool_v, chunks, lo: int, hi: int, num_kv_heads: int, head_dim: int,
               with_offsets: bool = False):
    """Gather one request's stored K, V (in chunk-table order) and the position of every key.

    Record i covers keys j < len at position pos_offset + j; head g of that key is stored at
    k_offset + (g * k_stride + j) * D (V likewise with v_offset / v_stride).
    Returns K [Hkv, L, D], V [Hkv, L, D] (fp64) and positions [L] (int64); with ``with_offsets`` also the
    pos_offset of every key's record [L].
    """
    ks, vs, ps, os_ = [], [], [], []
    d = head_dim
    for i in range(lo, hi):
        rec = chunks[i]
        n = int(rec["len"])
        ko, vo = int(rec["k_offset"]), int(rec["v_offset"])
        kst, vst = int(rec["k_stride"]), int(rec["v_stride"])
        k = np.empty((num_kv_heads, n, d), dtype=np.float64)
        v = np.empty((num_kv_heads, n, d), dtype=np.float64)
        for g in range(num_kv_heads):
            a = ko + g * kst * d
            k[g] = np.asarray(pool_k[a : a + n * d], dtype=np.float64).reshape(n, d)
            b = vo + g * vst * d
            v[g] = np.asarray(pool_v[b : b + n * d], dtype=np.float64).reshape(n, d)
        ks.append(k)
        vs.append(v)
        ps.append(int(rec["pos_offset"]) + np.arange(n, dtype=np.int64))
        os_.append(np.full(n, int(rec["pos_offset"]), dtype=np.int64))
    if not ks:
        z = np.zeros((num_kv_heads, 0, d))
        e = np.zeros(0, dtype=np.int64)
        return (z, z.copy(), e, e.copy()) if with_offsets else (z, z.copy(), e)
    res = (np.concatenate(ks, axis=1), np.concatenate(vs, axis=1), np.concatenate(ps))
    return res + (np.concatenate(os_),) if with_offsets else res


def key_rotation_positions(kpos, offs, key_positions: str):
    """Position by which each stored key is rotated: its full position for a NoPE store, its record's pos_offset
    for a local-position store (the key is already encoded at its local index j)."""
    if key_positions == "nope":
        return kpos
    if key_positions == "local":
        return offs
    raise ValueError(f"unknown key_positions {key_positions!r}")


def alibi_slopes(num_q_heads: int, slopes=None) -> np.ndarray:
    """ALiBi slopes: 2^(-8 (h+1) / Hq) for h < Hq (the geometric sequence of the ALiBi paper for Hq a power of two),
    or a given table verbatim."""
    if slopes is not None:
        return np.asarray(slopes, dtype=np.float64)
    return np.power(2.0, -8.0 * (np.arange(num_q_heads, dtype=np.float64) + 1.0) / num_q_heads)


def attend(q_rot, k_rot, v, q_pos, k_pos, causal: bool, scale: float, slopes=None):
    """Plain softmax attention over explicit, already rotated operands (Eqn. standard attention).

    q_rot [Lq, Hq, D], k_rot / v [Hkv, L, D]; query head h uses KV head h // (Hq / Hkv).  With ``slopes`` [Hq],
    slopes[h] * (k_pos - q_pos) is added to every scaled score of head h (ALiBi).
    Returns o [Lq, Hq, D] and lse [Lq, Hq] (natural log of the sum of exp(score)), fp64.
    """
    lq, hq, d = q_rot.shape
    hkv = k_rot.shape[0]
    group = hq // hkv
    o = np.zeros((lq, hq, d), dtype=np.float64)
    lse = np.full((lq, hq), -np.inf, dtype=np.float64)
    if k_rot.shape[1] == 0:
        return o, lse
    if causal:
        visible = k_pos[None, :] <= q_pos[:, None]  # [Lq, L]
    else:
        visible = np.ones((lq, k_pos.size), dtype=bool)
    any_visible = visible.any(axis=1)
    for h in range(hq):
        g = h // group
        s = (q_rot[:, h, :] @ k_rot[g].T) * scale  # [Lq, L]
        if slopes is not None:
            s = s + slopes[h] * (k_pos[None, :].astype(np.float64) - q_pos[:, None].astype(np.float64))
        s = np.where(visible, s, -np.inf)
        m = np.where(any_visible, s.max(axis=1), 0.0)
        w = np.exp(s - m[:, None])
        den = w.sum(axis=1)
        num = w @ v[g]
        ok = any_visible
        o[ok, h, :] = num[ok] / den[ok, None]
        lse[ok, h] = m[ok] + np.log(den[ok])
    return o, lse


def lazy_attention(q, q_start, q_pos0, pool_k, pool_v, chunks, chunk_start, num_q_heads: int, num_kv_heads: int,
                   head_dim: int, rope_base: float, causal: bool = True, softmax_scale: float | None = None,
                   inv_freq=None, requests=None, key_positions: str = "nope", pairing: str = "half"):
    """Attention of every request's query tokens over its chunk table, keys re-encoded at their positions.

    q [total_q, Hq, D] (NoPE queries), q_start [B+1], q_pos0 [B]: token i of request r is at q_pos0[r] + i.
    key_positions: "nope" or "local" store convention (module docstring); pairing: "half" or "interleaved" RoPE,
    or "alibi" (no rotation; ``inv_freq`` then optionally holds the Hq slopes).
    Returns out [total_q, Hq, D] and lse [total_q, Hq] in fp64.  ``requests`` restricts the work to a subset of
    request indices (other rows stay 0 / -inf).
    """
    assert num_q_heads % num_kv_heads == 0
    scale = 1.0 / math.sqrt(head_dim) if not softmax_scale else float(softmax_scale)
    theta = None if pairing == "alibi" else rope_frequencies(head_dim, rope_base, inv_freq)
    total_q = int(q_start[-1])
    out = np.zeros((total_q, num_q_heads, head_dim), dtype=np.float64)
    lse = np.full((total_q, num_q_heads), -np.inf, dtype=np.float64)
    batch = len(q_start) - 1
    for r in range(batch) if requests is None else requests:
        a, b = int(q_start[r]), int(q_start[r + 1])
        if b == a:
            continue
        k, v, kpos, offs = request_kv(pool_k, pool_v, chunks, int(chunk_start[r]), int(chunk_start[r + 1]),
                                      num_kv_heads, head_dim, with_offsets=True)
        qpos = int(q_pos0[r]) + np.arange(b - a, dtype=np.int64)
        if pairing == "alibi":
            o, l = attend(np.asarray(q[a:b], dtype=np.float64), k, v, qpos, kpos, causal, scale,
                          alibi_slopes(num_q_heads, inv_freq))
        else:
            k_rot = rotate(k, key_rotation_positions(kpos, offs, key_positions), theta, pairing)  # re-encoded copy
            q_rot = rotate(np.swapaxes(np.asarray(q[a:b], dtype=np.float64), 0, 1), qpos, theta, pairing)
            o, l = attend(np.swapaxes(q_rot, 0, 1), k_rot, v, qpos, kpos, causal, scale)
        out[a:b] = o
        lse[a:b] = l
    return out, lse


def lazy_decode(q, q_pos, pool_k, pool_v, chunks, chunk_start, num_q_heads, num_kv_heads, head_dim, rope_base,
                causal=True, softmax_scale=None, inv_freq=None, requests=None, key_positions: str = "nope",
                pairing: str = "half"):
    """One query token per request at q_pos[r] (decode, Sec. 3.2 "Decoding"): q [B, Hq, D]."""
    batch = len(q_pos)
    q_start = np.arange(batch + 1)
    return lazy_attention(q, q_start, q_pos, pool_k, pool_v, chunks, chunk_start, num_q_heads, num_kv_heads,
                          head_dim, rope_base, causal, softmax_scale, inv_freq, requests, key_positions, pairing)


def materialize_k(pool_k, chunks, chunk_start, num_kv_heads: int, head_dim: int, rope_base: float, inv_freq=None,
                  key_positions: str = "nope", pairing: str = "half"):
    """Re-encoded key copy of every request (the materialise-then-attend baseline's first step): a list over
    requests of K' [Hkv, L_r, D], keys in chunk-table order, each encoded at pos_offset + j."""
    theta = rope_frequencies(head_dim, rope_base, inv_freq)
    res = []
    for r in range(len(chunk_start) - 1):
        k, _, kpos, offs = request_kv(pool_k, pool_k, chunks, int(chunk_start[r]), int(chunk_start[r + 1]),
                                      num_kv_heads, head_dim, with_offsets=True)
        res.append(rotate(k, key_rotation_positions(kpos, offs, key_positions), theta, pairing))
    return res


def partial_softmax(q_rot, k_rot, v, q_pos, k_pos, causal: bool, scale: float):
    """Softmax statistics over one subset of keys: m (max score), l (sum of exp(s - m)), acc (sum of exp(s - m) v).

    Shapes as in ``attend``; returns m [Lq, Hq], l [Lq, Hq], acc [Lq, Hq, D].  An empty or fully hidden subset
    gives m = -inf, l = 0, acc = 0.
    """
    lq, hq, d = q_rot.shape
    hkv = k_rot.shape[0]
    group = hq // hkv
    m = np.full((lq, hq), -np.inf)
    l = np.zeros((lq, hq))
    acc = np.zeros((lq, hq, d))
    if k_rot.shape[1] == 0:
        return m, l, acc
    visible = (k_pos[None, :] <= q_pos[:, None]) if causal else np.ones((lq, k_pos.size), dtype=bool)
    for h in range(hq):
        s = np.where(visible, (q_rot[:, h, :] @ k_rot[h // group].T) * scale, -np.inf)
        mh = s.max(axis=1)
        fin = np.isfinite(mh)
        w = np.zeros_like(s)
        w[fin] = np.exp(s[fin] - mh[fin, None])
        m[:, h] = mh
        l[:, h] = w.sum(axis=1)
        acc[:, h, :] = w @ v[h // group]
    return m, l, acc


def merge_partials(m, l, acc):
    """Combine statistics over disjoint key sets s: with M = max_s m_s and w_s = exp(m_s - M),
    o = sum_s w_s acc_s / sum_s w_s l_s and lse = M + ln(sum_s w_s l_s).

    m, l: [S, ...]; acc: [S, ..., D].  Rows where every m_s is -inf give o = 0, lse = -inf.
    """
    m = np.asarray(m, dtype=np.float64)
    l = np.asarray(l, dtype=np.float64)
    acc = np.asarray(acc, dtype=np.float64)
    big = m.max(axis=0)
    fin = np.isfinite(big)
    safe = np.where(fin, big, 0.0)
    w = np.where(np.isfinite(m), np.exp(m - safe[None]), 0.0)
    den = (w * l).sum(axis=0)
    num = (w[..., None] * acc).sum(axis=0)
    ok = fin & (den > 0)
    o = np.zeros_like(num)
    o[ok] = num[ok] / den[ok][..., None]
    lse = np.full(big.shape, -np.inf)
    lse[ok] = big[ok] + np.log(den[ok])
    return o, lse
