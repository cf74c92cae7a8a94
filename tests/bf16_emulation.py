"""CPU emulation of where the GPU path rounds to bf16, used to size the error bars of the position-discrimination
tests (test infrastructure, like the oracle; nothing on the product path uses it).

The kernels compute in fp32 from bf16 inputs and round at four places: the rotated query (the MFMA operand), the
rotated key, the unnormalised probabilities exp(s - m) that enter the P V product (also summed for the denominator),
and the normalised output.  This module rounds at exactly those places and does everything else in fp64, with the
exact row maximum as the reference (the kernels' lazily moved maximum only scales P by a power of two below 2^8,
which bf16 rounding does not see).  Its error against the fp64 oracle is therefore the error the kernels cannot
avoid; their own fp32 arithmetic adds little to it.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import lazy_oracle as O


def bf16(x):
    """Round to the nearest bf16 value (ties to even), returned as fp64."""
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    b = a.view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return b.astype(np.uint32).view(np.float32).astype(np.float64)


def emulate(w, q=None):
    """Output [total_q, Hq, D] of the emulated bf16 path for a prefill or decode workload (NoPE keys, half-split
    RoPE, the workload's causal flag); ``q`` overrides the workload's queries."""
    q = w.q if q is None else q
    hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
    grp = hq // hkv
    theta = O.rope_frequencies(d, w.rope_base)
    scale = 1.0 / math.sqrt(d)
    q_start = np.arange(w.batch + 1) if w.kind == "decode" else w.q_start
    out = np.zeros((int(q_start[-1]), hq, d))
    for r in range(w.batch):
        a, b = int(q_start[r]), int(q_start[r + 1])
        if b == a:
            continue
        k, v, kpos = O.request_kv(w.pool, w.pool, w.chunks, int(w.chunk_start[r]), int(w.chunk_start[r + 1]), hkv, d)
        kr = bf16(O.rotate(k, kpos, theta))
        qpos = int(w.q_pos0[r]) + np.arange(b - a)
        qr = bf16(O.rotate(np.swapaxes(np.asarray(q[a:b], np.float64), 0, 1), qpos, theta))  # [Hq, n, D]
        vis = (kpos[None, :] <= qpos[:, None]) if w.causal else np.ones((b - a, kpos.size), bool)
        for h in range(hq):
            s = np.where(vis, qr[h] @ kr[h // grp].T * scale, -np.inf)
            m = s.max(axis=1, keepdims=True)
            ok = np.isfinite(m[:, 0])
            p = bf16(np.exp(np.where(ok[:, None], s - np.where(ok[:, None], m, 0.0), -np.inf)))
            den = p.sum(axis=1)
            o = p @ v[h // grp]
            out[a:b, h] = np.where(ok[:, None], bf16(o / np.where(den > 0, den, 1.0)[:, None]), 0.0)
    return out
