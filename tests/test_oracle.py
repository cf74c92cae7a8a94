"""CPU pins for the fp64 oracle.  Each test checks the oracle against something other than itself: textbook RoPE
attention written independently (complex multiplication + torch's fp64 attention), the paper's relative-rotation
Fact and rotate-the-query Example, closed forms, a hand-derived worked example, and pure-Python brute force."""
import cmath
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import lazy_oracle as O
from paper_2606_04302_amd import accounting, workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def run(w, **kw):
    return O.lazy_attention(w.q, w.q_start, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, w.num_q_heads,
                            w.num_kv_heads, w.head_dim, w.rope_base, w.causal, **kw)


def contiguous_workload(seed=0, hq=4, hkv=2, d=16, base=1.0e4, lens=(5, 7, 3), q_len=4, batch=2):
    reqs = []
    for r in range(batch):
        pos, ch = 0, []
        for n in lens:
            ch.append((n, pos))
            pos += n
        ch.append((q_len, pos))
        reqs.append(dict(chunks=ch, q_len=q_len, q_pos0=pos))
    return W.custom(seed, hq, hkv, d, base, reqs)


def textbook_rope_attention(w):
    """Independent reference: RoPE as multiplication of (x_t + i x_{t+D/2}) by exp(i p theta_t), then torch's
    fp64 scaled_dot_product_attention with an explicit causal (key index <= query position) mask."""
    d = w.head_dim
    half = d // 2
    theta = torch.tensor([w.rope_base ** (-2.0 * t / d) for t in range(half)], dtype=torch.float64)
    outs = []
    for r in range(w.batch):
        k_parts, v_parts = [], []
        for i in range(w.chunk_start[r], w.chunk_start[r + 1]):
            rec = w.chunks[i]
            n = int(rec["len"])
            k = np.stack([w.pool[int(rec["k_offset"]) + g * int(rec["k_stride"]) * d:][: n * d].reshape(n, d)
                          for g in range(w.num_kv_heads)])
            v = np.stack([w.pool[int(rec["v_offset"]) + g * int(rec["v_stride"]) * d:][: n * d].reshape(n, d)
                          for g in range(w.num_kv_heads)])
            k_parts.append(k)
            v_parts.append(v)
        k = torch.tensor(np.concatenate(k_parts, 1), dtype=torch.float64)
        v = torch.tensor(np.concatenate(v_parts, 1), dtype=torch.float64)
        L = k.shape[1]
        a, b = int(w.q_start[r]), int(w.q_start[r + 1])
        q = torch.tensor(w.q[a:b], dtype=torch.float64).transpose(0, 1)  # [Hq, Lq, D]
        qpos = torch.arange(int(w.q_pos0[r]), int(w.q_pos0[r]) + (b - a), dtype=torch.float64)
        kpos = torch.arange(L, dtype=torch.float64)

        def rope(x, pos):
            z = torch.complex(x[..., :half], x[..., half:]) * torch.polar(torch.ones_like(pos[:, None] * theta),
                                                                          pos[:, None] * theta)
            return torch.cat([z.real, z.imag], -1)

        qr, kr = rope(q, qpos), rope(k, kpos)
        g = w.num_q_heads // w.num_kv_heads
        kr = kr.repeat_interleave(g, 0)
        vv = v.repeat_interleave(g, 0)
        mask = kpos[None, :] <= qpos[:, None]
        o = torch.nn.functional.scaled_dot_product_attention(qr, kr, vv, attn_mask=mask)
        outs.append(o.transpose(0, 1).numpy())
    return np.concatenate(outs, 0)


def test_equals_textbook_rope_attention_at_contiguous_positions():
    w = contiguous_workload()
    out, _ = run(w)
    ref = textbook_rope_attention(w)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_equals_textbook_on_tiny_rag_workload():
    w = W.tiny_rag_prefill(seed=0)
    out, _ = run(w)
    np.testing.assert_allclose(out, textbook_rope_attention(w), rtol=0, atol=1e-12)


@pytest.mark.parametrize("shift", [1, 1000, 100000])
def test_relative_rotation_fact_shift_invariance(shift):
    """Fact (Sec. 3.2): scores depend only on n - m, so moving every key and query by the same amount changes
    nothing."""
    w = W.rag_prefill(seed=5, batch=2, hq=4, hkv=2, d=32, prefix_len=8, n_chunks=3, chunk_len=16,
                      pool_chunks=6, q_len=5)
    out0, lse0 = run(w)
    w2 = W.Workload(**{**w.__dict__})
    w2.chunks = w.chunks.copy()
    w2.chunks["pos_offset"] += shift
    w2.q_pos0 = w.q_pos0 + shift
    out1, lse1 = run(w2)
    np.testing.assert_allclose(out1, out0, rtol=0, atol=1e-9)
    np.testing.assert_allclose(lse1, lse0, rtol=0, atol=1e-9)


def test_example_rotate_query_back():
    """Example (Sec. 3.1): using a cache indexed from 0 after a document of length n1 is the same as rotating the
    query back by n1.  Here: chunk at offset n1 with the query at m  ==  chunk at offset 0 with the query at m - n1,
    checked on raw scores through lse with a one-token value."""
    d, n1, n2, m = 8, 11, 6, 40
    rng = np.random.default_rng(3)
    theta = O.rope_frequencies(d, 1e4)
    k = rng.standard_normal((1, n2, d))
    q = rng.standard_normal((1, 1, d))
    s_a = O.rotate(q[0], np.array([m]), theta) @ O.rotate(k, n1 + np.arange(n2), theta)[0].T
    s_b = O.rotate(q[0], np.array([m - n1]), theta) @ O.rotate(k, np.arange(n2), theta)[0].T
    np.testing.assert_allclose(s_a, s_b, rtol=0, atol=1e-12)
    # and through the full attention path
    reqs_a = [dict(chunks=[("doc", n2, n1)], q_len=1, q_pos0=m)]
    reqs_b = [dict(chunks=[("doc", n2, 0)], q_len=1, q_pos0=m - n1)]
    wa = W.custom(9, 2, 1, d, 1e4, reqs_a)
    wb = W.custom(9, 2, 1, d, 1e4, reqs_b)
    np.testing.assert_array_equal(wa.pool, wb.pool)
    oa, la = run(wa)
    ob, lb = run(wb)
    np.testing.assert_allclose(oa, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(la, lb, rtol=0, atol=1e-12)


def test_chunk_table_permutation_invariance():
    w = W.rag_prefill(seed=7, batch=3, hq=4, hkv=2, d=16, prefix_len=4, n_chunks=4, chunk_len=8, pool_chunks=9,
                      q_len=3)
    out0, _ = run(w)
    rng = np.random.default_rng(0)
    w2 = W.Workload(**{**w.__dict__})
    w2.chunks = w.chunks.copy()
    for r in range(w.batch):
        a, b = int(w.chunk_start[r]), int(w.chunk_start[r + 1])
        w2.chunks[a:b] = w.chunks[a:b][rng.permutation(b - a)]
    out1, _ = run(w2)
    np.testing.assert_allclose(out1, out0, rtol=0, atol=1e-12)


def test_d2_closed_form():
    """D = 2, theta_0 = 1: (R_m q).(R_n k) = |q||k| cos(phi_k - phi_q + (n - m)); softmax over those / sqrt(2)."""
    reqs = [dict(chunks=[(3, 2), (2, 9)], q_len=2, q_pos0=12)]
    w = W.custom(11, 1, 1, 2, 1e4, reqs)
    out, lse = run(w)
    keys, vals, kpos = [], [], []
    for rec in w.chunks:
        for j in range(int(rec["len"])):
            keys.append(complex(*w.pool[int(rec["k_offset"]) + 2 * j:][:2]))
            vals.append(w.pool[int(rec["v_offset"]) + 2 * j:][:2].astype(float))
            kpos.append(int(rec["pos_offset"]) + j)
    for i in range(2):
        qc = complex(*w.q[i, 0])
        m = 12 + i
        sc = [abs(qc) * abs(kc) * math.cos(cmath.phase(kc) - cmath.phase(qc) + (n - m)) / math.sqrt(2)
              for kc, n in zip(keys, kpos)]
        vis = [n <= m for n in kpos]
        mx = max(s for s, ok in zip(sc, vis) if ok)
        ws = [math.exp(s - mx) if ok else 0.0 for s, ok in zip(sc, vis)]
        den = sum(ws)
        o = sum(wt * v for wt, v in zip(ws, vals)) / den
        np.testing.assert_allclose(out[i, 0], o, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[i, 0], mx + math.log(den), rtol=0, atol=1e-12)


def test_golden_quarter_turn_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "quarter_turn.json")))
    d = g["head_dim"]
    theta = O.rope_frequencies(d, 1e4, g["inv_freq"])
    q = O.rotate(np.array([g["q"]]), np.array([g["q_pos"]]), theta)  # [1, 1, D]
    k = O.rotate(np.array([g["keys"]]), np.array(g["key_pos"]), theta)
    v = np.array([g["values"]], dtype=np.float64)
    o, lse = O.attend(q.reshape(1, 1, d), k, v, np.array([g["q_pos"]]), np.array(g["key_pos"]), True,
                      g["softmax_scale"])
    np.testing.assert_allclose(o[0, 0], g["expected_out"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse[0, 0], g["expected_lse"], rtol=0, atol=1e-15)


def test_all_positions_zero_is_plain_softmax_attention():
    reqs = [dict(chunks=[(1, 0)] * 6, q_len=1, q_pos0=0)]
    w = W.custom(13, 2, 1, 8, 1e4, reqs)
    out, _ = run(w)
    k = np.stack([w.pool[int(r["k_offset"]):][:8] for r in w.chunks]).astype(float)
    v = np.stack([w.pool[int(r["v_offset"]):][:8] for r in w.chunks]).astype(float)
    for h in range(2):
        s = k @ w.q[0, h].astype(float) / math.sqrt(8)
        p = np.exp(s - s.max())
        p /= p.sum()
        np.testing.assert_allclose(out[0, h], p @ v, rtol=0, atol=1e-13)


def test_single_visible_key_and_constant_values():
    # first query token at position 5 sees only the key at position 5
    reqs = [dict(chunks=[(4, 5)], q_len=2, q_pos0=5)]
    w = W.custom(17, 2, 1, 8, 1e4, reqs)
    out, _ = run(w)
    rec = w.chunks[0]
    v0 = w.pool[int(rec["v_offset"]):][:8]
    np.testing.assert_allclose(out[0, 0], v0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(out[0, 1], v0, rtol=0, atol=1e-14)
    # all value rows equal -> output equals that row whatever the weights
    w.pool[int(rec["v_offset"]): int(rec["v_offset"]) + 4 * 8] = np.tile(np.arange(8, dtype=np.float32), 4)
    out, _ = run(w)
    np.testing.assert_allclose(out[1, :], np.tile(np.arange(8.0), (2, 1)), rtol=0, atol=1e-13)


def test_visible_count_through_lse():
    """With q = 0 every score is 0, so lse = ln(#visible keys) and #visible = #{pos_k <= pos_q}."""
    reqs = [dict(chunks=[(5, 0), (3, 20), (4, 7)], q_len=6, q_pos0=4)]
    w = W.custom(19, 2, 1, 8, 1e4, reqs)
    w.q[:] = 0
    _, lse = run(w)
    kpos = np.concatenate([np.arange(5), 20 + np.arange(3), 7 + np.arange(4)])
    for i in range(6):
        cnt = int((kpos <= 4 + i).sum())
        np.testing.assert_allclose(lse[i], math.log(cnt), rtol=0, atol=1e-14)


def test_no_visible_key_gives_zero_and_minus_inf():
    reqs = [dict(chunks=[(4, 50)], q_len=2, q_pos0=10)]
    w = W.custom(23, 2, 1, 8, 1e4, reqs)
    out, lse = run(w)
    assert np.all(out == 0) and np.all(np.isneginf(lse))


def test_decode_equals_prefill_with_one_query():
    w = W.rag_decode(seed=3, batch=3, hq=4, hkv=2, d=16, n_chunks=3, chunk_len=9, pool_chunks=5, tail_len=4,
                     tail_cap=8)
    od, ld = O.lazy_decode(w.q, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, w.num_q_heads,
                           w.num_kv_heads, w.head_dim, w.rope_base)
    op, lp = run(w)
    np.testing.assert_array_equal(od, op)
    np.testing.assert_array_equal(ld, lp)


def brute_force(w):
    """Scalar loops with math.cos / math.sin straight from the rotation formula and the softmax definition."""
    d, half = w.head_dim, w.head_dim // 2
    theta = [w.rope_base ** (-2.0 * t / d) for t in range(half)]
    g = w.num_q_heads // w.num_kv_heads

    def rot(x, p):
        y = [0.0] * d
        for t in range(half):
            c, s = math.cos(p * theta[t]), math.sin(p * theta[t])
            y[t] = x[t] * c - x[t + half] * s
            y[t + half] = x[t] * s + x[t + half] * c
        return y

    out = np.zeros(w.q.shape)
    for r in range(w.batch):
        keys = []
        for i in range(w.chunk_start[r], w.chunk_start[r + 1]):
            rec = w.chunks[i]
            for j in range(int(rec["len"])):
                for h in range(w.num_kv_heads):
                    pass
                keys.append((int(rec["pos_offset"]) + j, rec, j))
        for qi in range(int(w.q_start[r]), int(w.q_start[r + 1])):
            m = int(w.q_pos0[r]) + qi - int(w.q_start[r])
            for h in range(w.num_q_heads):
                kv = h // g
                qr = rot([float(x) for x in w.q[qi, h]], m)
                sc, vs = [], []
                for p, rec, j in keys:
                    if p > m:
                        continue
                    a = int(rec["k_offset"]) + (kv * int(rec["k_stride"]) + j) * d
                    b = int(rec["v_offset"]) + (kv * int(rec["v_stride"]) + j) * d
                    kr = rot([float(x) for x in w.pool[a:a + d]], p)
                    sc.append(sum(x * y for x, y in zip(qr, kr)) / math.sqrt(d))
                    vs.append([float(x) for x in w.pool[b:b + d]])
                mx = max(sc)
                ws = [math.exp(s - mx) for s in sc]
                den = sum(ws)
                for e in range(d):
                    out[qi, h, e] = sum(wt * v[e] for wt, v in zip(ws, vs)) / den
    return out


def test_brute_force_tiny_gqa():
    reqs = [dict(chunks=[("a", 3, 7), (2, 0), ("b", 2, 2)], q_len=3, q_pos0=10),
            dict(chunks=[("b", 2, 30), ("a", 3, 0), (3, 33)], q_len=3, q_pos0=33)]
    w = W.custom(29, 4, 2, 6, 100.0, reqs)
    out, _ = run(w)
    np.testing.assert_allclose(out, brute_force(w), rtol=0, atol=1e-12)


def test_merge_of_partials_equals_unsplit():
    w = W.rag_prefill(seed=31, batch=1, hq=4, hkv=2, d=16, prefix_len=8, n_chunks=3, chunk_len=12,
                      pool_chunks=5, q_len=6)
    theta = O.rope_frequencies(16, w.rope_base)
    k, v, kpos = O.request_kv(w.pool, w.pool, w.chunks, 0, int(w.chunk_start[1]), 2, 16)
    qpos = int(w.q_pos0[0]) + np.arange(6)
    qr = O.rotate(np.swapaxes(w.q.astype(float), 0, 1), qpos, theta).swapaxes(0, 1)
    kr = O.rotate(k, kpos, theta)
    full_o, full_lse = O.attend(qr, kr, v, qpos, kpos, True, 0.25)
    rng = np.random.default_rng(1)
    L = kpos.size
    for parts in (1, 2, 5, 9):
        cuts = np.sort(rng.choice(np.arange(1, L), size=parts - 1, replace=False)) if parts > 1 else []
        bounds = [0, *cuts, L]
        ms, ls, accs = [], [], []
        for a, b in zip(bounds[:-1], bounds[1:]):
            m, l, acc = O.partial_softmax(qr, kr[:, a:b], v[:, a:b], qpos, kpos[a:b], True, 0.25)
            ms.append(m), ls.append(l), accs.append(acc)
        # an empty split as well
        m, l, acc = O.partial_softmax(qr, kr[:, :0], v[:, :0], qpos, kpos[:0], True, 0.25)
        ms.append(m), ls.append(l), accs.append(acc)
        o, lse = O.merge_partials(np.stack(ms), np.stack(ls), np.stack(accs))
        np.testing.assert_allclose(o, full_o, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, full_lse, rtol=0, atol=1e-12)


def test_materialized_keys_match_textbook_rotation():
    w = W.rag_prefill(seed=37, batch=2, hq=4, hkv=2, d=8, prefix_len=3, n_chunks=2, chunk_len=5, pool_chunks=4,
                      q_len=2)
    ks = O.materialize_k(w.pool, w.chunks, w.chunk_start, 2, 8, w.rope_base)
    theta = [w.rope_base ** (-2.0 * t / 8) for t in range(4)]
    for r in range(2):
        k, _, kpos = O.request_kv(w.pool, w.pool, w.chunks, int(w.chunk_start[r]), int(w.chunk_start[r + 1]), 2, 8)
        for g in range(2):
            for j, p in enumerate(kpos):
                z = [complex(k[g, j, t], k[g, j, t + 4]) * cmath.exp(1j * p * theta[t]) for t in range(4)]
                ref = [c.real for c in z] + [c.imag for c in z]
                np.testing.assert_allclose(ks[r][g, j], ref, rtol=0, atol=1e-12)


def test_positions_matter():
    """Moving one chunk by a single position changes the output by far more than rounding."""
    w = W.tiny_rag_prefill(seed=0)
    out0, _ = run(w)
    w2 = W.Workload(**{**w.__dict__})
    w2.chunks = w.chunks.copy()
    w2.chunks["pos_offset"][2] += 1
    out1, _ = run(w2)
    assert np.abs(out1 - out0).max() > 1e-2


def test_non_causal_sees_every_key():
    reqs = [dict(chunks=[(4, 50)], q_len=2, q_pos0=10)]
    w = W.custom(41, 2, 1, 8, 1e4, reqs, causal=False)
    w.q[:] = 0
    _, lse = run(w)
    np.testing.assert_allclose(lse, math.log(4), rtol=0, atol=1e-14)


def test_visible_pair_accounting_matches_oracle_visibility():
    w = W.varlen_rag(seed=4, batch=3, hq=4, hkv=1, d=8, pool_chunks=12, len_lo=3, len_hi=20, k_lo=2, k_hi=5,
                     q_lo=1, q_hi=9)
    cnt = 0
    for r in range(w.batch):
        _, _, kpos = O.request_kv(w.pool, w.pool, w.chunks, int(w.chunk_start[r]), int(w.chunk_start[r + 1]), 1, 8)
        qpos = int(w.q_pos0[r]) + np.arange(int(w.q_lens[r]))
        cnt += int((kpos[None, :] <= qpos[:, None]).sum())
    assert accounting.visible_pairs(w.q_start, w.q_pos0, w.chunks, w.chunk_start) == cnt
    # the tiny RAG workload's count: 256 keys before the query + 1..16 of its own
    t = W.tiny_rag_prefill()
    assert accounting.visible_pairs(t.q_start, t.q_pos0, t.chunks, t.chunk_start) == 16 * 256 + 136
    assert accounting.useful_flops(t) == 4 * 64 * 2 * (16 * 256 + 136)


def test_bf16_rounding_is_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, np.inf], dtype=np.float32)
    r = W.bf16_round(x)
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(r, ref)
    y = np.random.default_rng(0).standard_normal(100000).astype(np.float32)
    np.testing.assert_array_equal(W.bf16_round(y), torch.tensor(y).to(torch.bfloat16).float().numpy())


def test_brute_force_decode_with_capacity_slack():
    """Tails whose capacity exceeds their length: head g of a key lives at offset + (g * stride + j) * D."""
    w = W.rag_decode(seed=43, batch=2, hq=4, hkv=2, d=6, n_chunks=2, chunk_len=3, pool_chunks=3, tail_len=3,
                     tail_cap=7)
    assert (w.chunks["k_stride"] > w.chunks["len"]).any()
    out, _ = run(w)
    np.testing.assert_allclose(out, brute_force(w), rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------------------------------------------
# Local-position key stores (Sec. 3.2 "Prefilling": each document's cache is kept at local positions from 0 and
# reused at offset Delta with one fixed rotation; "Decoding": the query is rotated by the relative offset instead).
# ---------------------------------------------------------------------------------------------------------------
def local_store_from_nope(w):
    """A local-position copy of a NoPE pool, written independently of the oracle: capacity slot j of every physical
    chunk's K is multiplied, as the complex vector x_t + i x_{t+D/2}, by exp(i j theta_t).  V is left alone."""
    d = w.head_dim
    half = d // 2
    theta = np.array([w.rope_base ** (-2.0 * t / d) for t in range(half)])
    pool = w.pool.astype(np.float64).copy()
    done = set()
    for rec in w.chunks:
        ko, cap = int(rec["k_offset"]), int(rec["k_stride"])
        if ko in done:
            continue
        done.add(ko)
        for g in range(w.num_kv_heads):
            for j in range(cap):
                a = ko + (g * cap + j) * d
                x = pool[a: a + d]
                z = (x[:half] + 1j * x[half:]) * np.exp(1j * j * theta)
                pool[a: a + d] = np.concatenate([z.real, z.imag])
    return pool


def test_local_store_bridge_identity_prefill():
    """k_local = R(j) k_nope: a local-position store used with one rotation by pos_offset gives exactly the NoPE
    store's attention (shared chunks at different offsets, a causal query chunk, GQA)."""
    w = W.rag_prefill(seed=21, batch=3, hq=4, hkv=2, d=16, prefix_len=5, n_chunks=3, chunk_len=9, pool_chunks=4,
                      q_len=6)
    out0, lse0 = run(w)
    local = local_store_from_nope(w)
    out1, lse1 = O.lazy_attention(w.q, w.q_start, w.q_pos0, local, local, w.chunks, w.chunk_start, w.num_q_heads,
                                  w.num_kv_heads, w.head_dim, w.rope_base, w.causal, key_positions="local")
    np.testing.assert_allclose(out1, out0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse1, lse0, rtol=0, atol=1e-11)
    # the materialised copies agree as well
    m0 = O.materialize_k(w.pool, w.chunks, w.chunk_start, 2, 16, w.rope_base)
    m1 = O.materialize_k(local, w.chunks, w.chunk_start, 2, 16, w.rope_base, key_positions="local")
    for a, b in zip(m0, m1):
        np.testing.assert_allclose(b, a, rtol=0, atol=1e-12)


def test_local_store_bridge_identity_decode_with_capacity():
    w = W.rag_decode(seed=22, batch=3, hq=6, hkv=2, d=16, n_chunks=3, chunk_len=12, pool_chunks=4, tail_len=5,
                     tail_cap=9)
    o0, l0 = O.lazy_decode(w.q, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, 6, 2, 16, w.rope_base)
    local = local_store_from_nope(w)
    o1, l1 = O.lazy_decode(w.q, w.q_pos0, local, local, w.chunks, w.chunk_start, 6, 2, 16, w.rope_base,
                           key_positions="local")
    np.testing.assert_allclose(o1, o0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(l1, l0, rtol=0, atol=1e-11)


def test_local_store_decode_rotates_query_by_relative_offset():
    """Sec. 3.2 "Decoding": with local keys the query at m is rotated by m - Delta and meets the stored keys as they
    are.  Brute force in pure Python (complex arithmetic) on lse, for two chunks at different offsets."""
    d, base = 8, 1.0e4
    reqs = [dict(chunks=[("a", 5, 30), ("b", 4, 7)], q_len=1, q_pos0=61)]
    w = W.custom(23, 1, 1, d, base, reqs, kind="decode")
    _, lse = O.lazy_decode(w.q, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, 1, 1, d, base,
                           key_positions="local")
    half = d // 2
    th = [base ** (-2.0 * t / d) for t in range(half)]
    q = [complex(float(w.q[0, 0, t]), float(w.q[0, 0, t + half])) for t in range(half)]
    scores = []
    for rec in w.chunks:
        delta = int(rec["pos_offset"])
        rel = int(w.q_pos0[0]) - delta
        qr = [q[t] * cmath.exp(1j * rel * th[t]) for t in range(half)]
        for j in range(int(rec["len"])):
            a = int(rec["k_offset"]) + j * d
            k = [complex(float(w.pool[a + t]), float(w.pool[a + t + half])) for t in range(half)]
            scores.append(sum((qr[t].conjugate() * k[t]).real for t in range(half)) / math.sqrt(d))
    mx = max(scores)
    ref = mx + math.log(sum(math.exp(s - mx) for s in scores))
    assert abs(lse[0, 0] - ref) < 1e-12


def test_unknown_key_convention_is_rejected():
    w = W.tiny_rag_prefill(seed=0)
    with pytest.raises(ValueError):
        run(w, key_positions="absolute")


def test_paged_store_is_the_same_attention():
    """Paged (block-granular) copies of a store change only where keys live, not which keys sit at which positions:
    the oracle's result is unchanged (prefill with a causal query chunk, decode with capacity slack)."""
    w = W.rag_prefill(seed=31, batch=2, hq=4, hkv=2, d=16, prefix_len=7, n_chunks=3, chunk_len=50, pool_chunks=4,
                      q_len=9)
    for bt in (16, 64):
        p = W.paginate(w, bt, seed=bt)
        assert len(p.chunks) >= len(w.chunks) and p.meta["block_tokens"] == bt
        assert bt > 50 or len(p.chunks) > len(w.chunks)
        a, la = run(w)
        b, lb = run(p)
        np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(la, lb)
    d = W.rag_decode(seed=32, batch=3, hq=4, hkv=2, d=16, n_chunks=2, chunk_len=70, pool_chunks=3, tail_len=5,
                     tail_cap=40)
    p = W.paginate(d, 32, seed=3)
    a, _ = O.lazy_decode(d.q, d.q_pos0, d.pool, d.pool, d.chunks, d.chunk_start, 4, 2, 16, d.rope_base)
    b, _ = O.lazy_decode(p.q, p.q_pos0, p.pool, p.pool, p.chunks, p.chunk_start, 4, 2, 16, p.rope_base)
    np.testing.assert_array_equal(a, b)


# ---------------------------------------------------------------------------------------------------------------
# Interleaved RoPE pairing (Sec. 3.5 "RoPE-family variants": pairs (2t, 2t+1), as used by Llama).
# ---------------------------------------------------------------------------------------------------------------
def test_interleaved_pairing_brute_force():
    """Pure-Python complex arithmetic, z_t = x_{2t} + i x_{2t+1} rotated by exp(i p theta_t), on decode lse."""
    d, base = 8, 1.0e4
    reqs = [dict(chunks=[(6, 3), (4, 20)], q_len=1, q_pos0=31)]
    w = W.custom(41, 1, 1, d, base, reqs, kind="decode")
    _, lse = O.lazy_decode(w.q, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, 1, 1, d, base,
                           pairing="interleaved")
    th = [base ** (-2.0 * t / d) for t in range(d // 2)]
    m = int(w.q_pos0[0])
    q = [complex(float(w.q[0, 0, 2 * t]), float(w.q[0, 0, 2 * t + 1])) * cmath.exp(1j * m * th[t])
         for t in range(d // 2)]
    scores = []
    for rec in w.chunks:
        for j in range(int(rec["len"])):
            a = int(rec["k_offset"]) + j * d
            p = int(rec["pos_offset"]) + j
            k = [complex(float(w.pool[a + 2 * t]), float(w.pool[a + 2 * t + 1])) * cmath.exp(1j * p * th[t])
                 for t in range(d // 2)]
            scores.append(sum((q[t].conjugate() * k[t]).real for t in range(d // 2)) / math.sqrt(d))
    mx = max(scores)
    ref = mx + math.log(sum(math.exp(s - mx) for s in scores))
    assert abs(lse[0, 0] - ref) < 1e-12


def test_interleaved_equals_half_split_on_permuted_queries_and_keys():
    """Interleaved RoPE on (q, k) is half-split RoPE on (P q, P k) with P: 2t -> t, 2t+1 -> t + D/2 (values are not
    permuted).  Both key conventions."""
    w = W.rag_prefill(seed=42, batch=2, hq=4, hkv=2, d=16, prefix_len=5, n_chunks=3, chunk_len=11, pool_chunks=4,
                      q_len=6)
    d = w.head_dim
    perm = np.concatenate([np.arange(0, d, 2), np.arange(1, d, 2)])  # new index t holds old index perm[t]
    pool = w.pool.copy()
    done = set()
    for rec in w.chunks:
        ko, cap = int(rec["k_offset"]), int(rec["k_stride"])
        if ko in done:
            continue
        done.add(ko)
        blk = pool[ko: ko + w.num_kv_heads * cap * d].reshape(-1, d)
        blk[:] = blk[:, perm]
    q = w.q[..., perm]
    for kp in ("nope", "local"):
        a, la = O.lazy_attention(w.q, w.q_start, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, 4, 2, d,
                                 w.rope_base, key_positions=kp, pairing="interleaved")
        b, lb = O.lazy_attention(q, w.q_start, w.q_pos0, pool, pool, w.chunks, w.chunk_start, 4, 2, d, w.rope_base,
                                 key_positions=kp, pairing="half")
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
        np.testing.assert_allclose(la, lb, rtol=0, atol=1e-11)


def test_unknown_pairing_is_rejected():
    with pytest.raises(ValueError):
        O.rotate(np.zeros((1, 4)), np.zeros(1), np.ones(2), pairing="swapped")


# ---------------------------------------------------------------------------------------------------------------
# ALiBi (Sec. 3.5 "Score-space positional methods"): no rotation, bias slope_h * (k_pos - q_pos) on the scaled score.
# ---------------------------------------------------------------------------------------------------------------
def test_alibi_brute_force():
    d = 8
    reqs = [dict(chunks=[(5, 2), (3, 40), (2, 44)], q_len=2, q_pos0=44)]
    w = W.custom(51, 4, 2, d, 1.0, reqs)
    _, lse = run(w, pairing="alibi")
    for tok in range(2):
        m = 44 + tok
        for h in range(4):
            slope = 2.0 ** (-8.0 * (h + 1) / 4)
            g = h // 2
            scores = []
            for rec in w.chunks:
                for j in range(int(rec["len"])):
                    n = int(rec["pos_offset"]) + j
                    if n > m:
                        continue
                    a = int(rec["k_offset"]) + (g * int(rec["k_stride"]) + j) * d
                    dot = sum(float(w.q[tok, h, t]) * float(w.pool[a + t]) for t in range(d))
                    scores.append(dot / math.sqrt(d) + slope * (n - m))
            mx = max(scores)
            ref = mx + math.log(sum(math.exp(s - mx) for s in scores))
            assert abs(lse[tok, h] - ref) < 1e-12


def test_alibi_zero_slopes_is_attention_without_positions_and_shift_invariant():
    w = W.rag_prefill(seed=52, batch=2, hq=4, hkv=2, d=16, prefix_len=5, n_chunks=3, chunk_len=11, pool_chunks=4,
                      q_len=6)
    w.causal = False
    zero = np.zeros(4)
    a, _ = run(w, pairing="alibi", inv_freq=zero)
    # positions do not matter at all without a bias: a permuted table gives the same result
    w2 = W.Workload(**{**w.__dict__})
    w2.chunks = w.chunks.copy()
    w2.chunks["pos_offset"] = w.chunks["pos_offset"][::-1].copy()
    b, _ = run(w2, pairing="alibi", inv_freq=zero)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    # with the bias only relative positions matter (causal, every position moved by the same amount)
    w.causal = True
    c0, _ = run(w, pairing="alibi")
    w3 = W.Workload(**{**w.__dict__})
    w3.chunks = w.chunks.copy()
    w3.chunks["pos_offset"] += 777
    w3.q_pos0 = w.q_pos0 + 777
    c1, _ = run(w3, pairing="alibi")
    np.testing.assert_allclose(c0, c1, rtol=0, atol=1e-10)
    assert np.allclose(O.alibi_slopes(8), [2.0 ** -(i + 1) for i in range(8)])
