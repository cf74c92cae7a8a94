#!/usr/bin/env python3
"""Benchmark of the LazyAttention hot path on one MI355X.

Headline (the JSON line's ``value``): lazy prefill of the Llama-3-8B-shaped RAG batch (B=8, 32 query / 8 KV heads,
head_dim 128, RoPE base 5e5, shared 128-token prefix + 10 retrieved 512-token chunks from a 64-chunk pool at
per-request positions + a 64-token causal question), in useful TFLOP/s with inputs resident in HBM.  One step is
one ``lazy_attn_prefill`` call (prefill kernel + split-KV combine).  The same line carries the split-KV decode
(B=64, ~16.5K position-free keys per request, chunks shared across requests at different offsets) in logical HBM
GB/s, the materialise-then-attend baseline for both, a no-rotation diagnostic, the roofline of the dominant
kernel and the fp64 oracle timed on the host cores.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "RAG prefill ms & TFLOP/s (MFMA %), decode HBM GB/s, vs materialize baseline"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0     # MI355X HBM3E
KERNEL_SOURCE = os.path.join(ROOT, "paper_2606_04302_amd", "csrc", "lazy_attn_kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_hash() -> str:
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def recorded_traffic(kernel: str):
    """HBM bytes per launch measured with rocprofv3 --pmc (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known
    size); null when the kernel source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    entry = rec.get(kernel)
    if not entry or entry.get("kernel_source_sha256_16") != kernel_hash():
        return None
    return entry.get("bytes_per_launch")


LEG_WARMUP_MS = 30.0
_last_leg_warmup_calls = 0


def timed(fn, steps: int, warmup: int):
    """Average ms per call, measured with HIP events on the current stream around ``steps`` back-to-back calls.
    Before them: at least LEG_WARMUP_MS of GPU time of the same call (so that every leg starts from its own working
    set in the caches and from settled clocks, whatever the leg before it ran), then the --warmup calls."""
    import torch

    global _last_leg_warmup_calls
    _, _last_leg_warmup_calls = clock_warmup(fn, LEG_WARMUP_MS)
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def clock_warmup(fn, min_ms: float = 150.0):
    """Back-to-back calls of ``fn`` until at least ``min_ms`` of GPU time has elapsed (HIP events), so that the
    clocks have left their idle state before anything is timed; returns the GPU ms spent and the number of calls.
    Independent of the --warmup step count, which is still honoured as given before every timed leg."""
    import torch

    spent, batch, calls = 0.0, 8, 0
    while spent < min_ms:
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(batch):
            fn()
        b.record()
        torch.cuda.synchronize()
        spent += a.elapsed_time(b)
        calls += batch
        batch = min(batch * 2, 4096)
    return spent, calls


def paired_overhead(fn, base, loops: int = 15, inner: int = 20):
    """Relative cost of ``fn`` over ``base``: ``loops`` pairs of timed loops of ``inner`` back-to-back calls each,
    the two alternating so that clock drift affects both alike; the median, smallest and largest of the per-pair
    ratios minus one.  Each pair starts with one untimed call, so that the GPU is already busy when the first event
    is recorded (otherwise the first loop would also time the launch of its first call), and the pairs alternate
    which of the two runs first."""
    import torch

    ratios = []
    for i in range(loops):
        first, second = (fn, base) if i % 2 == 0 else (base, fn)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        first()
        ev[0].record()
        for _ in range(inner):
            first()
        ev[1].record()
        ev[2].record()
        for _ in range(inner):
            second()
        ev[3].record()
        torch.cuda.synchronize()
        t_first, t_second = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
        t_fn, t_base = (t_first, t_second) if i % 2 == 0 else (t_second, t_first)
        ratios.append(t_fn / t_base - 1.0)
    return {"median": round(float(np.median(ratios)), 4), "min": round(float(min(ratios)), 4),
            "max": round(float(max(ratios)), 4), "pairs": loops, "calls_per_loop": inner}


def timed_graph(fn, reps: int, inner: int = 20):
    """Average ms per call of a short GPU call whose host-side launch cost would otherwise dominate: ``inner``
    calls captured in one HIP graph, the graph replayed ``reps`` times between HIP events."""
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(3):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(inner):
            fn()
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        g.replay()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / (reps * inner)


def timed_median(fn, loops: int = 20, inner: int = 10):
    """Median over ``loops`` timed loops of ``inner`` back-to-back calls (ms per call), after the caller's warm-up."""
    import torch

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(loops)]
    for a, b in ev:
        a.record()
        for _ in range(inner):
            fn()
        b.record()
    torch.cuda.synchronize()
    return float(np.median([a.elapsed_time(b) / inner for a, b in ev]))


def timed_cold(fn, reps: int, scrub_mib: int = 512):
    """Average ms per call with cold caches: before every call a 512 MiB buffer (twice the 256 MB MALL, far more than
    the L2s) is overwritten, then the call alone is bracketed by HIP events.  The scrub is queued ahead of the call,
    so the events time the call and not its launch."""
    import torch

    scrub = torch.empty(scrub_mib << 20, dtype=torch.uint8, device="cuda")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    fn()
    for i in range(reps):
        scrub.fill_(i & 0x7F)
        ev[i][0].record()
        fn()
        ev[i][1].record()
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in ev) / reps
    del scrub
    return ms


def cpu_baseline(w, flops_per_pass: float, budget_s: float = 12.0):
    """The fp64 oracle on the host cores, whole passes over the same batch until ``budget_s`` has elapsed."""
    from oracle import lazy_oracle as O

    try:
        import threadpoolctl

        threads = max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:  # pragma: no cover - informational only
        threads = os.cpu_count() or 1
    passes, t0 = 0, time.perf_counter()
    while True:
        O.lazy_attention(w.q, w.q_start, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, w.num_q_heads,
                         w.num_kv_heads, w.head_dim, w.rope_base, w.causal)
        passes += 1
        el = time.perf_counter() - t0
        if el >= budget_s or passes >= 50:
            break
    per = el / passes
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover - informational only
        pass
    return {
        "value": flops_per_pass / per / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"full rag_prefill batch (8 requests), {passes} pass(es), {per:.2f} s per pass, numpy fp64 with "
                  f"{int(threads)} BLAS threads on {model} ({os.cpu_count()} logical CPUs visible)",
        "s_per_pass": per,
    }


def other_configs(dev, steps: int, warmup: int, log):
    """Per-configuration figures beyond the headline, lazy vs materialise-then-attend:
    - icl: many-shot ICL batch (B=4, 32/8 heads, D=128, a shared pool of 128 x 256-token exemplars permuted per
      request, 256-token causal query at 32,768), its prefill, then 128 decode steps (the query's own chunk grows
      by one token per step, one query per request at the newest position).  The baseline materialises the
      rotated keys once (at the final lengths, so the appended keys are included) and runs the plain kernels.
      Timed twice: with the tables in position order, and (``storage_order``) with every request's table in
      storage order, the baseline taking the same tables.
    - varlen_rag: 16 requests, 28/4 heads, D=128, base 1e6, 8-24 chunks of U[128, 2048] tokens per request drawn
      Zipf(2.1) without replacement from a 200-chunk pool, queries of U[32, 256] tokens."""
    import torch

    from paper_2606_04302_amd import accounting as A
    from paper_2606_04302_amd import ops
    from paper_2606_04302_amd import workloads as W

    res = {}

    def materialized(w, dw, chunks_np):
        total_kv = int(chunks_np["len"].astype(np.int64).sum())
        ch = ops.chunks_tensor(chunks_np, dev)
        k_out = torch.empty(dw.cfg.num_kv_heads * total_kv * dw.cfg.head_dim, dtype=torch.bfloat16, device=dev)
        ch_out = torch.empty_like(ch)
        mx = int(chunks_np["len"].max())
        fn = lambda: ops.materialize_k(dw.cfg, dw.pool, ch, mx, total_kv, k_out=k_out, chunks_out=ch_out)
        return fn, k_out, ch_out

    # ---- icl prefill + 128 decode steps ----
    log("icl workload: generating")
    w = W.icl_prefill(seed=3)
    dw = ops.upload(w, dev)
    cfg = dw.cfg
    flops = A.useful_flops(w)
    ws = torch.empty(max(16, ops.prefill_workspace_size(cfg, w.batch, w.total_q, w.max_q_len, w.max_kv_len)),
                     dtype=torch.uint8, device=dev)
    out = torch.empty_like(dw.q)
    pre = lambda: ops.prefill(cfg, dw.q, dw.q_start, dw.q_pos0, dw.pool, dw.pool, dw.chunks, dw.chunk_start,
                              w.max_q_len, w.max_kv_len, out=out, workspace=ws)
    log("icl: timing prefill")
    pre_ms = timed(pre, steps, warmup)

    n_steps = int(w.meta["decode_steps"])
    own = [int(w.chunk_start[r + 1]) - 1 for r in range(w.batch)]
    tables, dec_flops, dec_bytes, max_kv = [], 0, 0, 0
    hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
    for s in range(n_steps):
        ch = w.chunks.copy()
        qpos = np.empty(w.batch, dtype=np.int32)
        for r, i in enumerate(own):
            ch[i]["len"] = int(w.q_lens[r]) + s + 1
            qpos[r] = int(ch[i]["pos_offset"]) + int(ch[i]["len"]) - 1
        lens = [int(ch[int(w.chunk_start[r]):int(w.chunk_start[r + 1])]["len"].astype(np.int64).sum())
                for r in range(w.batch)]
        max_kv = max(max_kv, max(lens))
        dec_flops += 4 * d * hq * sum(lens)
        dec_bytes += sum(lens) * hkv * d * 2 * 2 + 2 * w.batch * hq * d * 2
        tables.append((ch, ops.chunks_tensor(ch, dev), torch.from_numpy(qpos).to(dev)))
    rng = np.random.default_rng(33)
    qd = ops.bf16_tensor(W.bf16_round(rng.standard_normal((w.batch, hq, d), dtype=np.float32)), dev)
    outd = torch.empty_like(qd)
    wsd = torch.empty(max(16, ops.decode_workspace_size(cfg, w.batch, max_kv)), dtype=torch.uint8, device=dev)

    def decode_all(kp=None, plain_tables=None):
        for s, (_, ch, qp) in enumerate(tables):
            if plain_tables is None:
                ops.decode(cfg, qd, qp, dw.pool, dw.pool, ch, dw.chunk_start, max_kv, out=outd, workspace=wsd)
            else:
                ops.decode(cfg, qd, qp, kp, dw.pool, plain_tables[s], dw.chunk_start, max_kv, out=outd,
                           workspace=wsd, plain=True)

    reps = max(3, steps // 40)
    log("icl: timing 128 decode steps")
    dec_ms = timed(decode_all, reps, 2)

    # The same prefill and decode steps over a local-position store (keys kept encoded at their index within the
    # chunk, the paper's own convention): the prefill rotates each K tile once by the record offset and the decode
    # rotates the query once per record instead of every key.  Its materialising copy is the same one rotation per
    # key as the NoPE store's, so it shares the baseline below.
    cfg_local = ops.config_of(w, key_positions=ops.KEYS_LOCAL)
    log("icl: timing the local-position store")
    local_pre_ms = timed(lambda: ops.prefill(cfg_local, dw.q, dw.q_start, dw.q_pos0, dw.pool, dw.pool, dw.chunks,
                                             dw.chunk_start, w.max_q_len, w.max_kv_len, out=out, workspace=ws),
                         steps, warmup)

    def decode_all_local():
        for _, ch, qp in tables:
            ops.decode(cfg_local, qd, qp, dw.pool, dw.pool, ch, dw.chunk_start, max_kv, out=outd, workspace=wsd)

    local_dec_ms = timed(decode_all_local, reps, 2)

    # Chunk-major shared decode steps: the exemplar pool is read once per step for the four requests.
    plans = [ops.upload_plan(ops.shared_decode_plan(cfg, ch, w.chunk_start), dev) for ch, _, _ in tables]
    wsh = torch.empty(max(16, max(ops.decode_shared_workspace_size(cfg, w.batch, pl.max_slots) for pl in plans)),
                      dtype=torch.uint8, device=dev)

    def decode_shared_all():
        for s, (_, _, qp) in enumerate(tables):
            ops.decode_shared(cfg, qd, qp, dw.pool, dw.pool, plans[s], out=outd, workspace=wsh)

    log("icl: timing 128 shared decode steps")
    shared_ms = timed(decode_shared_all, reps, 2)

    # Baseline: keys materialised once at their final lengths; per-step tables point into the copy.
    final = tables[-1][0]
    mat_fn, k_mat, ch_mat = materialized(w, dw, final)
    mat_fn()
    torch.cuda.synchronize()
    mat_np = ops.chunks_from_tensor(ch_mat)
    pre_tab = mat_np.copy()
    for r, i in enumerate(own):
        pre_tab[i]["len"] = int(w.chunks[i]["len"])
    pre_tab_t = ops.chunks_tensor(pre_tab, dev)
    plain_tabs = []
    for ch, _, _ in tables:
        t = mat_np.copy()
        for i in own:
            t[i]["len"] = int(ch[i]["len"])
        plain_tabs.append(ops.chunks_tensor(t, dev))
    log("icl: timing the baseline")
    mat_ms = timed(mat_fn, max(5, steps // 5), 2)
    plain_pre_ms = timed(lambda: ops.prefill(cfg, dw.q, dw.q_start, dw.q_pos0, k_mat, dw.pool, pre_tab_t,
                                             dw.chunk_start, w.max_q_len, w.max_kv_len, out=out, workspace=ws,
                                             plain=True), steps, warmup)
    plain_dec_ms = timed(lambda: decode_all(k_mat, plain_tabs), reps, 2)
    lazy_total = pre_ms + dec_ms
    base_total = mat_ms + plain_pre_ms + plain_dec_ms

    # The same per-request prefill and decode steps with every request's table in storage order
    # (lazy_chunk_table_storage_order; positions, not the table order, decide the attention).  The decode's
    # workgroups for one (split, KV head) of the four requests run together on one XCD, so with the exemplars listed
    # in the same order the requests read each one through one L2.  The baseline takes the same tables (its copy is
    # written in that order and V is still read from the pool).
    log("icl: storage-ordered tables")
    so_tables = []
    for ch, _, qp in tables:
        t = ops.storage_order(ch, w.chunk_start)
        so_tables.append((t, ops.chunks_tensor(t, dev), qp))
    so_own = []
    for r, i in enumerate(own):
        a, b = int(w.chunk_start[r]), int(w.chunk_start[r + 1])
        so_own.append(a + int(np.flatnonzero(so_tables[0][0]["k_offset"][a:b] == w.chunks[i]["k_offset"])[0]))
    so_pre_np = so_tables[0][0].copy()
    for r, i in enumerate(so_own):
        so_pre_np[i]["len"] = int(w.q_lens[r])
    so_pre_t = ops.chunks_tensor(so_pre_np, dev)

    def so_prefill(c):
        return lambda: ops.prefill(c, dw.q, dw.q_start, dw.q_pos0, dw.pool, dw.pool, so_pre_t, dw.chunk_start,
                                   w.max_q_len, w.max_kv_len, out=out, workspace=ws)

    def so_decode(c, kp=None, plain_tables=None):
        def run():
            for s, (_, ch, qp) in enumerate(so_tables):
                if plain_tables is None:
                    ops.decode(c, qd, qp, dw.pool, dw.pool, ch, dw.chunk_start, max_kv, out=outd, workspace=wsd)
                else:
                    ops.decode(c, qd, qp, kp, dw.pool, plain_tables[s], dw.chunk_start, max_kv, out=outd,
                               workspace=wsd, plain=True)
        return run

    so_pre_ms = timed(so_prefill(cfg), steps, warmup)
    so_dec_ms = timed(so_decode(cfg), reps, 2)
    so_local_pre_ms = timed(so_prefill(cfg_local), steps, warmup)
    so_local_dec_ms = timed(so_decode(cfg_local), reps, 2)
    so_mat_fn, so_k_mat, so_ch_mat = materialized(w, dw, so_tables[-1][0])
    so_mat_fn()
    torch.cuda.synchronize()
    so_mat_np = ops.chunks_from_tensor(so_ch_mat)
    so_pre_tab = so_mat_np.copy()
    for r, i in enumerate(so_own):
        so_pre_tab[i]["len"] = int(w.q_lens[r])
    so_pre_tab_t = ops.chunks_tensor(so_pre_tab, dev)
    so_plain_tabs = []
    for ch, _, _ in so_tables:
        t = so_mat_np.copy()
        for i in so_own:
            t[i]["len"] = int(ch[i]["len"])
        so_plain_tabs.append(ops.chunks_tensor(t, dev))
    so_mat_ms = timed(so_mat_fn, max(5, steps // 5), 2)
    so_plain_pre_ms = timed(lambda: ops.prefill(cfg, dw.q, dw.q_start, dw.q_pos0, so_k_mat, dw.pool, so_pre_tab_t,
                                                dw.chunk_start, w.max_q_len, w.max_kv_len, out=out, workspace=ws,
                                                plain=True), steps, warmup)
    so_plain_dec_ms = timed(so_decode(cfg, so_k_mat, so_plain_tabs), reps, 2)
    so_lazy_total = so_pre_ms + so_dec_ms
    so_base_total = so_mat_ms + so_plain_pre_ms + so_plain_dec_ms
    storage_order = {
        "prefill_ms": round(so_pre_ms, 5),
        "decode_128_steps_ms": round(so_dec_ms, 4),
        "decode_logical_gbps": round(dec_bytes / (so_dec_ms * 1e-3) / 1e9, 1),
        "local_keys_prefill_ms": round(so_local_pre_ms, 5),
        "local_keys_decode_128_steps_ms": round(so_local_dec_ms, 4),
        "materialize_ms": round(so_mat_ms, 5),
        "plain_prefill_ms": round(so_plain_pre_ms, 5),
        "plain_decode_128_steps_ms": round(so_plain_dec_ms, 4),
        "lazy_prefill_plus_decode_ms": round(so_lazy_total, 4),
        "materialize_then_attend_ms": round(so_base_total, 4),
        "speedup_vs_materialize": round(so_base_total / so_lazy_total, 3),
        "local_keys_speedup_vs_materialize": round(so_base_total / (so_local_pre_ms + so_local_dec_ms), 3),
        "speedup_vs_position_ordered_materialize": round(base_total / so_lazy_total, 3),
    }
    del so_k_mat
    res["icl"] = {
        "workload": "icl: batch 4, 32/8 heads, head_dim 128, base 5e5, 128 x 256-token exemplars (shared pool, "
                    "permuted per request), 256-token query at 32,768, then 128 decode steps; tables in position "
                    "order, and under storage_order the same runs with each request's table in storage order "
                    "(lazy and baseline alike)",
        "prefill_ms": round(pre_ms, 5),
        "prefill_tflops": round(flops / (pre_ms * 1e-3) / 1e12, 3),
        "prefill_mfma_frac": round(flops / (pre_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 5),
        "decode_128_steps_ms": round(dec_ms, 4),
        "decode_ms_per_step": round(dec_ms / n_steps, 5),
        "decode_logical_hbm_gbps": round(dec_bytes / (dec_ms * 1e-3) / 1e9, 1),
        "decode_logical_hbm_frac": round(dec_bytes / (dec_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "decode_logical_gb": round(dec_bytes / 1e9, 3),
        "shared_decode_128_steps_ms": round(shared_ms, 4),
        "shared_decode_logical_gbps": round(dec_bytes / (shared_ms * 1e-3) / 1e9, 1),
        "unique_kv_mb": round(A.unique_kv_bytes(w) / 1e6, 1),
        "lazy_prefill_plus_decode_ms": round(lazy_total, 4),
        "lazy_prefill_plus_shared_decode_ms": round(pre_ms + shared_ms, 4),
        "materialize_ms": round(mat_ms, 5),
        "plain_prefill_ms": round(plain_pre_ms, 5),
        "plain_decode_128_steps_ms": round(plain_dec_ms, 4),
        "materialize_then_attend_ms": round(base_total, 4),
        "speedup_vs_materialize": round(base_total / lazy_total, 3),
        "speedup_vs_materialize_shared_decode": round(base_total / (pre_ms + shared_ms), 3),
        "local_keys_prefill_ms": round(local_pre_ms, 5),
        "local_keys_decode_128_steps_ms": round(local_dec_ms, 4),
        "local_keys_speedup_vs_materialize": round(base_total / (local_pre_ms + local_dec_ms), 3),
        "storage_order": storage_order,
    }
    del k_mat, dw, ws, wsd

    # ---- overhead-ablation shape: one request, 5 x 4096-token chunks + a 64-token query ----
    log("e3_overhead workload: generating")
    w = W.rag_prefill(seed=5, batch=1, prefix_len=0, n_chunks=5, chunk_len=4096, pool_chunks=5, q_len=64)
    dw = ops.upload(w, dev)
    cfg = dw.cfg
    flops = A.useful_flops(w)
    ws = torch.empty(max(16, ops.prefill_workspace_size(cfg, w.batch, w.total_q, w.max_q_len, w.max_kv_len)),
                     dtype=torch.uint8, device=dev)
    out = torch.empty_like(dw.q)

    def e3(c, plain=False):
        return lambda: ops.prefill(c, dw.q, dw.q_start, dw.q_pos0, dw.pool, dw.pool, dw.chunks, dw.chunk_start,
                                   w.max_q_len, w.max_kv_len, out=out, workspace=ws, plain=plain)

    log("e3_overhead: timing")
    ms = timed(e3(cfg), steps, warmup)
    norot = timed(e3(cfg, True), steps, warmup)
    local = timed(e3(ops.config_of(w, key_positions=ops.KEYS_LOCAL)), steps, warmup)
    e3_spread = paired_overhead(e3(cfg), e3(cfg, True))
    e3_local_spread = paired_overhead(e3(ops.config_of(w, key_positions=ops.KEYS_LOCAL)), e3(cfg, True))
    mat_fn, k_mat, ch_mat = materialized(w, dw, w.chunks)
    mat_ms = timed(mat_fn, max(5, steps // 5), 2)
    res["e3_overhead"] = {
        "workload": "one request, 32/8 heads, head_dim 128, base 5e5, 5 x 4096-token chunks + 64-token causal query "
                    "(the shape of the paper's rotation-overhead ablation)",
        "prefill_ms": round(ms, 5),
        "tflops": round(flops / (ms * 1e-3) / 1e12, 3),
        "no_rotation_ms": round(norot, 5),
        "rotation_overhead": round(ms / norot - 1.0, 4),
        "rotation_overhead_spread": e3_spread,
        "local_keys_ms": round(local, 5),
        "local_keys_overhead": round(local / norot - 1.0, 4),
        "local_keys_overhead_spread": e3_local_spread,
        "materialize_ms": round(mat_ms, 5),
        "speedup_vs_materialize": round((mat_ms + norot) / ms, 3),
    }
    del dw, ws, k_mat

    # ---- icl decode with private pools: every request owns its 128 exemplars (no sharing, 537 MB) ----
    log("icl_private workload: generating")
    w = W.icl_prefill(seed=3, private=True)
    dw = ops.upload(w, dev)
    cfg = dw.cfg
    own = [int(w.chunk_start[r + 1]) - 1 for r in range(w.batch)]
    tables, pbytes, max_kv = [], 0, 0
    hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
    for s in range(int(w.meta["decode_steps"])):
        ch = w.chunks.copy()
        qpos = np.empty(w.batch, dtype=np.int32)
        for r, i in enumerate(own):
            ch[i]["len"] = int(w.q_lens[r]) + s + 1
            qpos[r] = int(ch[i]["pos_offset"]) + int(ch[i]["len"]) - 1
        lens = [int(ch[int(w.chunk_start[r]):int(w.chunk_start[r + 1])]["len"].astype(np.int64).sum())
                for r in range(w.batch)]
        max_kv = max(max_kv, max(lens))
        pbytes += sum(lens) * hkv * d * 2 * 2 + 2 * w.batch * hq * d * 2
        tables.append((ops.chunks_tensor(ch, dev), torch.from_numpy(qpos).to(dev)))
    rng = np.random.default_rng(33)
    qd = ops.bf16_tensor(W.bf16_round(rng.standard_normal((w.batch, hq, d), dtype=np.float32)), dev)
    outd = torch.empty_like(qd)
    wsd = torch.empty(max(16, ops.decode_workspace_size(cfg, w.batch, max_kv)), dtype=torch.uint8, device=dev)

    # Every request's context is private and larger than the last-level cache, and each decode step reads it
    # once: the calls pass the streaming cache hint (non-temporal K / V loads), as a caller with such contexts would.
    # The default hint is timed beside it.
    cfg_s = ops.config_of(w, cache_hint=ops.CACHE_STREAM)
    cfg_local = ops.config_of(w, key_positions=ops.KEYS_LOCAL)
    cfg_local_s = ops.config_of(w, key_positions=ops.KEYS_LOCAL, cache_hint=ops.CACHE_STREAM)

    def decode_private(c):
        def run():
            for ch, qp in tables:
                ops.decode(c, qd, qp, dw.pool, dw.pool, ch, dw.chunk_start, max_kv, out=outd, workspace=wsd)
        return run

    log("icl_private: timing 128 decode steps")
    pms = timed(decode_private(cfg_s), max(3, steps // 40), 2)
    pms_default = timed(decode_private(cfg), max(3, steps // 40), 2)
    # the same steps over a local-position store (the query rotated once per record)
    pms_local = timed(decode_private(cfg_local_s), max(3, steps // 40), 2)
    pms_local_default = timed(decode_private(cfg_local), max(3, steps // 40), 2)
    frac = lambda t: round(pbytes / (t * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)
    res["icl_private"] = {
        "workload": "icl with private pools: batch 4, 32/8 heads, head_dim 128, each request its own 128 x "
                    "256-token exemplars, 256-token query at 32,768, then 128 decode steps; cache hint stream "
                    "(private contexts larger than the last-level cache), the default hint timed beside it",
        "decode_128_steps_ms": round(pms, 4),
        "decode_ms_per_step": round(pms / len(tables), 5),
        "decode_logical_hbm_gbps": round(pbytes / (pms * 1e-3) / 1e9, 1),
        "decode_logical_hbm_frac": frac(pms),
        "default_hint_decode_128_steps_ms": round(pms_default, 4),
        "default_hint_decode_logical_hbm_frac": frac(pms_default),
        "local_keys_decode_128_steps_ms": round(pms_local, 4),
        "local_keys_decode_logical_hbm_frac": frac(pms_local),
        "local_keys_default_hint_decode_logical_hbm_frac": frac(pms_local_default),
        "unique_kv_mb": round(A.unique_kv_bytes(w) / 1e6, 1),
    }
    del dw, wsd, tables

    # ---- varlen_rag prefill ----
    log("varlen_rag workload: generating")
    w = W.varlen_rag(seed=4)
    dw = ops.upload(w, dev)
    cfg = dw.cfg
    flops = A.useful_flops(w)
    ws = torch.empty(max(16, ops.prefill_workspace_size(cfg, w.batch, w.total_q, w.max_q_len, w.max_kv_len)),
                     dtype=torch.uint8, device=dev)
    out = torch.empty_like(dw.q)
    log("varlen_rag: timing")
    ms = timed(lambda: ops.prefill(cfg, dw.q, dw.q_start, dw.q_pos0, dw.pool, dw.pool, dw.chunks, dw.chunk_start,
                                   w.max_q_len, w.max_kv_len, out=out, workspace=ws), steps, warmup)
    mat_fn, k_mat, ch_mat = materialized(w, dw, w.chunks)
    mat_ms = timed(mat_fn, max(5, steps // 5), 2)
    plain_ms = timed(lambda: ops.prefill(cfg, dw.q, dw.q_start, dw.q_pos0, k_mat, dw.pool, ch_mat, dw.chunk_start,
                                         w.max_q_len, w.max_kv_len, out=out, workspace=ws, plain=True), steps, warmup)
    res["varlen_rag"] = {
        "workload": "varlen_rag: batch 16, 28/4 heads, head_dim 128, base 1e6, 8-24 chunks of U[128, 2048] tokens "
                    "per request, Zipf(2.1) reuse over a 200-chunk pool, U[32, 256]-token queries",
        "prefill_ms": round(ms, 5),
        "useful_gflop": round(flops / 1e9, 3),
        "tflops": round(flops / (ms * 1e-3) / 1e12, 3),
        "mfma_frac": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 5),
        "logical_kv_mb": round(A.logical_kv_bytes(w) / 1e6, 1),
        "unique_kv_mb": round(A.unique_kv_bytes(w) / 1e6, 1),
        "materialize_ms": round(mat_ms, 5),
        "plain_prefill_ms": round(plain_ms, 5),
        "materialize_then_attend_ms": round(mat_ms + plain_ms, 5),
        "speedup_vs_materialize": round((mat_ms + plain_ms) / ms, 3),
    }
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=500,
                    help="untimed steps before every timed leg (a time-based clock warm-up of >= 150 ms of GPU "
                         "work runs once before the first leg whatever this is)")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode and baseline legs")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-other", action="store_true", help="skip the ICL and variable-length RAG configurations")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (reference kernel for HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: only one GPU is measured; --gpus {args.gpus} is not supported (the hot path would shard "
              "by request and KV head with no communication)", file=sys.stderr)
        return 2
    rank = int(os.environ.get("RANK", "0"))

    import torch

    from paper_2606_04302_amd import accounting as A
    from paper_2606_04302_amd import ops
    from paper_2606_04302_amd import workloads as W

    ops.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    # ---------------- prefill (headline) ----------------
    log("prefill workload: generating")
    wp = W.rag_prefill(seed=1)
    dp = ops.upload(wp, dev)
    cfg = dp.cfg
    flops = A.useful_flops(wp)
    alg_bytes = A.algorithmic_bytes(wp)
    ws_bytes = ops.prefill_workspace_size(cfg, wp.batch, wp.total_q, wp.max_q_len, wp.max_kv_len)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
    out = torch.empty_like(dp.q)
    lse = torch.empty((wp.total_q, wp.num_q_heads), dtype=torch.float32, device=dev)

    def prefill():
        ops.prefill(cfg, dp.q, dp.q_start, dp.q_pos0, dp.pool, dp.pool, dp.chunks, dp.chunk_start, wp.max_q_len,
                    wp.max_kv_len, out=out, lse=lse, workspace=ws)

    torch.cuda.synchronize()
    log("prefill: clock warm-up")
    warm_ms, warm_calls = clock_warmup(prefill)
    log(f"prefill: timing {args.steps} steps after {args.warmup} warmup")
    ms = timed(prefill, args.steps, args.warmup)
    head_leg_calls = _last_leg_warmup_calls

    # The combine kernel alone on the same partials, to isolate the prefill kernel's own duration.
    rows = wp.total_q * wp.num_q_heads
    part_o, part_lse = ops.split_views(ws, rows, wp.head_dim)
    splits = part_o.shape[0] if part_o is not None else 1
    combine_ms = 0.0
    if splits > 1:
        out2 = torch.empty((rows, wp.head_dim), dtype=torch.bfloat16, device=dev)
        lse2 = torch.empty(rows, dtype=torch.float32, device=dev)
        # Graph-replayed: a lone combine launch is shorter than its host-side call.
        combine_ms = timed_graph(lambda: ops.combine(part_o, part_lse, out=out2, lse=lse2), max(20, args.steps // 4))
    kernel_ms = ms - combine_ms

    median_ms = timed_median(prefill)

    # Cold caches: every launch after a 512 MiB scrub, so the store comes from HBM and not from the MALL / L2s.
    cold_ms = timed_cold(prefill, max(10, args.steps // 10))

    # No-rotation diagnostic: the same kernel with K rotation compiled out, over the unrotated store.
    norot = lambda: ops.prefill(cfg, dp.q, dp.q_start, dp.q_pos0, dp.pool, dp.pool, dp.chunks, dp.chunk_start,
                                wp.max_q_len, wp.max_kv_len, out=out, lse=lse, workspace=ws, plain=True)
    norot_ms = timed(norot, args.steps, args.warmup)
    rot_spread = paired_overhead(prefill, norot)

    # The same batch over a local-position key store (keys kept encoded at their local index; one rotation per
    # record offset).  The pool's values are read as such keys: same shapes and traffic.
    cfg_local = ops.config_of(wp, key_positions=ops.KEYS_LOCAL)
    local_ms = timed(lambda: ops.prefill(cfg_local, dp.q, dp.q_start, dp.q_pos0, dp.pool, dp.pool, dp.chunks,
                                         dp.chunk_start, wp.max_q_len, wp.max_kv_len, out=out, lse=lse, workspace=ws),
                     args.steps, args.warmup)

    # ALiBi instead of RoPE (score-space positions: no rotation, one bias per score).
    cfg_alibi = ops.config_of(wp, rope_style=ops.ALIBI)
    alibi_ms = timed(lambda: ops.prefill(cfg_alibi, dp.q, dp.q_start, dp.q_pos0, dp.pool, dp.pool, dp.chunks,
                                         dp.chunk_start, wp.max_q_len, wp.max_kv_len, out=out, lse=lse, workspace=ws),
                     args.steps, args.warmup)

    # The same batch over a paged store (64-token blocks scattered over the pool, one record per block).
    wpp = W.paginate(wp, 64, seed=7)
    dpp = ops.upload(wpp, dev)
    paged_ms = timed(lambda: ops.prefill(cfg, dpp.q, dpp.q_start, dpp.q_pos0, dpp.pool, dpp.pool, dpp.chunks,
                                         dpp.chunk_start, wpp.max_q_len, wpp.max_kv_len, out=out, lse=lse,
                                         workspace=ws), args.steps, args.warmup)
    del dpp

    # Materialise-then-attend baseline: rotate-and-copy K, then plain attention over the copy.
    total_kv = int(wp.chunks["len"].astype(np.int64).sum())
    k_mat = torch.empty(cfg.num_kv_heads * total_kv * cfg.head_dim, dtype=torch.bfloat16, device=dev)
    ch_mat = torch.empty_like(dp.chunks)
    max_chunk = int(wp.chunks["len"].max())
    mat_ms = timed(lambda: ops.materialize_k(cfg, dp.pool, dp.chunks, max_chunk, total_kv, k_out=k_mat,
                                             chunks_out=ch_mat), args.steps, args.warmup)
    plain_ms = timed(lambda: ops.prefill(cfg, dp.q, dp.q_start, dp.q_pos0, k_mat, dp.pool, ch_mat, dp.chunk_start,
                                         wp.max_q_len, wp.max_kv_len, out=out, lse=lse, workspace=ws, plain=True),
                     args.steps, args.warmup)

    tflops = flops / (ms * 1e-3) / 1e12
    kernel_tflops = flops / (kernel_ms * 1e-3) / 1e12
    result = {
        "metric": METRIC,
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "clock_warmup_ms": round(warm_ms, 1),
        "clock_warmup_calls": warm_calls,
        "leg_warmup_ms": LEG_WARMUP_MS,
        "headline_leg_warmup_calls": head_leg_calls,
        "config": {
            "workload": "rag_prefill: Llama-3-8B-shaped RAG prefill, batch 8, 32 query / 8 KV heads, head_dim 128, "
                        "RoPE base 5e5, 128-token shared prefix + 10 x 512-token chunks drawn from a 64-chunk pool "
                        "(random order, contiguous positions) + 64-token causal question",
            "batch": wp.batch,
            "q_tokens": wp.total_q,
            "kv_tokens_per_request": int(wp.max_kv_len),
            "splits": int(splits),
        },
        "roofline": {
            "bound": "mfma",
            "achieved": round(kernel_tflops, 3),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(kernel_tflops / PEAK_BF16_TFLOPS, 5),
            "traffic": recorded_traffic("prefill_kernel_rag_prefill"),
            "kernel": "prefill_kernel<128, rotate K>",
            "kernel_ms": round(kernel_ms, 5),
            "useful_gflop_per_launch": round(flops / 1e9, 4),
            "algorithmic_mb_per_launch": round(alg_bytes / 1e6, 3),
        },
        "prefill": {
            "ms": round(ms, 5),
            "tflops": round(tflops, 3),
            "mfma_frac": round(tflops / PEAK_BF16_TFLOPS, 5),
            "kernel_ms": round(kernel_ms, 5),
            "combine_ms": round(combine_ms, 5),
            "logical_hbm_gbps": round(alg_bytes / (ms * 1e-3) / 1e9, 1),
            "median_of_20_loops_ms": round(median_ms, 5),
            "cold_cache_ms": round(cold_ms, 5),
            "cold_cache_tflops": round(flops / (cold_ms * 1e-3) / 1e12, 3),
            "no_rotation_ms": round(norot_ms, 5),
            "rotation_overhead": round(ms / norot_ms - 1.0, 4),
            "rotation_overhead_spread": rot_spread,
            "local_keys_ms": round(local_ms, 5),
            "local_keys_tflops": round(flops / (local_ms * 1e-3) / 1e12, 3),
            "paged64_ms": round(paged_ms, 5),
            "alibi_ms": round(alibi_ms, 5),
            "materialize_ms": round(mat_ms, 5),
            "plain_attention_ms": round(plain_ms, 5),
            "materialize_then_attend_ms": round(mat_ms + plain_ms, 5),
            "speedup_vs_materialize": round((mat_ms + plain_ms) / ms, 3),
            "unique_kv_mb": round(A.unique_kv_bytes(wp) / 1e6, 2),
            "logical_kv_mb": round(A.logical_kv_bytes(wp) / 1e6, 2),
        },
    }
    del k_mat

    # ---------------- decode ----------------
    if not args.no_decode:
        log("decode workload: generating")
        wd = W.rag_decode(seed=2)
        dd = ops.upload(wd, dev)
        cfgd = dd.cfg
        dbytes = A.algorithmic_bytes(wd)
        wsd_bytes = ops.decode_workspace_size(cfgd, wd.batch, wd.max_kv_len)
        wsd = torch.empty(max(wsd_bytes, 16), dtype=torch.uint8, device=dev)
        outd = torch.empty_like(dd.q)
        lsed = torch.empty((wd.batch, wd.num_q_heads), dtype=torch.float32, device=dev)
        log("decode: timing")
        dms = timed(lambda: ops.decode(cfgd, dd.q, dd.q_pos0, dd.pool, dd.pool, dd.chunks, dd.chunk_start,
                                       wd.max_kv_len, out=outd, lse=lsed, workspace=wsd), args.steps, args.warmup)
        dcold = timed_cold(lambda: ops.decode(cfgd, dd.q, dd.q_pos0, dd.pool, dd.pool, dd.chunks, dd.chunk_start,
                                              wd.max_kv_len, out=outd, lse=lsed, workspace=wsd),
                           max(10, args.steps // 20))
        dec_lazy = lambda: ops.decode(cfgd, dd.q, dd.q_pos0, dd.pool, dd.pool, dd.chunks, dd.chunk_start,
                                      wd.max_kv_len, out=outd, lse=lsed, workspace=wsd)
        dec_norot = lambda: ops.decode(cfgd, dd.q, dd.q_pos0, dd.pool, dd.pool, dd.chunks, dd.chunk_start,
                                       wd.max_kv_len, out=outd, lse=lsed, workspace=wsd, plain=True)
        dnorot = timed(dec_norot, args.steps, args.warmup)
        drot_spread = paired_overhead(dec_lazy, dec_norot)
        cfgd_local = ops.config_of(wd, key_positions=ops.KEYS_LOCAL)
        dlocal = timed(lambda: ops.decode(cfgd_local, dd.q, dd.q_pos0, dd.pool, dd.pool, dd.chunks, dd.chunk_start,
                                          wd.max_kv_len, out=outd, lse=lsed, workspace=wsd), args.steps, args.warmup)
        # Chunk-major shared decode of the same batch: every stored chunk is read once for all of its users.
        t0 = time.perf_counter()
        plan = ops.shared_decode_plan(cfgd, wd.chunks, wd.chunk_start)
        plan_ms = (time.perf_counter() - t0) * 1e3
        dplan = ops.upload_plan(plan, dev)
        wss = torch.empty(max(16, ops.decode_shared_workspace_size(cfgd, wd.batch, plan.max_slots)),
                          dtype=torch.uint8, device=dev)
        dshared = timed(lambda: ops.decode_shared(cfgd, dd.q, dd.q_pos0, dd.pool, dd.pool, dplan, out=outd,
                                                  lse=lsed, workspace=wss), args.steps, args.warmup)
        dshared_local = timed(lambda: ops.decode_shared(cfgd_local, dd.q, dd.q_pos0, dd.pool, dd.pool, dplan,
                                                        out=outd, lse=lsed, workspace=wss), args.steps, args.warmup)
        shared_read_mb = float(plan.read_keys()) * wd.num_kv_heads * wd.head_dim * 2 * 2 / 1e6
        cfgd_alibi = ops.config_of(wd, rope_style=ops.ALIBI)
        dalibi = timed(lambda: ops.decode(cfgd_alibi, dd.q, dd.q_pos0, dd.pool, dd.pool, dd.chunks, dd.chunk_start,
                                          wd.max_kv_len, out=outd, lse=lsed, workspace=wsd), args.steps, args.warmup)
        # The same batch over a paged store: 64-token blocks scattered over the pool, one record per block.
        wpg = W.paginate(wd, 64, seed=7)
        dpg = ops.upload(wpg, dev)
        wspg = torch.empty(max(16, ops.decode_workspace_size(cfgd, wpg.batch, wpg.max_kv_len)), dtype=torch.uint8,
                           device=dev)
        dpaged = timed(lambda: ops.decode(cfgd, dpg.q, dpg.q_pos0, dpg.pool, dpg.pool, dpg.chunks, dpg.chunk_start,
                                          wpg.max_kv_len, out=outd, lse=lsed, workspace=wspg), args.steps, args.warmup)
        plan_pg = ops.upload_plan(ops.shared_decode_plan(cfgd, wpg.chunks, wpg.chunk_start), dev)
        wss_pg = torch.empty(max(16, ops.decode_shared_workspace_size(cfgd, wpg.batch, plan_pg.max_slots)),
                             dtype=torch.uint8, device=dev)
        dpaged_shared = timed(lambda: ops.decode_shared(cfgd, dpg.q, dpg.q_pos0, dpg.pool, dpg.pool, plan_pg,
                                                        out=outd, lse=lsed, workspace=wss_pg), args.steps,
                              args.warmup)
        del dpg, wspg, wss_pg
        tkv = int(wd.chunks["len"].astype(np.int64).sum())
        kmd = torch.empty(cfgd.num_kv_heads * tkv * cfgd.head_dim, dtype=torch.bfloat16, device=dev)
        chd = torch.empty_like(dd.chunks)
        mxc = int(wd.chunks["len"].max())
        dmat = timed(lambda: ops.materialize_k(cfgd, dd.pool, dd.chunks, mxc, tkv, k_out=kmd, chunks_out=chd),
                     max(5, args.steps // 5), 2)
        dplain = timed(lambda: ops.decode(cfgd, dd.q, dd.q_pos0, kmd, dd.pool, chd, dd.chunk_start, wd.max_kv_len,
                                          out=outd, lse=lsed, workspace=wsd, plain=True), args.steps, args.warmup)
        # Every request's table in storage order (lazy_chunk_table_storage_order), for the lazy decode and the
        # baseline alike: the 64 requests' workgroups of one KV head run on one XCD and read the chunks they share
        # in the same order.
        so_t = ops.chunks_tensor(ops.storage_order(wd.chunks, wd.chunk_start), dev)
        dso = timed(lambda: ops.decode(cfgd, dd.q, dd.q_pos0, dd.pool, dd.pool, so_t, dd.chunk_start, wd.max_kv_len,
                                       out=outd, lse=lsed, workspace=wsd), args.steps, args.warmup)
        dso_mat = timed(lambda: ops.materialize_k(cfgd, dd.pool, so_t, mxc, tkv, k_out=kmd, chunks_out=chd),
                        max(5, args.steps // 5), 2)
        dso_plain = timed(lambda: ops.decode(cfgd, dd.q, dd.q_pos0, kmd, dd.pool, chd, dd.chunk_start,
                                             wd.max_kv_len, out=outd, lse=lsed, workspace=wsd, plain=True),
                          args.steps, args.warmup)
        gbps = dbytes / (dms * 1e-3) / 1e9
        result["decode"] = {
            "workload": "rag_decode: batch 64, 32/8 heads, head_dim 128, 16 x 1024-token chunks from a 256-chunk "
                        "pool + 65-token private tail, one query per request; tables in position order, and under "
                        "storage_order in storage order (lazy and baseline alike)",
            "ms": round(dms, 5),
            "logical_hbm_gbps": round(gbps, 1),
            "hbm_frac": round(gbps / PEAK_HBM_GBPS, 4),
            "cold_cache_ms": round(dcold, 5),
            "logical_mb": round(dbytes / 1e6, 1),
            "unique_kv_mb": round(A.unique_kv_bytes(wd) / 1e6, 1),
            "splits": int(wsd_bytes // (wd.batch * wd.num_q_heads * (2 * wd.head_dim + 4))) if wsd_bytes else 1,
            "no_rotation_ms": round(dnorot, 5),
            "rotation_overhead": round(dms / dnorot - 1.0, 4),
            "rotation_overhead_spread": drot_spread,
            "local_keys_ms": round(dlocal, 5),
            "local_keys_logical_hbm_gbps": round(dbytes / (dlocal * 1e-3) / 1e9, 1),
            "shared_ms": round(dshared, 5),
            "shared_logical_gbps": round(dbytes / (dshared * 1e-3) / 1e9, 1),
            "shared_local_keys_ms": round(dshared_local, 5),
            "shared_kv_read_mb": round(shared_read_mb, 1),
            "shared_items": int(plan.items.size),
            "shared_plan_host_ms": round(plan_ms, 3),
            "shared_speedup_vs_per_request": round(dms / dshared, 3),
            "paged64_ms": round(dpaged, 5),
            "alibi_ms": round(dalibi, 5),
            "paged64_shared_ms": round(dpaged_shared, 5),
            "materialize_ms": round(dmat, 5),
            "plain_decode_ms": round(dplain, 5),
            "materialize_then_attend_ms": round(dmat + dplain, 5),
            "speedup_vs_materialize": round((dmat + dplain) / dms, 3),
            "storage_order": {"ms": round(dso, 5),
                              "logical_hbm_gbps": round(dbytes / (dso * 1e-3) / 1e9, 1),
                              "logical_hbm_frac": round(dbytes / (dso * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
                              "materialize_ms": round(dso_mat, 5), "plain_decode_ms": round(dso_plain, 5),
                              "speedup_vs_materialize": round((dso_mat + dso_plain) / dso, 3)},
            "traffic": recorded_traffic("decode_kernel_rag_decode"),
        }
        del kmd, dd

    if not args.no_other:
        result["other_configs"] = other_configs(dev, args.steps, args.warmup, log)

    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_probe_bytes"] = n * 4

    if not args.no_cpu and rank == 0:
        log("cpu baseline: timing the oracle")
        result["cpu_baseline"] = cpu_baseline(wp, flops)

    if rank == 0:
        print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
