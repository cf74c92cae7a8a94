"""Seeded synthetic inputs for the LazyAttention hot path.

This module only draws random numbers and lays them out: it holds none of the method's arithmetic (no rotation,
no scores, no softmax).  Both the fp64 oracle tests and the GPU path take their inputs from here.

The workloads are shape-only stand-ins for the paper's RAG / in-context-learning workloads (retrieved documents
reused across requests at different positions, Sec. 1 and Sec. 4 "Models, Hardware, and Datasets"; few-shot
exemplar chunks recurring in different orders, Appendix "Beyond RAG").  The datasets themselves are not used.
Every value is N(0, 1) float32 rounded to bfloat16 (round-to-nearest-even) unless a workload keeps fp32
originals as well.

Chunk store layout (position-free, Sec. 3.1 "Deferred encoding": keys/values cached without positions):
one flat element array ``pool``; a physical chunk with capacity ``cap`` tokens stores
``K[Hkv][cap][D]`` at ``k_offset`` and ``V[Hkv][cap][D]`` at ``v_offset``.  A request refers to chunks through
records ``{k_offset, v_offset, len, pos_offset, k_stride, v_stride}`` (``CHUNK_DTYPE``, 32 bytes, identical to the
C struct ``lazy_chunk_t``); records of request ``r`` are ``chunks[chunk_start[r]:chunk_start[r+1]]``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

CHUNK_DTYPE = np.dtype(
    [
        ("k_offset", "<i8"),
        ("v_offset", "<i8"),
        ("len", "<i4"),
        ("pos_offset", "<i4"),
        ("k_stride", "<i4"),
        ("v_stride", "<i4"),
    ]
)
assert CHUNK_DTYPE.itemsize == 32


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32 holding exact bf16 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    flat_in = x.reshape(-1)
    flat_out = out.reshape(-1)
    step = 1 << 24
    for s in range(0, flat_in.size, step):
        u = flat_in[s : s + step].view(np.uint32)
        lsb = (u >> np.uint32(16)) & np.uint32(1)
        r = (u + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
        nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
        if nan.any():
            r = np.where(nan, (u | np.uint32(0x00400000)) & np.uint32(0xFFFF0000), r)
        flat_out[s : s + step] = r.view(np.float32)
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already exact bfloat16 numbers (see ``bf16_round``)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


@dataclass
class Workload:
    """One batch of synthetic attention inputs (host arrays)."""

    name: str
    kind: str  # "prefill" or "decode"
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    rope_base: float
    causal: bool
    q: np.ndarray  # float32 [total_q, Hq, D], bf16-exact
    q_start: np.ndarray  # int32 [B+1]
    q_pos0: np.ndarray  # int32 [B]; query token i of request r sits at q_pos0[r] + i
    pool: np.ndarray  # float32 [pool_elems], bf16-exact; holds K and V of every physical chunk
    chunks: np.ndarray  # CHUNK_DTYPE [n_records]
    chunk_start: np.ndarray  # int32 [B+1]
    q_fp32: np.ndarray | None = None  # fp32 originals (tiny workload only)
    pool_fp32: np.ndarray | None = None
    meta: dict = field(default_factory=dict)

    @property
    def batch(self) -> int:
        return int(self.q_start.size - 1)

    @property
    def total_q(self) -> int:
        return int(self.q_start[-1])

    @property
    def q_lens(self) -> np.ndarray:
        return np.diff(self.q_start)

    @property
    def kv_lens(self) -> np.ndarray:
        lens = self.chunks["len"].astype(np.int64)
        return np.array(
            [lens[self.chunk_start[r] : self.chunk_start[r + 1]].sum() for r in range(self.batch)], dtype=np.int64
        )

    @property
    def max_q_len(self) -> int:
        return int(self.q_lens.max()) if self.batch else 0

    @property
    def max_kv_len(self) -> int:
        return int(self.kv_lens.max()) if self.batch else 0

    def q_positions(self) -> np.ndarray:
        """Absolute position of every query token, [total_q] int64."""
        pos = np.empty(self.total_q, dtype=np.int64)
        for r in range(self.batch):
            a, b = int(self.q_start[r]), int(self.q_start[r + 1])
            pos[a:b] = int(self.q_pos0[r]) + np.arange(b - a)
        return pos


class _Store:
    """Allocates physical chunks ``K[Hkv][cap][D]`` + ``V[Hkv][cap][D]`` back to back in one flat pool."""

    def __init__(self, hkv: int, d: int):
        self.hkv, self.d = hkv, d
        self.size = 0
        self.phys = []  # (k_offset, v_offset, cap)

    def add(self, cap: int) -> int:
        block = self.hkv * cap * self.d
        k_off = self.size
        v_off = k_off + block
        self.size = v_off + block
        self.phys.append((k_off, v_off, cap))
        return len(self.phys) - 1


def _records(store: _Store, uses):
    """uses: list (per request) of lists of (phys_id, length, pos_offset)."""
    n = sum(len(u) for u in uses)
    rec = np.zeros(n, dtype=CHUNK_DTYPE)
    start = np.zeros(len(uses) + 1, dtype=np.int32)
    i = 0
    for r, u in enumerate(uses):
        for pid, length, pos in u:
            k_off, v_off, cap = store.phys[pid]
            assert 0 < length <= cap
            rec[i] = (k_off, v_off, length, pos, cap, cap)
            i += 1
        start[r + 1] = i
    return rec, start


def _fill(rng, n, keep_fp32=False, slack=None):
    vals = rng.standard_normal(n, dtype=np.float32)
    fp32 = vals.copy() if keep_fp32 else None
    return bf16_round(vals), fp32


def _finish(name, kind, hq, hkv, d, base, store, uses, q_lens, q_pos0, rng, causal=True, keep_fp32=False,
            slack_fill=None, meta=None):
    rec, cstart = _records(store, uses)
    pool, pool32 = _fill(rng, store.size, keep_fp32)
    if slack_fill is not None:
        # Poison capacity slack (tokens >= len of a physical chunk's last use) so out-of-range reads show up.
        used = {}
        for u in uses:
            for pid, length, _ in u:
                used[pid] = max(used.get(pid, 0), length)
        for pid, (k_off, v_off, cap) in enumerate(store.phys):
            ln = used.get(pid, cap)
            if ln < cap:
                for off in (k_off, v_off):
                    blk = pool[off : off + hkv * cap * d].reshape(hkv, cap, d)
                    blk[:, ln:, :] = slack_fill
    q_start = np.zeros(len(q_lens) + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(q_lens)
    qv, q32 = _fill(rng, int(q_start[-1]) * hq * d, keep_fp32)
    q = qv.reshape(int(q_start[-1]), hq, d)
    m = dict(meta or {})
    m.update(_reuse_stats(uses, store))
    return Workload(
        name=name, kind=kind, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, rope_base=float(base),
        causal=causal, q=q, q_start=q_start, q_pos0=np.asarray(q_pos0, dtype=np.int32), pool=pool,
        chunks=rec, chunk_start=cstart, q_fp32=None if q32 is None else q32.reshape(q.shape),
        pool_fp32=pool32, meta=m,
    )


def _reuse_stats(uses, store):
    count = {}
    offsets = {}
    for u in uses:
        for pid, _, pos in u:
            count[pid] = count.get(pid, 0) + 1
            offsets.setdefault(pid, set()).add(pos)
    shared = [c for c in count.values()]
    return {
        "physical_chunks_used": len(count),
        "records": sum(len(u) for u in uses),
        "uses_per_used_chunk": float(np.mean(shared)) if shared else 0.0,
        "distinct_offsets_per_used_chunk": float(np.mean([len(s) for s in offsets.values()])) if offsets else 0.0,
    }


# --------------------------------------------------------------------------------------------------------------
# Workloads.  Defaults are the full sizes; tests pass smaller sizes for the same structure.
# --------------------------------------------------------------------------------------------------------------


def tiny_rag_prefill(seed: int = 0, slack_fill=None) -> Workload:
    """4 stored-unrotated chunks of 64 tokens at offsets 0/64/128/192, 16 causal query tokens at 256..271,
    2 query heads over 1 KV head, head_dim 64, RoPE base 1e4, batch 1; fp32 originals kept."""
    rng = np.random.default_rng(seed)
    hq, hkv, d, base = 2, 1, 64, 1.0e4
    store = _Store(hkv, d)
    docs = [store.add(64) for _ in range(4)]
    own = store.add(16)
    uses = [[(docs[i], 64, 64 * i) for i in range(4)] + [(own, 16, 256)]]
    return _finish("tiny_rag_prefill", "prefill", hq, hkv, d, base, store, uses, [16], [256], rng,
                   keep_fp32=True, slack_fill=slack_fill)


def rag_prefill(seed: int = 1, batch: int = 8, hq: int = 32, hkv: int = 8, d: int = 128, base: float = 5.0e5,
                prefix_len: int = 128, n_chunks: int = 10, chunk_len: int = 512, pool_chunks: int = 64,
                q_len: int = 64, slack_fill=None) -> Workload:
    """Llama-3-8B-shaped RAG prefill: shared system prefix at 0, then ``n_chunks`` distinct chunks drawn uniformly
    from a pool, random order, placed contiguously, then the causal question (its own K/V is the last record)."""
    rng = np.random.default_rng(seed)
    store = _Store(hkv, d)
    prefix = store.add(prefix_len) if prefix_len > 0 else None
    pool_ids = [store.add(chunk_len) for _ in range(pool_chunks)]
    uses, q_pos0 = [], []
    for _ in range(batch):
        pick = rng.choice(pool_chunks, size=n_chunks, replace=False)
        u = [(prefix, prefix_len, 0)] if prefix is not None else []
        pos = prefix_len
        for c in pick:
            u.append((pool_ids[int(c)], chunk_len, pos))
            pos += chunk_len
        uses.append(u)
        q_pos0.append(pos)
    for r in range(batch):
        own = store.add(q_len)
        uses[r].append((own, q_len, q_pos0[r]))
    return _finish("rag_prefill", "prefill", hq, hkv, d, base, store, uses, [q_len] * batch, q_pos0, rng,
                   slack_fill=slack_fill,
                   meta=dict(prefix_len=prefix_len, n_chunks=n_chunks, chunk_len=chunk_len, pool_chunks=pool_chunks))


def rag_decode(seed: int = 2, batch: int = 64, hq: int = 32, hkv: int = 8, d: int = 128, base: float = 5.0e5,
               n_chunks: int = 16, chunk_len: int = 1024, pool_chunks: int = 256, tail_len: int = 65,
               tail_cap: int = 128, slack_fill=None) -> Workload:
    """Llama-3-8B-shaped decode: ``n_chunks`` distinct chunks from a shared pool in random order, contiguous,
    then a private tail of ``tail_len`` generated tokens whose last token is the new one (already appended);
    one query per request at the last tail position."""
    rng = np.random.default_rng(seed)
    store = _Store(hkv, d)
    pool_ids = [store.add(chunk_len) for _ in range(pool_chunks)]
    uses, q_pos = [], []
    for _ in range(batch):
        pick = rng.choice(pool_chunks, size=n_chunks, replace=False)
        u = [(pool_ids[int(c)], chunk_len, i * chunk_len) for i, c in enumerate(pick)]
        uses.append(u)
    for r in range(batch):
        tail = store.add(max(tail_cap, tail_len))
        start = n_chunks * chunk_len
        uses[r].append((tail, tail_len, start))
        q_pos.append(start + tail_len - 1)
    return _finish("rag_decode", "decode", hq, hkv, d, base, store, uses, [1] * batch, q_pos, rng,
                   slack_fill=slack_fill,
                   meta=dict(n_chunks=n_chunks, chunk_len=chunk_len, pool_chunks=pool_chunks, tail_len=tail_len))


def icl_prefill(seed: int = 3, batch: int = 4, hq: int = 32, hkv: int = 8, d: int = 128, base: float = 5.0e5,
                n_chunks: int = 128, chunk_len: int = 256, q_len: int = 256, decode_steps: int = 128,
                slack_fill=None, private: bool = False) -> Workload:
    """Many-shot in-context learning: one shared pool of exemplar chunks, an independent permutation of all of
    them per request (contiguous), then a causal query; the query's own K/V chunk has room for
    ``decode_steps`` more tokens.  ``private``: every request gets its own pool of exemplars instead (no sharing)."""
    rng = np.random.default_rng(seed)
    store = _Store(hkv, d)
    pool_ids = [store.add(chunk_len) for _ in range(n_chunks)]
    uses, q_pos0 = [], []
    for r in range(batch):
        if private and r > 0:
            pool_ids = [store.add(chunk_len) for _ in range(n_chunks)]
        perm = rng.permutation(n_chunks)
        uses.append([(pool_ids[int(c)], chunk_len, i * chunk_len) for i, c in enumerate(perm)])
        q_pos0.append(n_chunks * chunk_len)
    for r in range(batch):
        own = store.add(q_len + decode_steps)
        uses[r].append((own, q_len, q_pos0[r]))
    return _finish("icl_prefill", "prefill", hq, hkv, d, base, store, uses, [q_len] * batch, q_pos0, rng,
                   slack_fill=slack_fill,
                   meta=dict(n_chunks=n_chunks, chunk_len=chunk_len, decode_steps=decode_steps))


def icl_decode_step(w: Workload, step: int, seed: int = 33) -> Workload:
    """Decode step ``step`` (0-based) after ``icl_prefill``: the query's own chunk has grown by step+1 tokens
    (fresh N(0,1) K/V written into its capacity), one new query per request at the last position."""
    rng = np.random.default_rng(seed + step)
    pool = w.pool.copy()
    chunks = w.chunks.copy()
    hkv, d = w.num_kv_heads, w.head_dim
    q_pos = []
    for r in range(w.batch):
        i = int(w.chunk_start[r + 1]) - 1
        rec = chunks[i]
        new_len = int(w.q_lens[r]) + step + 1
        assert new_len <= int(rec["k_stride"])
        for off, stride in ((int(rec["k_offset"]), int(rec["k_stride"])), (int(rec["v_offset"]), int(rec["v_stride"]))):
            blk = pool[off : off + hkv * stride * d].reshape(hkv, stride, d)
            lo = int(rec["len"])
            blk[:, lo:new_len, :] = bf16_round(rng.standard_normal((hkv, new_len - lo, d), dtype=np.float32))
        chunks[i]["len"] = new_len
        q_pos.append(int(rec["pos_offset"]) + new_len - 1)
    q = bf16_round(rng.standard_normal((w.batch, w.num_q_heads, d), dtype=np.float32))
    q_start = np.arange(w.batch + 1, dtype=np.int32)
    return Workload(name=f"icl_decode_step{step}", kind="decode", num_q_heads=w.num_q_heads, num_kv_heads=hkv,
                    head_dim=d, rope_base=w.rope_base, causal=w.causal, q=q, q_start=q_start,
                    q_pos0=np.asarray(q_pos, dtype=np.int32), pool=pool, chunks=chunks,
                    chunk_start=w.chunk_start.copy(), meta=dict(w.meta, step=step))


def varlen_rag(seed: int = 4, batch: int = 16, hq: int = 28, hkv: int = 4, d: int = 128, base: float = 1.0e6,
               pool_chunks: int = 200, len_lo: int = 128, len_hi: int = 2048, k_lo: int = 8, k_hi: int = 24,
               q_lo: int = 32, q_hi: int = 256, zipf_alpha: float = 2.1, slack_fill=None) -> Workload:
    """Variable-length RAG: chunk lengths uniform in [len_lo, len_hi]; each request takes U[k_lo, k_hi] chunks
    drawn without replacement with Zipf(alpha) popularity over the pool (skewed reuse), in random order, placed
    contiguously; query length uniform in [q_lo, q_hi]; ragged tables as flat arrays with prefix sums."""
    rng = np.random.default_rng(seed)
    store = _Store(hkv, d)
    lens = rng.integers(len_lo, len_hi + 1, size=pool_chunks)
    pool_ids = [store.add(int(n)) for n in lens]
    p = np.arange(1, pool_chunks + 1, dtype=np.float64) ** (-zipf_alpha)
    p /= p.sum()
    uses, q_pos0, q_lens = [], [], []
    for _ in range(batch):
        k = int(rng.integers(k_lo, k_hi + 1))
        pick = rng.choice(pool_chunks, size=k, replace=False, p=p)
        rng.shuffle(pick)
        u, pos = [], 0
        for c in pick:
            u.append((pool_ids[int(c)], int(lens[c]), pos))
            pos += int(lens[c])
        uses.append(u)
        q_pos0.append(pos)
        q_lens.append(int(rng.integers(q_lo, q_hi + 1)))
    for r in range(batch):
        own = store.add(q_lens[r])
        uses[r].append((own, q_lens[r], q_pos0[r]))
    return _finish("varlen_rag", "prefill", hq, hkv, d, base, store, uses, q_lens, q_pos0, rng,
                   slack_fill=slack_fill, meta=dict(pool_chunks=pool_chunks, zipf_alpha=zipf_alpha))


def custom(seed: int, hq: int, hkv: int, d: int, base: float, requests, kind: str = "prefill", causal: bool = True,
           slack_fill=None, name: str = "custom") -> Workload:
    """Free-form workload.  ``requests``: list of dicts with ``chunks`` (list of (length, pos_offset) for private
    chunks, or (phys_key, length, pos_offset) to share a chunk between requests through a common key),
    ``q_len`` and ``q_pos0``."""
    rng = np.random.default_rng(seed)
    store = _Store(hkv, d)
    shared = {}
    uses = []
    for req in requests:
        u = []
        for item in req["chunks"]:
            if len(item) == 3:
                key, length, pos = item
                if key not in shared:
                    shared[key] = store.add(length)
                pid = shared[key]
                assert store.phys[pid][2] >= length
            else:
                length, pos = item
                pid = store.add(length)
            u.append((pid, length, pos))
        uses.append(u)
    return _finish(name, kind, hq, hkv, d, base, store, uses, [r["q_len"] for r in requests],
                   [r["q_pos0"] for r in requests], rng, causal=causal, slack_fill=slack_fill)


def paginate(w: Workload, block_tokens: int, seed: int = 0) -> Workload:
    """Block-granular (paged) copy of a workload's store, as a paged KV allocator would hold it (Sec. 3.2 mentions
    PagedAttention's block layout).  Every physical chunk is cut into blocks of ``block_tokens`` tokens; each block
    stores ``K[Hkv][block_tokens][D]`` and ``V[Hkv][block_tokens][D]`` at its own place in a new pool, the blocks in
    a random order.  Each record becomes one record per block it covers: len = the block's share of the record,
    pos_offset = record offset + block start, strides = block_tokens.  Pure data movement: the attention inputs are
    the same keys at the same positions (for a local-position store each block then holds keys at block-relative
    local positions, which is a different but equally valid store)."""
    rng = np.random.default_rng(seed)
    hkv, d, bt = w.num_kv_heads, w.head_dim, int(block_tokens)
    phys = {}
    for rec in w.chunks:
        key = (int(rec["k_offset"]), int(rec["v_offset"]))
        phys[key] = max(phys.get(key, 0), int(rec["k_stride"]), int(rec["v_stride"]))
    blocks = []  # (k_offset, v_offset, block index) of every block of every physical chunk
    for (ko, vo), cap in phys.items():
        for b in range(-(-cap // bt)):
            blocks.append((ko, vo, b))
    order = rng.permutation(len(blocks))
    blk_elems = hkv * bt * d
    pool = np.zeros(2 * blk_elems * len(blocks), dtype=np.float32)
    where = {}
    for slot, bi in enumerate(order):
        ko, vo, b = blocks[bi]
        where[(ko, vo, b)] = slot
    new_recs = []
    for rec in w.chunks:
        ko, vo = int(rec["k_offset"]), int(rec["v_offset"])
        n = int(rec["len"])
        for b in range(-(-n // bt)):
            slot = where[(ko, vo, b)]
            nk = min(bt, n - b * bt)
            new_recs.append((2 * slot * blk_elems, (2 * slot + 1) * blk_elems, nk, int(rec["pos_offset"]) + b * bt,
                             bt, bt))
    # copy the data block by block (whole capacity, so capacity slack travels with it)
    recs_by_phys = {}
    for rec in w.chunks:
        recs_by_phys.setdefault((int(rec["k_offset"]), int(rec["v_offset"])), rec)
    for (ko, vo, b), slot in where.items():
        rec = recs_by_phys[(ko, vo)]
        kst, vst = int(rec["k_stride"]), int(rec["v_stride"])
        for base_old, st, base_new in ((ko, kst, 2 * slot * blk_elems), (vo, vst, (2 * slot + 1) * blk_elems)):
            lo, hi = b * bt, min(st, (b + 1) * bt)
            if hi <= lo:
                continue
            src = w.pool[base_old: base_old + hkv * st * d].reshape(hkv, st, d)[:, lo:hi, :]
            dst = pool[base_new: base_new + blk_elems].reshape(hkv, bt, d)
            dst[:, : hi - lo, :] = src
    chunks = np.array(new_recs, dtype=CHUNK_DTYPE)
    counts = []
    for r in range(w.batch):
        counts.append(sum(-(-int(rec["len"]) // bt) for rec in w.chunks[w.chunk_start[r]: w.chunk_start[r + 1]]))
    chunk_start = np.zeros(w.batch + 1, dtype=np.int32)
    chunk_start[1:] = np.cumsum(counts)
    meta = dict(w.meta, block_tokens=bt, blocks=len(blocks))
    return Workload(name=f"{w.name}_paged{bt}", kind=w.kind, num_q_heads=w.num_q_heads, num_kv_heads=hkv,
                    head_dim=d, rope_base=w.rope_base, causal=w.causal, q=w.q, q_start=w.q_start, q_pos0=w.q_pos0,
                    pool=pool, chunks=chunks, chunk_start=chunk_start, meta=meta)


def by_name(name: str, **kw) -> Workload:
    table = {
        "tiny_rag_prefill": tiny_rag_prefill,
        "rag_prefill": rag_prefill,
        "rag_decode": rag_decode,
        "icl_prefill": icl_prefill,
        "varlen_rag": varlen_rag,
    }
    return table[name](**kw)
