"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle, element by element on seeded inputs.

Tolerance (bf16 outputs): max |gpu - oracle| <= 2e-2 and mean |gpu - oracle| <= 2e-3; lse within 2e-2 where finite
and -inf exactly where the oracle has no visible key.  Lazy (in-kernel rotation) and materialise-then-attend
compute the same rotated bf16 keys, so they must agree bit for bit.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

from oracle import lazy_oracle as O
from paper_2606_04302_amd import ops
from paper_2606_04302_amd import workloads as W

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS, LSE_ABS = 2e-2, 2e-3, 2e-2


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ops.lib()
    torch.cuda.init()
    yield


def oracle(w, requests=None, **kw):
    if w.kind == "decode":
        return O.lazy_decode(w.q, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, w.num_q_heads, w.num_kv_heads,
                             w.head_dim, w.rope_base, w.causal, requests=requests, **kw)
    return O.lazy_attention(w.q, w.q_start, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, w.num_q_heads,
                            w.num_kv_heads, w.head_dim, w.rope_base, w.causal, requests=requests, **kw)


def rows_of(w, requests):
    idx = []
    for r in requests:
        idx.extend(range(int(w.q_start[r]), int(w.q_start[r + 1])))
    return np.array(idx, dtype=np.int64)


def assert_close(out, lse, ref_o, ref_l, rows=None, tag=""):
    o = out.float().cpu().numpy().astype(np.float64)
    l = lse.cpu().numpy().astype(np.float64) if lse is not None else None
    if rows is not None:
        o, ref_o = o[rows], ref_o[rows]
        if l is not None:
            l, ref_l = l[rows], ref_l[rows]
    assert np.isfinite(o).all(), f"{tag}: non-finite output"
    err = np.abs(o - ref_o)
    print(f"{tag}: max_abs={err.max():.3e} mean_abs={err.mean():.3e} rms_ref={np.sqrt((ref_o ** 2).mean()):.3e}",
          flush=True)
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, f"{tag}: max {err.max()} mean {err.mean()}"
    if l is not None:
        inf = np.isneginf(ref_l)
        assert np.array_equal(np.isneginf(l), inf), f"{tag}: lse -inf pattern differs"
        if (~inf).any():
            le = np.abs(l[~inf] - ref_l[~inf]).max()
            assert le <= LSE_ABS, f"{tag}: lse err {le}"


def oracle_kw(cfg_kw):
    """The oracle's arguments for a launch configured with ``cfg_kw``."""
    cfg_kw = cfg_kw or {}
    okw = {}
    if cfg_kw.get("softmax_scale"):
        okw["softmax_scale"] = cfg_kw["softmax_scale"]
    if cfg_kw.get("key_positions") == ops.KEYS_LOCAL:
        okw["key_positions"] = "local"
    if cfg_kw.get("rope_style") == ops.ROPE_INTERLEAVED:
        okw["pairing"] = "interleaved"
    if cfg_kw.get("rope_style") == ops.ALIBI:
        okw["pairing"] = "alibi"
    return okw


def run_and_check(w, tag, cfg_kw=None, requests=None):
    dw = ops.upload(w)
    cfg = ops.config_of(w, **(cfg_kw or {}))
    out, lse = ops.run_lazy(dw, cfg)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle(w, requests=requests, **oracle_kw(cfg_kw))
    rows = None if requests is None else rows_of(w, requests)
    assert_close(out, lse, ref_o, ref_l, rows, tag)
    return dw, out, lse


# --------------------------------------------------------------------------------------------------------------


def test_tiny_rag_prefill_matches_oracle():
    w = W.tiny_rag_prefill(seed=0)
    dw, out, lse = run_and_check(w, "tiny bf16")
    # against the fp32 originals as well (the bf16 rounding of inputs is inside the tolerance)
    ref_o, _ = O.lazy_attention(w.q_fp32, w.q_start, w.q_pos0, w.pool_fp32, w.pool_fp32, w.chunks, w.chunk_start,
                                w.num_q_heads, w.num_kv_heads, w.head_dim, w.rope_base, w.causal)
    err = np.abs(out.float().cpu().numpy() - ref_o)
    print(f"tiny vs fp32 originals: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


PREFILL_CASES = {
    # name: (builder, kwargs, cfg kwargs)
    "rag_d128_g4": (W.rag_prefill, dict(seed=11, batch=2, hq=8, hkv=2, d=128, prefix_len=40, n_chunks=3,
                                        chunk_len=100, pool_chunks=5, q_len=37), {}),
    "rag_d64_g2_split3": (W.rag_prefill, dict(seed=12, batch=3, hq=4, hkv=2, d=64, prefix_len=0, n_chunks=4,
                                              chunk_len=70, pool_chunks=6, q_len=50), dict(num_splits=3)),
    "rag_d128_g1_split1": (W.rag_prefill, dict(seed=13, batch=2, hq=2, hkv=2, d=128, prefix_len=17, n_chunks=2,
                                               chunk_len=64, pool_chunks=3, q_len=129), dict(num_splits=1)),
    "varlen_g7": (W.varlen_rag, dict(seed=14, batch=4, hq=28, hkv=4, d=128, pool_chunks=10, len_lo=1, len_hi=200,
                                     k_lo=2, k_hi=5, q_lo=1, q_hi=40), {}),
    "varlen_g8_d64": (W.varlen_rag, dict(seed=15, batch=3, hq=16, hkv=2, d=64, pool_chunks=8, len_lo=30,
                                         len_hi=300, k_lo=1, k_hi=4, q_lo=20, q_hi=70), dict(num_splits=2)),
    # ragged batch of 8: batch x splits is a multiple of 8, so the workgroups take the interleaved XCD map
    "varlen_g7_b8": (W.varlen_rag, dict(seed=30, batch=8, hq=28, hkv=4, d=128, pool_chunks=10, len_lo=40,
                                        len_hi=300, k_lo=2, k_hi=4, q_lo=10, q_hi=90), {}),
    "icl_small": (W.icl_prefill, dict(seed=16, batch=2, hq=8, hkv=2, d=128, n_chunks=12, chunk_len=32, q_len=80,
                                      decode_steps=4), {}),
    # eight-wave workgroups (80 x 4 = 320 packed rows: a full and a partial row tile) writing the final output and
    # log-sum-exp directly (one split)
    "icl_small_split1": (W.icl_prefill, dict(seed=17, batch=2, hq=8, hkv=2, d=128, n_chunks=12, chunk_len=32, q_len=80,
                                             decode_steps=4), dict(num_splits=1)),
}


@pytest.mark.parametrize("name", list(PREFILL_CASES))
def test_prefill_matches_oracle(name):
    fn, kw, ckw = PREFILL_CASES[name]
    run_and_check(fn(**kw), name, ckw)


def test_prefill_non_causal_and_scale_override():
    w = W.rag_prefill(seed=21, batch=2, hq=8, hkv=4, d=128, prefix_len=8, n_chunks=2, chunk_len=90, pool_chunks=4,
                      q_len=20)
    w.causal = False
    run_and_check(w, "non-causal")
    w.causal = True
    run_and_check(w, "scale 0.05", dict(softmax_scale=0.05))


DECODE_CASES = {
    "d128_g4": (dict(seed=31, batch=3, hq=8, hkv=2, d=128, n_chunks=5, chunk_len=200, pool_chunks=7, tail_len=9,
                     tail_cap=16), {}),
    "d128_g4_split1": (dict(seed=32, batch=2, hq=8, hkv=2, d=128, n_chunks=3, chunk_len=130, pool_chunks=4,
                            tail_len=1, tail_cap=8), dict(num_splits=1)),
    "d64_g7_split5": (dict(seed=33, batch=2, hq=14, hkv=2, d=64, n_chunks=4, chunk_len=150, pool_chunks=5,
                           tail_len=33, tail_cap=40), dict(num_splits=5)),
    "d128_g20_two_head_groups": (dict(seed=34, batch=2, hq=40, hkv=2, d=128, n_chunks=2, chunk_len=300,
                                      pool_chunks=3, tail_len=5, tail_cap=8), {}),
    "d128_mha": (dict(seed=35, batch=2, hq=4, hkv=4, d=128, n_chunks=2, chunk_len=257, pool_chunks=3, tail_len=2,
                      tail_cap=2), dict(num_splits=2)),
}


@pytest.mark.parametrize("name", list(DECODE_CASES))
def test_decode_matches_oracle(name):
    kw, ckw = DECODE_CASES[name]
    run_and_check(W.rag_decode(**kw), "decode " + name, ckw)


# Cache hint LAZY_CACHE_STREAM: the decode entry points read K and V with non-temporal loads.  Only the cache policy
# of those loads changes, so every output must be bit-identical to the default hint's; the streamed NoPE result is
# also checked against the oracle.
STREAM_MODES = {"nope": {}, "local": dict(key_positions=ops.KEYS_LOCAL), "interleaved": dict(rope_style=ops.ROPE_INTERLEAVED),
                "alibi": dict(rope_style=ops.ALIBI), "plain": {}, "noalloc": {}, "shared": {},
                "shared_local": dict(key_positions=ops.KEYS_LOCAL)}


@pytest.mark.parametrize("mode", list(STREAM_MODES))
@pytest.mark.parametrize("name", ["d128_g4", "d128_g4_split1", "d64_g7_split5"])
def test_stream_cache_hint_decode_is_bitwise_the_default(name, mode):
    kw, ckw = DECODE_CASES[name]
    w = W.rag_decode(**kw)
    dw = ops.upload(w)
    plain = None
    if mode == "plain":
        total = int(w.chunks["len"].astype(np.int64).sum())
        plain = ops.materialize_k(dw.cfg, dw.pool, dw.chunks, int(w.chunks["len"].max()), total)
    res = []
    for hint in (ops.CACHE_DEFAULT, ops.CACHE_STREAM):
        cfg = ops.config_of(w, **ckw, **STREAM_MODES[mode], cache_hint=hint)
        if mode == "noalloc":
            out = torch.empty_like(dw.q)
            lse = torch.empty((w.total_q, w.num_q_heads), dtype=torch.float32, device="cuda")
            ops.decode_noalloc(cfg, dw.q, dw.q_pos0, dw.pool, dw.pool, dw.chunks, dw.chunk_start,
                               max(1, w.max_kv_len), out, lse)
            torch.cuda.synchronize()
            res.append((out.clone(), lse.clone()))
        elif mode.startswith("shared"):
            lse = torch.empty((w.total_q, w.num_q_heads), dtype=torch.float32, device="cuda")
            plan = ops.upload_plan(ops.shared_decode_plan(cfg, w.chunks, w.chunk_start, 256))
            out, lse = ops.decode_shared(cfg, dw.q, dw.q_pos0, dw.pool, dw.pool, plan, lse=lse)
            torch.cuda.synchronize()
            res.append((out.clone(), lse.clone()))
        elif plain is not None:
            res.append(ops.run_lazy(dw, cfg, plain_k=plain[0], plain_chunks=plain[1]))
        else:
            res.append(ops.run_lazy(dw, cfg))
    torch.cuda.synchronize()
    (o0, l0), (o1, l1) = res
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16)), (name, mode)
    assert torch.equal(l0, l1), (name, mode)
    if mode in ("nope", "shared"):
        ref_o, ref_l = oracle(w)
        assert_close(o1, l1, ref_o, ref_l, tag=f"stream hint {mode} {name}")


@pytest.mark.parametrize("kind", ["prefill", "decode"])
def test_lazy_equals_materialize_then_attend_bitwise(kind):
    if kind == "prefill":
        w = W.rag_prefill(seed=41, batch=3, hq=8, hkv=2, d=128, prefix_len=30, n_chunks=3, chunk_len=150,
                          pool_chunks=5, q_len=70)
    else:
        w = W.rag_decode(seed=42, batch=3, hq=8, hkv=2, d=128, n_chunks=4, chunk_len=190, pool_chunks=6,
                         tail_len=7, tail_cap=12)
    dw = ops.upload(w)
    out_l, lse_l = ops.run_lazy(dw)
    (out_m, lse_m), (k_out, ch_out) = ops.run_materialized(dw)
    torch.cuda.synchronize()
    assert torch.equal(out_l.view(torch.int16), out_m.view(torch.int16))
    assert torch.equal(lse_l, lse_m)


def test_materialized_keys_match_oracle():
    w = W.rag_prefill(seed=43, batch=2, hq=4, hkv=2, d=128, prefix_len=10, n_chunks=2, chunk_len=77, pool_chunks=3,
                      q_len=5)
    dw = ops.upload(w)
    cfg = dw.cfg
    total = int(w.chunks["len"].astype(np.int64).sum())
    k_out, ch_out = ops.materialize_k(cfg, dw.pool, dw.chunks, int(w.chunks["len"].max()), total)
    torch.cuda.synchronize()
    recs = ops.chunks_from_tensor(ch_out)
    ref = O.materialize_k(w.pool, w.chunks, w.chunk_start, 2, 128, w.rope_base)
    got = k_out.float().cpu().numpy()
    base = 0
    for r in range(w.batch):
        a, b = int(w.chunk_start[r]), int(w.chunk_start[r + 1])
        assert int(recs[a]["k_offset"]) == base
        start = 0
        for i in range(a, b):
            n = int(recs[i]["len"])
            assert int(recs[i]["k_stride"]) == n and int(recs[i]["v_offset"]) == int(w.chunks[i]["v_offset"])
            blk = got[int(recs[i]["k_offset"]): int(recs[i]["k_offset"]) + 2 * n * 128].reshape(2, n, 128)
            # one bf16 rounding of an fp32 rotation: relative error <= 2^-8 plus fp32 angle error
            np.testing.assert_allclose(blk, ref[r][:, start:start + n], rtol=2 ** -8, atol=1e-5)
            start += n
            base += 2 * n * 128


# Split counts cover each merge variant (up to 4 splits; 5..32; more) and, past 64 splits, several rounds of loads
# whose running maximum must be rescaled.
@pytest.mark.parametrize("s,rows,d", [(5, 37, 128), (2, 300, 64), (3, 12, 128), (13, 70, 128), (32, 10, 128),
                                      (33, 50, 128), (64, 9, 64), (129, 20, 128), (200, 11, 64)])
def test_combine_entry_point_matches_oracle_merge(s, rows, d):
    rng = np.random.default_rng(5 + s)
    m = rng.normal(0, 3, size=(s, rows))
    m[1, :4] = -np.inf  # empty splits
    m[:, 7] = -np.inf   # a row with no key at all
    l = np.where(np.isfinite(m), rng.uniform(1, 50, size=(s, rows)), 0.0)
    acc = np.where(np.isfinite(m)[..., None], rng.normal(size=(s, rows, d)), 0.0)
    ref_o, ref_l = O.merge_partials(m, l, acc)
    # the kernels' partial format: per split the normalised output (bf16) and its log-sum-exp m + ln(l)
    fin = np.isfinite(m)
    part_o = np.where(fin[..., None], acc / np.where(fin, l, 1.0)[..., None], 0.0)
    part_lse = np.where(fin, m + np.log(np.where(fin, l, 1.0)), -np.inf)
    po = torch.tensor(part_o, dtype=torch.float32, device="cuda").to(torch.bfloat16)
    pl = torch.tensor(part_lse, dtype=torch.float32, device="cuda")
    lse = torch.empty(rows, dtype=torch.float32, device="cuda")
    out, _ = ops.combine(po, pl, lse=lse)
    torch.cuda.synchronize()
    assert_close(out, lse, ref_o, ref_l, tag="combine")


def test_edge_cases_empty_request_no_visible_key_len1_chunks_nan_slack():
    reqs = [
        dict(chunks=[(5, 100)], q_len=3, q_pos0=2),                        # keys after every query: none visible
        dict(chunks=[(1, 0), (1, 1), (1, 2), ("s", 65, 3)], q_len=0, q_pos0=68),  # no query tokens
        dict(chunks=[("s", 65, 10), (1, 80), (130, 81)], q_len=64, q_pos0=150),
        dict(chunks=[], q_len=2, q_pos0=0),                                # no chunk at all
        dict(chunks=[(1, 0)], q_len=1, q_pos0=0),                          # single key
    ]
    w = W.custom(51, 8, 2, 128, 1e4, reqs, slack_fill=np.nan)
    run_and_check(w, "edge prefill")
    run_and_check(w, "edge prefill split4", dict(num_splits=4))
    wd = W.rag_decode(seed=52, batch=2, hq=8, hkv=2, d=128, n_chunks=2, chunk_len=64, pool_chunks=3, tail_len=3,
                      tail_cap=64, slack_fill=np.nan)
    run_and_check(wd, "edge decode NaN slack")


def test_store_is_read_only():
    w = W.rag_prefill(seed=61, batch=4, hq=8, hkv=2, d=128, prefix_len=20, n_chunks=3, chunk_len=64, pool_chunks=3,
                      q_len=16)
    dw = ops.upload(w)
    before = dw.pool.clone()
    ops.run_lazy(dw)
    ops.run_materialized(dw)
    torch.cuda.synchronize()
    assert torch.equal(before.view(torch.int16), dw.pool.view(torch.int16))


DISCRIMINATION_REQS = [dict(chunks=[(24, 5 + 37 * r), (24, 300 + 11 * r), (4, 400 + 3 * r)], q_len=4,
                            q_pos0=400 + 3 * r) for r in range(4)]


def test_position_discrimination():
    """Off-by-one position bugs cannot hide under the tolerance: on short chunks that each carry real attention
    mass, the GPU result of every request is far closer (in mean error) to the oracle than to the oracle with any
    one of its chunks moved by one position.

    The bar comes from the CPU emulation of the kernels' bf16 rounding points (tests/bf16_emulation.py): on this
    workload (seed 71) the emulated output is 22.8x closer to the oracle than to the worst shifted oracle (seeds 72
    and 73 of the same recipe: 25.1x and 18.7x), with max / mean error 4.6e-3 / 5.1e-4.  The test asks for 8x,
    below the emulated worst case by more than 2x, to leave room for the kernels' own fp32 rounding."""
    w = W.custom(71, 4, 2, 128, 1e4, DISCRIMINATION_REQS)
    dw = ops.upload(w)
    out, lse = ops.run_lazy(dw)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    ref, ref_l = oracle(w)
    assert_close(out, lse, ref, ref_l, tag="discrimination workload")
    for i in range(len(w.chunks)):
        r = int(np.searchsorted(w.chunk_start, i, side="right")) - 1
        rows = slice(int(w.q_start[r]), int(w.q_start[r + 1]))
        e0 = np.abs(o[rows] - ref[rows]).mean()
        for d in (-1, 1):
            w2 = W.Workload(**{**w.__dict__})
            w2.chunks = w.chunks.copy()
            w2.chunks["pos_offset"][i] += d
            e1 = np.abs(o[rows] - oracle(w2)[0][rows]).mean()
            assert e1 > 8 * e0, (i, d, e0, e1)


def test_position_discrimination_sharpened_scores():
    """Sharpened scores (queries scaled by 8, nearly one-hot softmax).  Two things change against the unsharpened
    case, both visible in the CPU emulation of the kernels' bf16 rounding points (tests/bf16_emulation.py):
     - the bf16 rounding of the rotated keys is amplified 8x in the scores, so the error against the fp64 oracle
       exceeds the tolerance bar of max 2e-2 (emulated max / mean 3.9e-2..6.6e-2 / 2.7e-3..3.3e-3 on seeds 71-74 of this
       recipe; the GPU's own max error is held to 1.5x the emulated one, computed here);
     - a chunk whose keys carry no mass moves the output very little when shifted, so against the fp64 oracle
       the shift margin falls to 1.2x-1.9x (mean error).
    Discrimination is therefore checked against the emulation itself, which rounds where the kernels round: for
    every chunk and shift +-1 the GPU result must be at least 10x closer (mean error over the request's rows) to
    the emulation at the true positions than to the emulation with that chunk shifted.  On this workload (seed 74)
    the smallest emulated displacement of a shift is 4.0e-3 (mean), the emulation's own error against the oracle
    is 6.6e-2 / 3.3e-3 (max / mean), and on an MI355X the kernels' output lies 9.3e-5 (mean) from the emulation,
    a worst shift margin of 42x."""
    import bf16_emulation as E

    w = W.custom(74, 4, 2, 128, 1e4, DISCRIMINATION_REQS)
    w = dataclasses.replace(w, q=w.q * 8.0)  # exact in bf16
    dw = ops.upload(w)
    out, _ = ops.run_lazy(dw)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy().astype(np.float64)
    ref, _ = oracle(w)
    em = E.emulate(w)
    em_max = np.abs(em - ref).max()
    gpu_max = np.abs(o - ref).max()
    print(f"sharpened: gpu max {gpu_max:.3e} mean {np.abs(o - ref).mean():.3e}; emulated max {em_max:.3e} "
          f"mean {np.abs(em - ref).mean():.3e}; gpu vs emulation max {np.abs(o - em).max():.3e} "
          f"mean {np.abs(o - em).mean():.3e}", flush=True)
    assert gpu_max <= 1.5 * em_max, (gpu_max, em_max)
    worst = np.inf
    for i in range(len(w.chunks)):
        r = int(np.searchsorted(w.chunk_start, i, side="right")) - 1
        rows = slice(int(w.q_start[r]), int(w.q_start[r + 1]))
        d0 = np.abs(o[rows] - em[rows]).mean()
        for d in (-1, 1):
            w2 = W.Workload(**{**w.__dict__})
            w2.chunks = w.chunks.copy()
            w2.chunks["pos_offset"][i] += d
            d1 = np.abs(o[rows] - E.emulate(w2)[rows]).mean()
            worst = min(worst, d1 / max(d0, 1e-12))
            assert d1 > 10 * d0, (i, d, d0, d1)
    print(f"sharpened: worst shift margin against the emulation {worst:.1f}x", flush=True)


def test_inv_freq_table_variant():
    w = W.rag_prefill(seed=81, batch=2, hq=8, hkv=2, d=128, prefix_len=8, n_chunks=2, chunk_len=100, pool_chunks=3,
                      q_len=12)
    # a scaled table (every frequency divided by 4, NTK-like) passed explicitly
    theta = (np.power(5.0e5, -2.0 * np.arange(64) / 128) / 4.0).astype(np.float32)
    dw = ops.upload(w)
    cfg = ops.config_of(w, inv_freq=torch.tensor(theta, device="cuda"))
    out, lse = ops.run_lazy(dw, cfg)
    torch.cuda.synchronize()
    ref_o, ref_l = O.lazy_attention(w.q, w.q_start, w.q_pos0, w.pool, w.pool, w.chunks, w.chunk_start, 8, 2, 128,
                                    w.rope_base, True, inv_freq=theta.astype(np.float64))
    assert_close(out, lse, ref_o, ref_l, tag="inv_freq")


# Full sizes, default launch configuration (the one the benchmark times); the oracle checks sampled requests.
FULL = {
    "rag_prefill": (lambda: W.rag_prefill(seed=1), list(range(8))),
    "icl_decode_step0": (lambda: W.icl_decode_step(W.icl_prefill(seed=3), 0), list(range(4))),
    "icl_decode_step127": (lambda: W.icl_decode_step(W.icl_prefill(seed=3), 127), list(range(4))),
    "rag_decode": (lambda: W.rag_decode(seed=2), [0, 37, 63]),
    "icl_prefill": (lambda: W.icl_prefill(seed=3), [2]),
    "varlen_rag": (lambda: W.varlen_rag(seed=4), [0, 9, 15]),
}


def _storage_ordered(w):
    return dataclasses.replace(w, chunks=ops.storage_order(w.chunks, w.chunk_start))


# The benchmark's storage-order legs at full size: the same records, each request's table in storage order.
FULL_STORAGE_ORDER = {
    "icl_decode_step64": (lambda: _storage_ordered(W.icl_decode_step(W.icl_prefill(seed=3), 64)), list(range(4))),
    "rag_decode": (lambda: _storage_ordered(W.rag_decode(seed=2)), [0, 37, 63]),
}


@pytest.mark.parametrize("name", list(FULL))
def test_full_size_sampled(name):
    make, reqs = FULL[name]
    w = make()
    print(f"{name}: batch={w.batch} total_q={w.total_q} max_kv={w.max_kv_len} meta={w.meta}", flush=True)
    run_and_check(w, "full " + name, requests=reqs)


@pytest.mark.parametrize("name", list(FULL_STORAGE_ORDER))
def test_full_size_storage_order_sampled(name):
    make, reqs = FULL_STORAGE_ORDER[name]
    run_and_check(make(), "full storage order " + name, requests=reqs)


# --------------------------------------------------------------------------------------------------------------
# Local-position key stores (LAZY_KEYS_LOCAL): the same random pools, read as keys already encoded at their local
# index j; the oracle applies the one rotation by pos_offset (its pins: test_oracle.py, local-store section).
LOCAL = dict(key_positions=ops.KEYS_LOCAL)


@pytest.mark.parametrize("name", ["rag_d128_g4", "rag_d64_g2_split3", "rag_d128_g1_split1", "varlen_g7",
                                  "varlen_g7_b8", "icl_small", "icl_small_split1"])
def test_local_key_store_prefill_matches_oracle(name):
    fn, kw, ckw = PREFILL_CASES[name]
    run_and_check(fn(**kw), "local " + name, {**ckw, **LOCAL})


@pytest.mark.parametrize("name", list(DECODE_CASES))
def test_local_key_store_decode_matches_oracle(name):
    kw, ckw = DECODE_CASES[name]
    run_and_check(W.rag_decode(**kw), "local decode " + name, {**ckw, **LOCAL})


def test_local_key_store_decode_many_short_records():
    """Decode re-rotates the query at every record change: 40 records of 1..70 keys (partial tiles, records shorter
    than a tile, waves that cross several records per tile step), non-causal as well."""
    rng = np.random.default_rng(91)
    reqs = []
    for r in range(3):
        pos, ch = 0, []
        for i in range(40):
            n = int(rng.integers(1, 71))
            ch.append((n, pos + int(rng.integers(0, 5))))
            pos = ch[-1][1] + n
        reqs.append(dict(chunks=ch, q_len=1, q_pos0=pos + 3))
    w = W.custom(92, 8, 2, 128, 5e5, reqs, kind="decode")
    run_and_check(w, "local decode short records", LOCAL)
    w.causal = False
    run_and_check(w, "local decode short records non-causal", LOCAL)


def test_local_lazy_prefill_equals_materialize_then_attend_bitwise():
    w = W.rag_prefill(seed=93, batch=3, hq=8, hkv=2, d=128, prefix_len=30, n_chunks=3, chunk_len=150, pool_chunks=5,
                      q_len=70)
    dw = ops.upload(w)
    cfg = ops.config_of(w, **LOCAL)
    out_l, lse_l = ops.run_lazy(dw, cfg)
    (out_m, lse_m), _ = ops.run_materialized(dw, cfg)
    torch.cuda.synchronize()
    assert torch.equal(out_l.view(torch.int16), out_m.view(torch.int16))
    assert torch.equal(lse_l, lse_m)


def test_local_materialized_keys_match_oracle():
    w = W.rag_prefill(seed=94, batch=2, hq=4, hkv=2, d=128, prefix_len=10, n_chunks=2, chunk_len=77, pool_chunks=3,
                      q_len=5)
    dw = ops.upload(w)
    cfg = ops.config_of(w, **LOCAL)
    total = int(w.chunks["len"].astype(np.int64).sum())
    k_out, ch_out = ops.materialize_k(cfg, dw.pool, dw.chunks, int(w.chunks["len"].max()), total)
    torch.cuda.synchronize()
    recs = ops.chunks_from_tensor(ch_out)
    ref = O.materialize_k(w.pool, w.chunks, w.chunk_start, 2, 128, w.rope_base, key_positions="local")
    got = k_out.float().cpu().numpy()
    for r in range(w.batch):
        start = 0
        for i in range(int(w.chunk_start[r]), int(w.chunk_start[r + 1])):
            n = int(recs[i]["len"])
            blk = got[int(recs[i]["k_offset"]): int(recs[i]["k_offset"]) + 2 * n * 128].reshape(2, n, 128)
            np.testing.assert_allclose(blk, ref[r][:, start:start + n], rtol=2 ** -8, atol=1e-5)
            start += n


def test_local_key_store_position_discrimination():
    """As test_position_discrimination, for the local-position convention (prefill and decode)."""
    reqs = DISCRIMINATION_REQS
    w = W.custom(95, 4, 2, 128, 1e4, reqs)
    for kind in ("prefill", "decode"):
        if kind == "decode":
            w = W.custom(96, 4, 2, 128, 1e4, [dict(chunks=c["chunks"], q_len=1, q_pos0=c["q_pos0"] + 3)
                                               for c in reqs], kind="decode")
        dw = ops.upload(w)
        out, lse = ops.run_lazy(dw, ops.config_of(w, **LOCAL))
        torch.cuda.synchronize()
        o = out.float().cpu().numpy()
        ref, ref_l = oracle(w, key_positions="local")
        assert_close(out, lse, ref, ref_l, tag=f"local discrimination workload {kind}")
        for i in range(len(w.chunks)):
            r = int(np.searchsorted(w.chunk_start, i, side="right")) - 1
            rows = slice(int(w.q_start[r]), int(w.q_start[r + 1]))
            e0 = np.abs(o[rows] - ref[rows]).mean()
            for d in (-1, 1):
                w2 = W.Workload(**{**w.__dict__})
                w2.chunks = w.chunks.copy()
                w2.chunks["pos_offset"][i] += d
                e1 = np.abs(o[rows] - oracle(w2, key_positions="local")[0][rows]).mean()
                assert e1 > 8 * e0, (kind, i, d, e0, e1)


# --------------------------------------------------------------------------------------------------------------
# Chunk-major shared decode: a host plan groups records that read the same stored keys; every group's keys are read
# once for all of its users.  Same results as the per-request decode (the oracle decides).
def run_shared_and_check(w, tag, cfg_kw=None, step=0):
    cfg = ops.config_of(w, **(cfg_kw or {}))
    plan = ops.shared_decode_plan(cfg, w.chunks, w.chunk_start, step)
    dw = ops.upload(w)
    dp = ops.upload_plan(plan)
    lse = torch.empty((w.batch, w.num_q_heads), dtype=torch.float32, device="cuda")
    out, _ = ops.decode_shared(cfg, dw.q, dw.q_pos0, dw.pool, dw.pool, dp, lse=lse)
    torch.cuda.synchronize()
    okw = {"key_positions": "local"} if (cfg_kw or {}).get("key_positions") == ops.KEYS_LOCAL else {}
    if (cfg_kw or {}).get("rope_style") == ops.ROPE_INTERLEAVED:
        okw["pairing"] = "interleaved"
    if (cfg_kw or {}).get("rope_style") == ops.ALIBI:
        okw["pairing"] = "alibi"
    ref_o, ref_l = oracle(w, **okw)
    print(f"{tag}: {plan.items.size} items for {len(w.chunks)} records, max slots {plan.max_slots}", flush=True)
    assert_close(out, lse, ref_o, ref_l, tag=tag)
    return plan


SHARED_CASES = {
    # name: (rag_decode kwargs, cfg kwargs, max keys per item)
    "g4_shared": (dict(seed=101, batch=6, hq=8, hkv=2, d=128, n_chunks=4, chunk_len=300, pool_chunks=5, tail_len=9,
                       tail_cap=16), {}, 0),
    "g4_shared_split100": (dict(seed=102, batch=6, hq=8, hkv=2, d=128, n_chunks=4, chunk_len=300, pool_chunks=5,
                                tail_len=9, tail_cap=16), {}, 100),
    "g7_d64_split37": (dict(seed=103, batch=5, hq=14, hkv=2, d=64, n_chunks=3, chunk_len=150, pool_chunks=4,
                            tail_len=33, tail_cap=40), {}, 37),
    "mha_g1": (dict(seed=104, batch=20, hq=4, hkv=4, d=128, n_chunks=2, chunk_len=257, pool_chunks=3, tail_len=2,
                    tail_cap=2), {}, 0),
    "g16_one_user_per_item": (dict(seed=105, batch=3, hq=32, hkv=2, d=128, n_chunks=2, chunk_len=90,
                                   pool_chunks=2, tail_len=5, tail_cap=8), {}, 64),
}


@pytest.mark.parametrize("local", [False, True])
@pytest.mark.parametrize("name", list(SHARED_CASES))
def test_shared_decode_matches_oracle(name, local):
    kw, ckw, step = SHARED_CASES[name]
    ckw = {**ckw, **(LOCAL if local else {})}
    plan = run_shared_and_check(W.rag_decode(**kw), f"shared {name} {'local' if local else 'nope'}", ckw, step)
    if name == "g4_shared":
        assert plan.items.size < sum(1 for _ in W.rag_decode(**kw).chunks)  # chunks really are shared


def test_shared_decode_edge_cases():
    """A request without records (out = 0, lse = -inf), one whose only chunk lies after the query (causal: nothing
    visible), records shorter than a tile, the same chunk twice in one request at different offsets, non-causal."""
    reqs = [
        dict(chunks=[("a", 70, 0), ("b", 5, 70), ("a", 70, 200)], q_len=1, q_pos0=300),
        dict(chunks=[], q_len=1, q_pos0=10),
        dict(chunks=[("b", 5, 50)], q_len=1, q_pos0=20),
        dict(chunks=[("a", 70, 1000), (1, 1070), ("b", 5, 5)], q_len=1, q_pos0=1070),
    ]
    w = W.custom(106, 8, 2, 128, 1e4, reqs, kind="decode", slack_fill=np.nan)
    for local in (False, True):
        run_shared_and_check(w, f"shared edge {local}", LOCAL if local else {})
    w.causal = False
    run_shared_and_check(w, "shared edge non-causal")


@pytest.mark.parametrize("paged", [False, True])
def test_shared_decode_full_size_sampled(paged):
    """The benchmark's decode batch (64 requests, chunks shared ~4x) through the shared path, sampled requests; also
    over the benchmark's paged store (64-token blocks), read in block runs."""
    w = W.rag_decode(seed=2)
    if paged:
        w = W.paginate(w, 64, seed=7)
    cfg = ops.config_of(w)
    plan = ops.shared_decode_plan(cfg, w.chunks, w.chunk_start)
    if paged:
        assert plan.items["num_ranges"].max() == 16 and plan.items.size == 424
    dw = ops.upload(w)
    out, _ = ops.decode_shared(cfg, dw.q, dw.q_pos0, dw.pool, dw.pool, ops.upload_plan(plan))
    torch.cuda.synchronize()
    ref_o, ref_l = oracle(w, requests=[0, 31, 63])
    rows = rows_of(w, [0, 31, 63])
    assert_close(out, None, ref_o, ref_l, rows, tag=f"shared full rag_decode {'paged64' if paged else ''}")


def _long_tables(seed, kind, n_records):
    """Requests of many short records (1..12 keys, contiguous positions): the tile walk counts tiles 256 records at a
    time and finds a split's first record 64 records at a time, so tables longer than 256 records take the paths
    past the first block."""
    rng = np.random.default_rng(seed)
    reqs = []
    for n in n_records:
        lens = rng.integers(1, 13, size=n)
        pos = np.concatenate([[0], np.cumsum(lens)[:-1]])
        q_len = 1 if kind == "decode" else 5
        reqs.append(dict(chunks=[(int(a), int(b)) for a, b in zip(lens, pos)], q_len=q_len,
                         q_pos0=int(pos[-1] + lens[-1]) - (q_len - 1 if kind == "decode" else 0)))
    return W.custom(seed, 8, 2, 128, 1e4, reqs, kind=kind)


@pytest.mark.parametrize("kind", ["prefill", "decode"])
@pytest.mark.parametrize("splits", [0, 5])
def test_long_chunk_tables(kind, splits):
    w = _long_tables(140 + splits, kind, [300, 700, 64])
    ckw = dict(num_splits=splits) if splits else {}
    run_and_check(w, f"{kind} long tables splits={splits}", ckw)
    run_and_check(w, f"{kind} long tables splits={splits} local", {**ckw, **LOCAL})


# --------------------------------------------------------------------------------------------------------------
# Paged (block-granular) stores: each chunk's K/V in fixed-size blocks scattered over the pool, one record per
# block.  The kernels see ordinary records (tiles never straddle a record); block sizes below a tile exercise the
# partial-tile paths.
@pytest.mark.parametrize("bt", [16, 64])
@pytest.mark.parametrize("local", [False, True])
def test_paged_prefill_matches_oracle(bt, local):
    w = W.paginate(W.rag_prefill(seed=111, batch=3, hq=8, hkv=2, d=128, prefix_len=40, n_chunks=3, chunk_len=150,
                                 pool_chunks=5, q_len=37), bt, seed=bt)
    run_and_check(w, f"paged{bt} prefill {'local' if local else 'nope'}", LOCAL if local else {})


@pytest.mark.parametrize("bt", [16, 32, 96])
def test_paged_decode_matches_oracle_per_request_and_shared(bt):
    w = W.paginate(W.rag_decode(seed=112, batch=6, hq=8, hkv=2, d=128, n_chunks=4, chunk_len=200, pool_chunks=5,
                                tail_len=9, tail_cap=32), bt, seed=bt)
    for local in (False, True):
        ckw = LOCAL if local else {}
        run_and_check(w, f"paged{bt} decode {'local' if local else 'nope'}", ckw)
        run_shared_and_check(w, f"paged{bt} shared decode {'local' if local else 'nope'}", ckw)


@pytest.mark.parametrize("mode", ["nope", "interleaved", "alibi", "prerotated"])
@pytest.mark.parametrize("bt,step", [(64, 0), (32, 100), (64, 160), (128, 0)])
def test_shared_decode_multi_range_runs(bt, step, mode):
    """Paged stores read in runs of blocks (items of several ranges): tiles cross range boundaries at multiples of
    32 keys, runs are capped by the item size, and the last range of a run is partial.  G = 4 and G = 7 (d = 64)."""
    for kw in (dict(seed=121, batch=6, hq=8, hkv=2, d=128, n_chunks=4, chunk_len=250, pool_chunks=5, tail_len=41,
                    tail_cap=64),
               dict(seed=122, batch=4, hq=14, hkv=2, d=64, n_chunks=3, chunk_len=333, pool_chunks=4, tail_len=3,
                    tail_cap=40)):
        w = W.paginate(W.rag_decode(**kw), bt, seed=bt + step)
        cfg = {"nope": {}, "interleaved": IL, "alibi": ALIBI, "prerotated": {}}[mode]
        if mode == "prerotated":
            check_prerotated(w, f"runs bt{bt} step{step} prerotated", {}, shared=True)
            continue
        plan = run_shared_and_check(w, f"runs bt{bt} step{step} {mode} d{kw['d']}", cfg, step)
        assert plan.items["num_ranges"].max() > 1


# --------------------------------------------------------------------------------------------------------------
# Interleaved RoPE pairing (pairs (2t, 2t+1), Sec. 3.5): every kernel, both key conventions.
IL = dict(rope_style=ops.ROPE_INTERLEAVED)


@pytest.mark.parametrize("local", [False, True])
@pytest.mark.parametrize("name", ["rag_d128_g4", "rag_d64_g2_split3", "varlen_g7"])
def test_interleaved_prefill_matches_oracle(name, local):
    fn, kw, ckw = PREFILL_CASES[name]
    run_and_check(fn(**kw), f"interleaved {name} {'local' if local else 'nope'}", {**ckw, **IL, **(LOCAL if local else {})})


@pytest.mark.parametrize("local", [False, True])
@pytest.mark.parametrize("name", ["d128_g4", "d64_g7_split5", "d128_g20_two_head_groups"])
def test_interleaved_decode_matches_oracle(name, local):
    kw, ckw = DECODE_CASES[name]
    w = W.rag_decode(**kw)
    ck = {**ckw, **IL, **(LOCAL if local else {})}
    run_and_check(w, f"interleaved decode {name} {'local' if local else 'nope'}", ck)
    if name != "d128_g20_two_head_groups":  # G = 20 does not fit the shared decode's 16 columns
        run_shared_and_check(w, f"interleaved shared decode {name} {'local' if local else 'nope'}",
                             {k: v for k, v in ck.items() if k != "num_splits"})


@pytest.mark.parametrize("local", [False, True])
def test_interleaved_lazy_prefill_equals_materialize_then_attend_bitwise(local):
    w = W.rag_prefill(seed=121, batch=3, hq=8, hkv=2, d=128, prefix_len=30, n_chunks=3, chunk_len=150,
                      pool_chunks=5, q_len=70)
    dw = ops.upload(w)
    cfg = ops.config_of(w, **IL, **(LOCAL if local else {}))
    out_l, lse_l = ops.run_lazy(dw, cfg)
    (out_m, lse_m), (k_out, ch_out) = ops.run_materialized(dw, cfg)
    torch.cuda.synchronize()
    assert torch.equal(out_l.view(torch.int16), out_m.view(torch.int16))
    assert torch.equal(lse_l, lse_m)
    # the copy holds the interleaved-encoded keys
    recs = ops.chunks_from_tensor(ch_out)
    ref = O.materialize_k(w.pool, w.chunks, w.chunk_start, 2, 128, w.rope_base,
                          key_positions="local" if local else "nope", pairing="interleaved")
    got = k_out.float().cpu().numpy()
    start = 0
    for i in range(int(w.chunk_start[0]), int(w.chunk_start[1])):
        n = int(recs[i]["len"])
        blk = got[int(recs[i]["k_offset"]): int(recs[i]["k_offset"]) + 2 * n * 128].reshape(2, n, 128)
        np.testing.assert_allclose(blk, ref[0][:, start:start + n], rtol=2 ** -8, atol=1e-5)
        start += n


# --------------------------------------------------------------------------------------------------------------
# ALiBi (score-space positions, Sec. 3.5): no rotation, slope_h (k_pos - q_pos) added to the scaled scores.
ALIBI = dict(rope_style=ops.ALIBI)


@pytest.mark.parametrize("name", ["rag_d128_g4", "rag_d64_g2_split3", "varlen_g7"])
def test_alibi_prefill_matches_oracle(name):
    fn, kw, ckw = PREFILL_CASES[name]
    run_and_check(fn(**kw), f"alibi {name}", {**ckw, **ALIBI})


@pytest.mark.parametrize("name", ["d128_g4", "d64_g7_split5", "d128_g20_two_head_groups"])
def test_alibi_decode_matches_oracle(name):
    kw, ckw = DECODE_CASES[name]
    w = W.rag_decode(**kw)
    run_and_check(w, f"alibi decode {name}", {**ckw, **ALIBI})
    if name != "d128_g20_two_head_groups":
        run_shared_and_check(w, f"alibi shared decode {name}", ALIBI)


def test_alibi_slope_table_and_non_causal():
    w = W.rag_prefill(seed=131, batch=2, hq=8, hkv=2, d=128, prefix_len=20, n_chunks=2, chunk_len=90,
                      pool_chunks=3, q_len=30)
    slopes = np.linspace(0.5, 0.01, 8).astype(np.float32)
    dw = ops.upload(w)
    cfg = ops.config_of(w, rope_style=ops.ALIBI, inv_freq=torch.tensor(slopes, device="cuda"))
    for causal in (True, False):
        w.causal = causal
        cfg.causal = causal
        out, lse = ops.run_lazy(dw, cfg)
        torch.cuda.synchronize()
        ref_o, ref_l = oracle(w, pairing="alibi", inv_freq=slopes.astype(np.float64))
        assert_close(out, lse, ref_o, ref_l, tag=f"alibi table causal={causal}")


# --------------------------------------------------------------------------------------------------------------
# Pre-rotated queries (q_prerotated = 1): the caller passes R(q_pos) q, as the paper's prefill assumes.  The queries
# are rotated here by the oracle (fp64) and rounded to bf16; the result must match the oracle on the raw queries.
def with_prerotated_q(w, pairing="half"):
    if w.kind == "decode":
        pos = np.asarray(w.q_pos0, dtype=np.int64)
    else:
        pos = np.concatenate([int(w.q_pos0[r]) + np.arange(int(w.q_start[r + 1] - w.q_start[r]))
                              for r in range(w.batch)]).astype(np.int64)
    theta = O.rope_frequencies(w.head_dim, w.rope_base)
    q = O.rotate(np.transpose(w.q, (1, 0, 2)), pos, theta, pairing)  # [Hq, n, D]
    w2 = dataclasses.replace(w, q=W.bf16_round(np.transpose(q, (1, 0, 2)).astype(np.float32)))
    return w2


def check_prerotated(w, tag, ckw, shared=False):
    okw = {}
    if ckw.get("key_positions") == ops.KEYS_LOCAL:
        okw["key_positions"] = "local"
    pairing = "interleaved" if ckw.get("rope_style") == ops.ROPE_INTERLEAVED else "half"
    if pairing == "interleaved":
        okw["pairing"] = "interleaved"
    w2 = with_prerotated_q(w, pairing)
    cfg = ops.config_of(w, q_prerotated=True, **ckw)
    dw = ops.upload(w2)
    if shared:
        dp = ops.upload_plan(ops.shared_decode_plan(cfg, w.chunks, w.chunk_start, 0))
        lse = torch.empty((w.batch, w.num_q_heads), dtype=torch.float32, device="cuda")
        out, _ = ops.decode_shared(cfg, dw.q, dw.q_pos0, dw.pool, dw.pool, dp, lse=lse)
    else:
        out, lse = ops.run_lazy(dw, cfg)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle(w, **okw)
    assert_close(out, lse, ref_o, ref_l, tag=tag)
    # the flag really changes the computation: without it the pre-rotated queries are rotated twice
    if not shared:
        out2, _ = ops.run_lazy(dw, ops.config_of(w, **ckw))
        torch.cuda.synchronize()
        assert np.abs(out2.float().cpu().numpy() - ref_o).max() > 5 * MAX_ABS, tag


PREROT = {"nope": {}, "local": LOCAL, "interleaved": IL, "interleaved_local": {**IL, **LOCAL}}


@pytest.mark.parametrize("mode", list(PREROT))
@pytest.mark.parametrize("name", ["rag_d128_g4", "rag_d64_g2_split3", "varlen_g7"])
def test_prerotated_queries_prefill(name, mode):
    fn, kw, ckw = PREFILL_CASES[name]
    check_prerotated(fn(**kw), f"prerotated prefill {name} {mode}", {**ckw, **PREROT[mode]})


@pytest.mark.parametrize("mode", list(PREROT))
@pytest.mark.parametrize("name", ["d128_g4", "d64_g7_split5", "d128_g20_two_head_groups"])
def test_prerotated_queries_decode(name, mode):
    kw, ckw = DECODE_CASES[name]
    check_prerotated(W.rag_decode(**kw), f"prerotated decode {name} {mode}", {**ckw, **PREROT[mode]})


@pytest.mark.parametrize("mode", ["nope", "local", "interleaved"])
@pytest.mark.parametrize("name", ["g4_shared", "g7_d64_split37"])
def test_prerotated_queries_shared_decode(name, mode):
    kw, _, _ = SHARED_CASES[name]
    check_prerotated(W.rag_decode(**kw), f"prerotated shared {name} {mode}", PREROT[mode], shared=True)


def test_prerotated_queries_plain_attention_equals_lazy_bitwise():
    """The materialise-then-attend baseline honours the flag too: bit-identical to the lazy kernel."""
    fn, kw, ckw = PREFILL_CASES["rag_d128_g4"]
    w = fn(**kw)
    w2 = with_prerotated_q(w)
    cfg = ops.config_of(w, q_prerotated=True, **ckw)
    dw = ops.upload(w2)
    lazy, lse_l = ops.run_lazy(dw, cfg)
    (plain, lse_m), _ = ops.run_materialized(dw, cfg)
    torch.cuda.synchronize()
    assert torch.equal(lazy.view(torch.int16), plain.view(torch.int16))
    assert torch.equal(lse_l, lse_m)


# --------------------------------------------------------------------------------------------------------------
# Decode tables whose records are not in position order.  Positions, not table indices, decide visibility, so a
# record that lies after the query may precede visible ones; each decode wave owns every fourth tile of its split
# and must process each visible tile exactly once (the tile walk's CPU model: tests/test_tile_walk.py).
def _out_of_order_decode(seed):
    reqs = [
        dict(chunks=[(70, 1000), (500, 0), (1, 600)], q_len=1, q_pos0=600),
        dict(chunks=[(64, 0), (100, 900), (512, 64), (1, 700)], q_len=1, q_pos0=700),
        dict(chunks=[(300, 2000), (33, 5000), (200, 100), (150, 300), (1, 450)], q_len=1, q_pos0=450),
        # a record straddling the query (keys after it masked) ahead of visible ones, and tiles of one record on
        # both sides of the query
        dict(chunks=[(200, 250), (40, 5000), (256, 0), (1, 330)], q_len=1, q_pos0=330),
    ]
    return W.custom(seed, 8, 2, 128, 1e4, reqs, kind="decode")


OOO_MODES = {"nope": {}, "local": LOCAL, "interleaved": IL, "alibi": ALIBI}


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("mode", list(OOO_MODES))
def test_decode_records_out_of_position_order(mode, splits):
    w = _out_of_order_decode(151)
    ckw = {**OOO_MODES[mode], "num_splits": splits}
    dw, out, lse = run_and_check(w, f"decode out-of-order {mode} splits={splits}", ckw)
    if mode == "alibi":
        return  # nothing to materialise
    (out_m, lse_m), _ = ops.run_materialized(dw, ops.config_of(w, **ckw))
    torch.cuda.synchronize()
    ref_o, ref_l = oracle(w, **oracle_kw(ckw))
    assert_close(out_m, lse_m, ref_o, ref_l, tag=f"plain decode out-of-order {mode} splits={splits}")
    if mode == "nope":  # lazy and materialise-then-attend round the rotated keys identically
        assert torch.equal(out.view(torch.int16), out_m.view(torch.int16))


# --------------------------------------------------------------------------------------------------------------
# Positions near LAZY_MAX_POS = 2^24 (the appendix on long-context stability evaluates 128K positions; the ABI
# allows up to 2^24): angles are reduced in fp64 before the fp32 sine / cosine.
BIG = (1 << 24) - 10_000


@pytest.mark.parametrize("mode", ["nope", "local", "interleaved", "alibi"])
def test_positions_near_max_pos(mode):
    ckw = OOO_MODES[mode]
    reqs = [dict(chunks=[(300, BIG), (200, BIG + 300), (40, BIG + 500)], q_len=40, q_pos0=BIG + 500),
            dict(chunks=[(130, BIG + 7000), (64, 5), (2000, (1 << 24) - 2040), (40, (1 << 24) - 40)], q_len=40,
                 q_pos0=(1 << 24) - 40)]
    for base in (1e4, 5e5):
        w = W.custom(161, 8, 2, 128, base, reqs)
        run_and_check(w, f"prefill near 2^24 {mode} base {base:g}", ckw)
        run_and_check(w, f"prefill near 2^24 {mode} base {base:g} split 3", {**ckw, "num_splits": 3})
        wd = W.custom(162, 8, 2, 128, base, [dict(chunks=r["chunks"], q_len=1, q_pos0=r["q_pos0"] + 39)
                                             for r in reqs], kind="decode")
        run_and_check(wd, f"decode near 2^24 {mode} base {base:g}", ckw)
        run_shared_and_check(wd, f"shared decode near 2^24 {mode} base {base:g}", ckw)


# --------------------------------------------------------------------------------------------------------------
# The eight-wave prefill (256 packed rows: 64 tokens x G = 4) runs its upper four waves one tile ahead on the
# loader side (they store their share of the next tile at the start of each interval).  Splits holding one, two or
# three tiles start and end that pipeline in every way it can: no next tile, a next tile but none after it, and a
# first tile that the causal rule skips (a record placed after the query ahead of visible ones).
PHASE_REQS = [dict(chunks=[(64, 0)], q_len=64, q_pos0=64),
              dict(chunks=[(10, 0), (64, 100), (40, 500)], q_len=64, q_pos0=600),
              dict(chunks=[(64, 5000), (130, 0), (1, 300)], q_len=64, q_pos0=400)]


@pytest.mark.parametrize("mode", ["nope", "local", "interleaved", "alibi"])
def test_eight_wave_prefill_short_splits(mode):
    ckw = OOO_MODES[mode]
    w = W.custom(171, 8, 2, 128, 1e4, PHASE_REQS)
    assert w.max_q_len * (w.num_q_heads // w.num_kv_heads) >= 256  # the eight-wave kernel
    for splits in (1, 2, 3, 4, 6):
        run_and_check(w, f"eight-wave prefill {mode} splits={splits}", {**ckw, "num_splits": splits})


# --------------------------------------------------------------------------------------------------------------
# Chunk tables in storage order (lazy_chunk_table_storage_order): the same records, each request's sorted by
# k_offset.  Positions decide the attention, so the results match the oracle of the position-ordered table, and the
# lazy path still equals materialise-then-attend over the reordered table bit for bit.
@pytest.mark.parametrize("kind,ckw", [("decode", {}), ("decode", dict(num_splits=3)),
                                      ("decode", dict(key_positions=ops.KEYS_LOCAL)), ("prefill", {}),
                                      ("prefill", dict(num_splits=2)), ("paged_decode", dict(num_splits=2)),
                                      ("g7_decode", dict(cache_hint=ops.CACHE_STREAM))])
def test_storage_ordered_tables_match_oracle(kind, ckw):
    if kind == "paged_decode":  # 32-token blocks scattered over the pool: storage order interleaves chunks
        w = W.paginate(W.rag_decode(seed=173, batch=3, hq=8, hkv=2, n_chunks=3, chunk_len=150, pool_chunks=4,
                                    tail_len=5, tail_cap=8), 32, seed=3)
    elif kind == "g7_decode":
        w = W.rag_decode(seed=174, batch=4, hq=28, hkv=4, n_chunks=4, chunk_len=120, pool_chunks=6, tail_len=7,
                         tail_cap=12)
    else:
        w = W.icl_prefill(seed=171, batch=3, hq=8, hkv=2, d=128, n_chunks=6, chunk_len=96, q_len=40,
                          decode_steps=4)
        if kind == "decode":
            w = W.icl_decode_step(w, 2, seed=172)
    ws = dataclasses.replace(w, chunks=ops.storage_order(w.chunks, w.chunk_start))
    assert not np.array_equal(ws.chunks.view(np.uint8), w.chunks.view(np.uint8))  # the order did change
    dw, out, lse = run_and_check(ws, f"storage order {kind} {ckw}", ckw)
    ref_o, ref_l = oracle(w, **oracle_kw(ckw))  # the position-ordered table
    assert_close(out, lse, ref_o, ref_l, tag=f"storage order vs position-order oracle {kind} {ckw}")
    if not ckw.get("key_positions"):
        (out_m, lse_m), _ = ops.run_materialized(dw, ops.config_of(ws, **ckw))
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), out_m.view(torch.int16))


@pytest.mark.parametrize("paged", [False, True])
def test_shared_decode_on_storage_ordered_tables(paged):
    """The shared decode's planner groups records by the stored keys they read, whatever the table order; on a paged
    store in storage order the blocks of a chunk no longer follow each other in a request's table, so the planner
    keeps them as separate items, and the results stay those of the position-ordered tables."""
    w = W.rag_decode(seed=175, batch=5, hq=8, hkv=2, n_chunks=3, chunk_len=160, pool_chunks=4, tail_len=6, tail_cap=8)
    if paged:
        w = W.paginate(w, 32, seed=4)
    ws = _storage_ordered(w)
    plan = run_shared_and_check(ws, f"shared decode, storage order, paged={paged}")
    base = ops.shared_decode_plan(ops.config_of(w), w.chunks, w.chunk_start)
    assert plan.read_keys() == base.read_keys()  # every stored key still read once per step
    assert plan.items.size == base.items.size if not paged else plan.items.size > base.items.size
