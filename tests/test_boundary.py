"""CPU tests of the C ABI boundary: exported symbols, struct layouts, host-side table validation, scalar argument
checks and workspace sizing.  Nothing here launches a kernel."""
import ctypes
import os
import re
import shutil
import subprocess

import numpy as np
import pytest

from paper_2606_04302_amd import build as B
from paper_2606_04302_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lazy_attn.h")


@pytest.fixture(scope="module")
def ops():
    from paper_2606_04302_amd import ops as O

    if not os.path.exists(O.LIB_PATH):
        B.build()
    O.lib()
    return O


def declared_functions():
    text = open(HEADER).read()
    return re.findall(r"LAZY_API\s+[\w\s\*]+?\b(lazy_\w+)\s*\(", text)


def test_library_exports_every_declared_symbol(ops):
    names = declared_functions()
    assert len(names) >= 11, names
    lib = ctypes.CDLL(ops.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", ops.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (\w+)", out))
    assert set(names) <= exported
    # only the C ABI is exported
    assert {n for n in exported if not n.startswith("_")} == set(names)
    assert set(names) == set(ops.SIGNATURES)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_struct_layout_matches_header(tmp_path, ops):
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stdio.h>\n#include <stddef.h>\n#include "lazy_attn.h"\n'
        "int main(void){"
        'printf("%zu %zu %zu %zu %zu %zu %zu\\n", sizeof(lazy_chunk_t), offsetof(lazy_chunk_t, v_offset),'
        " offsetof(lazy_chunk_t, len), offsetof(lazy_chunk_t, pos_offset), offsetof(lazy_chunk_t, k_stride),"
        " offsetof(lazy_chunk_t, v_stride), sizeof(lazy_attn_params_t));"
        'printf("%zu %zu %zu %zu\\n", offsetof(lazy_attn_params_t, rope_base), offsetof(lazy_attn_params_t, inv_freq),'
        " offsetof(lazy_attn_params_t, num_splits), offsetof(lazy_attn_params_t, key_positions));"
        'printf("%zu %zu %zu\\n", offsetof(lazy_attn_params_t, rope_style), offsetof(lazy_attn_params_t, q_prerotated),'
        " offsetof(lazy_attn_params_t, cache_hint));"
        "return 0;}"
    )
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    a, b, e = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")[:3]
    c = [int(x) for x in a.split()]
    p = [int(x) for x in b.split()]
    LC, LP = ops.LazyChunk, ops.LazyAttnParams
    assert [int(x) for x in e.split()] == [LP.rope_style.offset, LP.q_prerotated.offset, LP.cache_hint.offset]
    assert c == [ctypes.sizeof(LC), LC.v_offset.offset, LC.len.offset, LC.pos_offset.offset, LC.k_stride.offset,
                 LC.v_stride.offset, ctypes.sizeof(LP)]
    assert p == [LP.rope_base.offset, LP.inv_freq.offset, LP.num_splits.offset, LP.key_positions.offset]
    dt = W.CHUNK_DTYPE
    assert [dt.fields[n][1] for n in ("k_offset", "v_offset", "len", "pos_offset", "k_stride", "v_stride")] == [
        0, c[1], c[2], c[3], c[4], c[5]]


def _valid(w, ops, **kw):
    cfg = ops.config_of(w, **kw)
    return ops.validate(cfg, w.q_start if w.kind == "prefill" else None, w.q_pos0, w.chunks, w.chunk_start,
                        w.pool.size, w.pool.size)


def test_validate_accepts_generated_workloads(ops):
    for w in (W.tiny_rag_prefill(), W.rag_prefill(batch=2, n_chunks=3, chunk_len=64, pool_chunks=4, q_len=8, hq=8,
                                                     hkv=2),
              W.rag_decode(batch=3, n_chunks=2, chunk_len=70, pool_chunks=3, hq=8, hkv=2),
              W.varlen_rag(batch=3, pool_chunks=6, len_hi=300, k_lo=2, k_hi=4, q_hi=40, hq=8, hkv=2)):
        code, bad, why = _valid(w, ops)
        assert code == ops.LAZY_OK, (w.name, bad, why)


def _w():
    return W.rag_prefill(seed=3, batch=2, hq=4, hkv=2, d=64, prefix_len=8, n_chunks=2, chunk_len=16, pool_chunks=3,
                         q_len=4)


@pytest.mark.parametrize("mutate,reason", [
    (lambda w: w.chunk_start.__setitem__(0, 1), "chunk_start[0]"),
    (lambda w: w.chunk_start.__setitem__(1, w.chunk_start[2] + 1), "non-decreasing"),
    (lambda w: w.chunks["len"].__setitem__(1, 0), "len"),
    (lambda w: w.chunks["pos_offset"].__setitem__(0, -1), "pos_offset"),
    (lambda w: w.chunks["pos_offset"].__setitem__(0, (1 << 24) - 3), "LAZY_MAX_POS"),
    (lambda w: w.chunks["k_stride"].__setitem__(2, 1), "stride"),
    (lambda w: w.chunks["k_offset"].__setitem__(1, w.chunks["k_offset"][1] + 4), "multiples of 8"),
    (lambda w: w.chunks["k_offset"].__setitem__(1, w.pool.size - 8), "K range"),
    (lambda w: w.chunks["v_offset"].__setitem__(1, w.pool.size - 8), "V range"),
    (lambda w: w.q_start.__setitem__(0, 1), "q_start[0]"),
    (lambda w: w.q_pos0.__setitem__(1, -5), "query position"),
    (lambda w: w.chunks["pos_offset"].__setitem__(slice(0, 4), 10 ** 6), "sees no key"),
])
def test_validate_rejects_every_contract_violation(ops, mutate, reason):
    w = _w()
    assert _valid(w, ops)[0] == ops.LAZY_OK
    mutate(w)
    code, bad, why = _valid(w, ops)
    assert code == ops.LAZY_EDATA and reason in why, (code, bad, why)
    assert bad >= 0


def test_validate_non_causal_request_without_keys(ops):
    reqs = [dict(chunks=[(4, 0)], q_len=2, q_pos0=4), dict(chunks=[], q_len=3, q_pos0=0)]
    w = W.custom(1, 2, 1, 64, 1e4, reqs, causal=False)
    code, bad, why = _valid(w, ops)
    assert code == ops.LAZY_EDATA and bad == 1 and "no keys" in why


def test_scalar_argument_errors_return_before_any_launch(ops):
    L = ops.lib()
    P = ops.LazyAttnParams
    fake = ctypes.c_void_p(0x1000)

    def prefill(p, batch=1, total_q=4, max_q=4, max_kv=16, ws=None, ws_bytes=0, q=fake, out=fake):
        return L.lazy_attn_prefill(ctypes.byref(p) if p is not None else None, q, fake, fake, fake, fake, fake,
                                   fake, batch, total_q, max_q, max_kv, out, None, ws, ws_bytes, None)

    good = P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0)
    assert prefill(None) == ops.LAZY_EINVAL
    assert prefill(P(8, 3, 128, 1, 1e4, 0.0, None, 0, 0)) == ops.LAZY_EINVAL          # Hq % Hkv != 0
    assert prefill(P(8, 2, 96, 1, 1e4, 0.0, None, 0, 0)) == ops.LAZY_EUNSUPPORTED     # head_dim
    assert prefill(P(8, 2, 128, 2, 1e4, 0.0, None, 0, 0)) == ops.LAZY_EINVAL          # causal flag
    assert prefill(P(8, 2, 128, 1, -1.0, 0.0, None, 0, 0)) == ops.LAZY_EINVAL         # rope base
    assert prefill(P(8, 2, 128, 1, 1e4, -0.5, None, 0, 0)) == ops.LAZY_EINVAL         # softmax scale
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, -1, 0)) == ops.LAZY_EINVAL         # splits
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 7)) == ops.LAZY_EINVAL          # key convention
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, -1)) == ops.LAZY_EINVAL
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0, 3)) == ops.LAZY_EINVAL      # positional method
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 1, 2)) == ops.LAZY_EINVAL      # ALiBi with local keys
    L = ops.lib()
    alibi = P(8, 2, 128, 1, 0.0, 0.0, None, 0, 0, 2)                                  # rope_base unused
    assert L.lazy_plain_attn_prefill(ctypes.byref(alibi), *([1] * 7), 1, 1, 1, 1, 1, None, None, 0,
                                     None) == ops.LAZY_EUNSUPPORTED
    assert L.lazy_materialize_k(ctypes.byref(alibi), 1, 1, 1, 1, 1, 1, 1, None) == ops.LAZY_EUNSUPPORTED
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0, 0, 2)) == ops.LAZY_EINVAL   # q_prerotated is 0 or 1
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0, 0, -1)) == ops.LAZY_EINVAL
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0, 0, 1), batch=0) == ops.LAZY_OK
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0, 0, 0, 2)) == ops.LAZY_EINVAL  # cache hint is 0 or 1
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0, 0, 0, -1)) == ops.LAZY_EINVAL
    assert prefill(P(8, 2, 128, 1, 1e4, 0.0, None, 0, 0, 0, 0, 1), batch=0) == ops.LAZY_OK
    assert prefill(good, batch=-1) == ops.LAZY_EINVAL
    assert prefill(good, batch=0) == ops.LAZY_OK                                       # nothing to do
    assert prefill(good, total_q=0) == ops.LAZY_OK
    assert prefill(good, max_q=0) == ops.LAZY_EINVAL
    assert prefill(good, q=None) == ops.LAZY_EINVAL
    assert prefill(good, out=None) == ops.LAZY_EINVAL
    # a workload that needs a split workspace but gets none
    big = P(8, 2, 128, 1, 1e4, 0.0, None, 4, 0)
    assert prefill(big, max_kv=4096) == ops.LAZY_EWORKSPACE
    assert prefill(big, max_kv=4096, ws=ctypes.c_void_p(0x1004), ws_bytes=1 << 30) == ops.LAZY_EWORKSPACE  # misaligned
    # decode
    assert L.lazy_attn_decode(ctypes.byref(good), None, fake, fake, fake, fake, fake, 2, 100, fake, None, None, 0,
                              None) == ops.LAZY_EINVAL
    assert L.lazy_attn_decode(ctypes.byref(good), fake, fake, fake, fake, fake, fake, 0, 100, fake, None, None, 0,
                              None) == ops.LAZY_OK
    # decode without allocation: argument checks and the scratch limit come before any HIP call
    noalloc = lambda p, batch=2, max_kv=100: L.lazy_attn_decode_noalloc(
        ctypes.byref(p) if p is not None else None, fake, fake, fake, fake, fake, fake, batch, max_kv, fake, None, None)
    assert noalloc(None) == ops.LAZY_EINVAL
    assert noalloc(P(8, 2, 96, 1, 1e4, 0.0, None, 0, 0)) == ops.LAZY_EUNSUPPORTED
    assert noalloc(good, batch=-1) == ops.LAZY_EINVAL
    assert noalloc(good, batch=0) == ops.LAZY_OK
    many = P(32, 8, 128, 1, 5e5, 0.0, None, 64, 0)  # 64 splits x 64 x 32 rows x 260 B = 34 MB of partials
    assert noalloc(many, batch=64, max_kv=1 << 20) == ops.LAZY_EWORKSPACE
    # the default split count always fits the scratch array (about 1024 * min(G, 16) rows at most)
    for hq, hkv, d in ((32, 8, 128), (64, 4, 128), (16, 16, 64), (128, 4, 128)):
        cfg = ops.Config(hq, hkv, d, 1e4)
        for batch in (1, 2, 3, 5, 31, 64, 200):
            assert ops.decode_workspace_size(cfg, batch, 1 << 20) <= ops.NOALLOC_SCRATCH_BYTES, (hq, hkv, d, batch)
    # combine / materialize
    assert L.lazy_attn_combine(fake, fake, 0, 10, 128, fake, None, None) == ops.LAZY_EINVAL
    assert L.lazy_attn_combine(fake, fake, 2, 10, 80, fake, None, None) == ops.LAZY_EUNSUPPORTED
    assert L.lazy_attn_combine(fake, fake, 2, 0, 128, fake, None, None) == ops.LAZY_OK
    assert L.lazy_materialize_k(ctypes.byref(good), fake, fake, -1, 10, 10, fake, fake, None) == ops.LAZY_EINVAL
    assert L.lazy_materialize_k(ctypes.byref(good), fake, fake, 0, 10, 10, fake, fake, None) == ops.LAZY_OK


def test_workspace_size_matches_split_formula(ops):
    cfg = ops.Config(32, 8, 128, 5e5, num_splits=4)
    # per split and row: the bf16 normalised output (2 D bytes) and its fp32 log-sum-exp
    assert ops.prefill_workspace_size(cfg, 8, 512, 64, 5312) == 4 * 512 * 32 * (2 * 128 + 4)
    cfg1 = ops.Config(32, 8, 128, 5e5, num_splits=1)
    assert ops.prefill_workspace_size(cfg1, 8, 512, 64, 5312) == 0
    auto = ops.Config(32, 8, 128, 5e5)
    n = ops.prefill_workspace_size(auto, 8, 512, 64, 5312)
    assert n % (512 * 32 * (2 * 128 + 4)) == 0 and n == ops.prefill_workspace_size(auto, 8, 512, 64, 5312)
    assert ops.decode_workspace_size(ops.Config(32, 8, 128, 5e5, num_splits=3), 64, 16449) == 3 * 64 * 32 * (2 * 128 + 4)
    assert ops.decode_workspace_size(auto, 0, 100) == 0


def test_prefill_xcd_map_choice(ops):
    """The interleaved XCD map applies to ragged batches (mean query length under 3/4 of the maximum) whose
    batch x splits is a multiple of 8; the prefill parity case varlen_g7_b8 is built to take it."""
    w = W.varlen_rag(seed=30, batch=8, hq=28, hkv=4, d=128, pool_chunks=10, len_lo=40, len_hi=300, k_lo=2, k_hi=4,
                     q_lo=10, q_hi=90)
    cfg = ops.config_of(w)
    assert 4 * w.total_q < 3 * w.batch * w.max_q_len
    per_split = w.total_q * w.num_q_heads * (2 * w.head_dim + 4)
    n = ops.prefill_workspace_size(cfg, w.batch, w.total_q, w.max_q_len, w.max_kv_len)
    splits = max(1, n // per_split)
    assert n == (0 if splits == 1 else splits * per_split)
    assert (w.batch * splits) % 8 == 0 and splits >= 2
    # several query tiles per KV head (256-row tiles at head_dim 128) and a ragged tail
    assert w.max_q_len * (w.num_q_heads // w.num_kv_heads) > 256


def test_strerror_and_version(ops):
    assert ops.strerror(0) == "success"
    assert "workspace" in ops.strerror(-3)
    assert ops.strerror(12345) == "unknown error"
    assert ops.lib().lazy_attn_version() >= 100


def test_binding_rejects_host_tensors(ops):
    import torch

    cfg = ops.Config(2, 1, 64, 1e4)
    t = torch.zeros(4, 2, 64, dtype=torch.bfloat16)
    i = torch.zeros(2, dtype=torch.int32)
    with pytest.raises(ValueError):
        ops.prefill(cfg, t, i, i, t, t, torch.zeros(32, dtype=torch.uint8), i, 4, 4)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ missing")
def test_validator_under_address_and_ub_sanitizers(tmp_path):
    """Host validation code built with ASan/UBSan and driven through valid and invalid tables."""
    drv = tmp_path / "drv.cpp"
    drv.write_text(r'''
#include <cstdio>
#include <vector>
#include "lazy_attn.h"
int main() {
  lazy_attn_params_t p = {4, 2, 64, 1, 1e4f, 0.f, nullptr, 0, 0};
  std::vector<lazy_chunk_t> c = {{0, 2048, 16, 0, 16, 16}, {4096, 6144, 8, 16, 8, 8}, {8192, 10240, 4, 24, 4, 4}};
  std::vector<int> cs = {0, 2, 3}, qs = {0, 2, 4}, qp = {24, 24};
  int64_t bad; const char* why;
  int rc = lazy_attn_validate(&p, qs.data(), qp.data(), c.data(), cs.data(), 2, 1 << 16, 1 << 16, &bad, &why);
  if (rc != LAZY_OK) { printf("valid tables rejected: %s\n", why); return 1; }
  int fails = 0;
  for (int k = 0; k < 8; ++k) {
    std::vector<lazy_chunk_t> m = c; std::vector<int> mcs = cs, mqs = qs, mqp = qp;
    switch (k) {
      case 0: m[0].len = 0; break;
      case 1: m[1].pos_offset = -1; break;
      case 2: m[2].k_offset = 3; break;
      case 3: m[0].k_stride = 2; break;
      case 4: m[1].k_offset = (1 << 16) - 8; break;
      case 5: mcs[1] = 5; break;
      case 6: mqs[1] = -1; break;
      case 7: mqp[1] = -3; break;
    }
    rc = lazy_attn_validate(&p, mqs.data(), mqp.data(), m.data(), mcs.data(), 2, 1 << 16, 1 << 16, &bad, &why);
    if (rc != LAZY_EDATA) { printf("case %d not rejected (%d)\n", k, rc); ++fails; }
  }
  if (lazy_attn_validate(nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0, 0, nullptr, nullptr) != LAZY_EINVAL) ++fails;
  printf("sanitized validator ok=%d\n", fails == 0);
  return fails;
}
''')
    exe = tmp_path / "drv"
    subprocess.run(["g++", "-std=c++17", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-I",
                    os.path.join(ROOT, "include"), str(drv), os.path.join(B.CSRC, "lazy_attn_validate.cpp"), "-o",
                    str(exe)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "ok=1" in res.stdout


# ---------------------------------------------------------------------------------------------------------------
# Chunk-major shared decode: the host planner (CPU) and the plan record layouts.
# ---------------------------------------------------------------------------------------------------------------
@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_shared_plan_layout_matches_header(tmp_path, ops):
    src = tmp_path / "plan_layout.c"
    src.write_text(
        '#include <stdio.h>\n#include <stddef.h>\n#include "lazy_attn.h"\n'
        "int main(void){"
        'printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(lazy_shared_range_t), offsetof(lazy_shared_range_t, v_offset),'
        " offsetof(lazy_shared_range_t, k_stride), offsetof(lazy_shared_range_t, v_stride),"
        " offsetof(lazy_shared_range_t, key_begin), offsetof(lazy_shared_range_t, key_end));"
        'printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(lazy_shared_item_t), offsetof(lazy_shared_item_t, num_ranges),'
        " offsetof(lazy_shared_item_t, range_keys), offsetof(lazy_shared_item_t, user_begin),"
        " offsetof(lazy_shared_item_t, num_users), offsetof(lazy_shared_item_t, reserved));"
        'printf("%zu %zu %zu %zu %d\\n", sizeof(lazy_shared_user_t), offsetof(lazy_shared_user_t, pos_offset),'
        " offsetof(lazy_shared_user_t, slot), offsetof(lazy_shared_user_t, reserved), LAZY_SHARED_MAX_RANGES);"
        "return 0;}"
    )
    exe = tmp_path / "plan_layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    a, b, c = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")[:3]
    rg, it, us = ops.RANGE_DTYPE, ops.ITEM_DTYPE, ops.USER_DTYPE
    assert [int(x) for x in a.split()] == [rg.itemsize] + [rg.fields[n][1] for n in (
        "v_offset", "k_stride", "v_stride", "key_begin", "key_end")]
    assert [int(x) for x in b.split()] == [it.itemsize] + [it.fields[n][1] for n in (
        "num_ranges", "range_keys", "user_begin", "num_users", "reserved")]
    assert [int(x) for x in c.split()] == [us.itemsize] + [us.fields[n][1] for n in ("pos_offset", "slot", "reserved")] \
        + [ops.SHARED_MAX_RANGES]


def _check_plan(w, plan, g, step, local=False):
    """Invariants of a plan.  Expanding every (item, user, key of the item's run) gives (request, position, stored
    key), which must be exactly the keys of the decode tables, each once.  Every (request, slot) belongs to one
    (item, user) and a request's slots are 0..n-1; items respect the column budget, the range rules (all ranges but
    the last hold range_keys keys, a multiple of 32 when there are several) and are sorted by run length."""
    per_item = 16 // g
    got, slots = [], {}
    keys = plan.item_keys()
    for n, it in enumerate(plan.items):
        assert 1 <= it["num_users"] <= per_item and it["reserved"] == 0
        nr, rk = int(it["num_ranges"]), int(it["range_keys"])
        assert 1 <= nr <= ops_max_ranges and keys[n] <= step
        rgs = plan.ranges[it["range_begin"]: it["range_begin"] + nr]
        lens = rgs["key_end"] - rgs["key_begin"]
        assert np.all(rgs["key_begin"] >= 0) and np.all(lens >= 1)
        assert np.all(lens[:-1] == rk) and 1 <= lens[-1] <= rk
        if nr > 1:
            assert rk % 32 == 0 and not local
        run = [(int(r["k_offset"]), int(r["v_offset"]), int(r["k_stride"]), int(r["v_stride"]), int(r["key_begin"]) + j)
               for r in rgs for j in range(int(r["key_end"] - r["key_begin"]))]
        for u in plan.users[it["user_begin"]: it["user_begin"] + it["num_users"]]:
            assert u["reserved"] == 0
            key = (int(u["request"]), int(u["slot"]))
            assert key not in slots
            slots[key] = n
            got.extend((int(u["request"]), int(u["pos_offset"]) + j, run[j]) for j in range(len(run)))
    assert np.all(np.diff(keys) <= 0)
    expect = []
    for r in range(w.batch):
        for rec in w.chunks[w.chunk_start[r]: w.chunk_start[r + 1]]:
            expect.extend((r, int(rec["pos_offset"]) + j, (int(rec["k_offset"]), int(rec["v_offset"]),
                                                           int(rec["k_stride"]), int(rec["v_stride"]), j))
                          for j in range(int(rec["len"])))
        n = int(plan.slot_start[r + 1] - plan.slot_start[r])
        assert sorted(s for (rr, s) in slots if rr == r) == list(range(n))
    assert len(got) == len(set(got)) and sorted(got) == sorted(expect)
    assert plan.slot_start[0] == 0


ops_max_ranges = 64


@pytest.mark.parametrize("step", [0, 100, 1000])
def test_shared_plan_covers_every_record_key_once(ops, step):
    w = W.rag_decode(seed=5, batch=9, hq=8, hkv=2, n_chunks=5, chunk_len=300, pool_chunks=7, tail_len=9,
                     tail_cap=16)
    plan = ops.shared_decode_plan(ops.config_of(w), w.chunks, w.chunk_start, step)
    _check_plan(w, plan, 4, step or 1024)
    # sharing: the 9 requests x 5 chunks read only 7 stored chunks, so there are far fewer items than records
    if step == 0:
        assert plan.items.size <= 7 * 3 + 9 and plan.users.size == len(w.chunks)


def test_shared_plan_g7_and_zipf_reuse(ops):
    w = W.varlen_rag(seed=6, batch=6, hq=28, hkv=4, pool_chunks=12, len_lo=10, len_hi=400, k_lo=3, k_hi=6,
                     q_lo=1, q_hi=1)
    plan = ops.shared_decode_plan(ops.config_of(w), w.chunks, w.chunk_start, 128)
    _check_plan(w, plan, 7, 128)


@pytest.mark.parametrize("bt,step", [(64, 0), (32, 0), (64, 200), (48, 0), (16, 0)])
def test_shared_plan_chains_paged_blocks(ops, bt, step):
    """A paged store (blocks of bt tokens, one record per block) is read in runs of blocks: with block sizes that
    are multiples of 32 the plan reads exactly the keys of the contiguous store's plan in as many items; other block
    sizes are not chained (one block per item) but still cover every key once.  A local-position store is never
    chained."""
    w = W.rag_decode(seed=8, batch=7, hq=8, hkv=2, n_chunks=4, chunk_len=300, pool_chunks=6, tail_len=40,
                     tail_cap=100)
    wp = W.paginate(w, bt, seed=3)
    cfg = ops.config_of(wp)
    plan = ops.shared_decode_plan(cfg, wp.chunks, wp.chunk_start, step)
    _check_plan(wp, plan, 4, step or 1024)
    base = ops.shared_decode_plan(ops.config_of(w), w.chunks, w.chunk_start, step)
    if bt % 32 == 0:
        assert plan.items["num_ranges"].max() > 1
        if step == 0:
            assert plan.items.size == base.items.size and plan.read_keys() == base.read_keys()
    else:
        assert plan.items["num_ranges"].max() == 1
    local = ops.shared_decode_plan(ops.config_of(wp, key_positions=ops.KEYS_LOCAL), wp.chunks, wp.chunk_start, step)
    _check_plan(wp, local, 4, step or 1024, local=True)


def test_shared_plan_breaks_runs_where_requests_diverge(ops):
    """Two requests read the blocks of chunk A and then of different chunks: the run covers A's blocks only."""
    rec = lambda ko, pos, n=64: (ko, ko + 100000, n, pos, 64, 64)
    a = [rec(1000 * k, 64 * k) for k in range(3)]
    t1 = [rec(50000 + 1000 * k, 192 + 64 * k) for k in range(2)]
    t2 = [rec(80000 + 1000 * k, 192 + 64 * k) for k in range(2)]
    chunks = np.array(a + t1 + a + t2, dtype=ops.CHUNK_DTYPE)
    cs = np.array([0, 5, 10], dtype=np.int32)
    plan = ops.shared_decode_plan(ops.Config(8, 2, 128, 1e4), chunks, cs)
    runs = sorted((int(it["num_ranges"]), int(it["num_users"])) for it in plan.items)
    assert runs == [(2, 1), (2, 1), (3, 2)]


def test_shared_plan_errors(ops):
    w = W.rag_decode(seed=7, batch=2, hq=8, hkv=2, n_chunks=2, chunk_len=40, pool_chunks=3, tail_len=2, tail_cap=4)
    L = ops.lib()
    p = ops.config_of(w).c()
    ch = np.ascontiguousarray(w.chunks)
    cs = np.ascontiguousarray(w.chunk_start, dtype=np.int32)
    items = np.zeros(1, dtype=ops.ITEM_DTYPE)
    ranges = np.zeros(1, dtype=ops.RANGE_DTYPE)
    users = np.zeros(1, dtype=ops.USER_DTYPE)
    ni, nr, nu = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
    ss = np.zeros(3, dtype=np.int32)
    code = L.lazy_shared_decode_plan(ctypes.byref(p), ch.ctypes.data, cs.ctypes.data, 2, 0, items.ctypes.data, 1,
                                     ranges.ctypes.data, 1, users.ctypes.data, 1, ctypes.byref(ni), ctypes.byref(nr),
                                     ctypes.byref(nu), ss.ctypes.data)
    assert code == ops.LAZY_EINVAL and ni.value > 1 and nr.value > 1 and nu.value == len(w.chunks)  # counts reported
    big = ops.Config(34, 2, 128, 1e4)  # G = 17 columns do not fit one workgroup
    pb = big.c()
    args = lambda pp, c, step: (ctypes.byref(pp), c.ctypes.data, cs.ctypes.data, 2, step, None, 0, None, 0, None, 0,
                                ctypes.byref(ni), ctypes.byref(nr), ctypes.byref(nu), ss.ctypes.data)
    assert L.lazy_shared_decode_plan(*args(pb, ch, 0)) == ops.LAZY_EUNSUPPORTED
    bad = ch.copy()
    bad["len"][1] = -3
    assert L.lazy_shared_decode_plan(*args(p, bad, 0)) == ops.LAZY_EDATA
    assert L.lazy_shared_decode_plan(*args(p, ch, -1)) == ops.LAZY_EINVAL
    # scalar checks of the device entry point (no launch)
    assert L.lazy_attn_decode_shared(ctypes.byref(pb), 1, 1, 1, 1, 1, 1, 1, 1, 1, 2, 1, 1, None, None, 0,
                                     None) == ops.LAZY_EUNSUPPORTED
    assert L.lazy_attn_decode_shared(ctypes.byref(p), 1, 1, 1, 1, 1, 3, 1, 1, 1, 2, 0, 1, None, None, 0,
                                     None) == ops.LAZY_EINVAL
    assert L.lazy_attn_decode_shared(ctypes.byref(p), 1, 1, 1, 1, 1, 3, None, 1, 1, 2, 4, 1, None, None, 0,
                                     None) == ops.LAZY_EINVAL                                # ranges missing
    assert L.lazy_attn_decode_shared(ctypes.byref(p), 1, 1, 1, 1, 1, 3, 1, 1, 1, 2, 4, 1, None, None, 0,
                                     None) == ops.LAZY_EWORKSPACE
    assert L.lazy_attn_decode_shared(ctypes.byref(p), 1, 1, 1, 1, 1, 3, 1, 1, 1, 0, 4, 1, None, None, 0,
                                     None) == ops.LAZY_OK
    assert ops.decode_shared_workspace_size(ops.config_of(w), 2, 5) == 5 * 2 * 8 * (2 * 128 + 4)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ missing")
def test_shared_plan_under_address_and_ub_sanitizers(tmp_path):
    drv = tmp_path / "plan_drv.cpp"
    drv.write_text(r"""
#include <stdio.h>
#include <vector>
#include "lazy_attn.h"
int main() {
  lazy_attn_params_t p = {8, 2, 128, 1, 1e4f, 0.f, nullptr, 0, 0};
  // 3 requests; records 0/2/4 read the same stored chunk at different offsets, one 2500-key private record, and a
  // paged run (64-key blocks 5..7 then 8..9) that requests 1 and 2 both read
  std::vector<lazy_chunk_t> c = {{0, 4096, 300, 0, 300, 300}, {9000, 9504, 20, 300, 32, 32},
                                 {0, 4096, 300, 50, 300, 300}, {20000, 90000, 2500, 0, 2500, 2500},
                                 {0, 4096, 300, 7, 300, 300},
                                 {100000, 200000, 64, 3000, 64, 64}, {101000, 201000, 64, 3064, 64, 64},
                                 {102000, 202000, 10, 3128, 64, 64},
                                 {100000, 200000, 64, 4000, 64, 64}, {101000, 201000, 64, 4064, 64, 64},
                                 {102000, 202000, 10, 4128, 64, 64}};
  int32_t cs[4] = {0, 2, 4, 5};
  int32_t cs2[4] = {0, 2, 8, 11};
  int fails = 0;
  for (int local = 0; local < 2; ++local)
    for (const int32_t* table : {cs, cs2})
      for (int step : {0, 1, 64, 200, 1000}) {
        p.key_positions = local;
        int32_t ni = 0, nr = 0, nu = 0, ss[4];
        int code = lazy_shared_decode_plan(&p, c.data(), table, 3, step, nullptr, 0, nullptr, 0, nullptr, 0, &ni,
                                           &nr, &nu, ss);
        if (code != LAZY_EINVAL || ni <= 0 || nr <= 0 || nu <= 0) ++fails;
        std::vector<lazy_shared_item_t> items(ni);
        std::vector<lazy_shared_range_t> ranges(nr);
        std::vector<lazy_shared_user_t> users(nu);
        code = lazy_shared_decode_plan(&p, c.data(), table, 3, step, items.data(), ni, ranges.data(), nr,
                                       users.data(), nu, &ni, &nr, &nu, ss);
        if (code != LAZY_OK || ss[0] != 0 || ss[3] > nu) ++fails;
        int32_t ms = 0;
        for (int r = 0; r < 3; ++r) ms = ss[r + 1] - ss[r] > ms ? ss[r + 1] - ss[r] : ms;
        int64_t bad; const char* why;
        int32_t qpos[3] = {5000, 5000, 5000};
        if (lazy_shared_decode_validate(&p, items.data(), ni, ranges.data(), nr, users.data(), nu, ss, 3, ms, qpos,
                                        1 << 20, 1 << 20, &bad, &why) != LAZY_OK) {
          printf("plan rejected: %s\n", why);
          ++fails;
        }
        if (ni > 0) {  // an item with too many users is rejected, and the validator stays in bounds doing so
          std::vector<lazy_shared_item_t> m = items;
          m[0].num_users = 1000;
          if (lazy_shared_decode_validate(&p, m.data(), ni, ranges.data(), nr, users.data(), nu, ss, 3, ms, qpos,
                                          1 << 20, 1 << 20, &bad, &why) != LAZY_EDATA)
            ++fails;
          m = items;
          m[0].range_begin = nr;
          if (lazy_shared_decode_validate(&p, m.data(), ni, ranges.data(), nr, users.data(), nu, ss, 3, ms, qpos,
                                          1 << 20, 1 << 20, &bad, &why) != LAZY_EDATA)
            ++fails;
        }
        for (const auto& it : items) {
          if (it.user_begin < 0 || it.user_begin + it.num_users > nu || it.num_users < 1 || it.num_users > 4) ++fails;
          if (it.range_begin < 0 || it.num_ranges < 1 || it.range_begin + it.num_ranges > nr) ++fails;
          if (local && it.num_ranges != 1) ++fails;
        }
      }
  int32_t ni = 0, nr = 0, nu = 0, ss[4];
  if (lazy_shared_decode_plan(&p, nullptr, cs, 3, 0, nullptr, 0, nullptr, 0, nullptr, 0, &ni, &nr, &nu, ss) !=
      LAZY_EINVAL)
    ++fails;
  int32_t empty[1] = {0};
  if (lazy_shared_decode_plan(&p, nullptr, empty, 0, 0, nullptr, 0, nullptr, 0, nullptr, 0, &ni, &nr, &nu, ss) !=
      LAZY_OK)
    ++fails;
  printf("sanitized planner ok=%d\n", fails == 0);
  return fails;
}
""")
    exe = tmp_path / "plan_drv"
    subprocess.run(["g++", "-std=c++17", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-I",
                    os.path.join(ROOT, "include"), str(drv), os.path.join(B.CSRC, "lazy_attn_plan.cpp"),
                    os.path.join(B.CSRC, "lazy_attn_validate.cpp"), "-o",
                    str(exe)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "ok=1" in res.stdout


# ---------------------------------------------------------------------------------------------------------------
# Host check of shared-decode plans (the kernel trusts its item / range / user tables).
# ---------------------------------------------------------------------------------------------------------------
def _plan_case(ops, local=False, paged=0):
    w = W.rag_decode(seed=9, batch=7, hq=8, hkv=2, n_chunks=4, chunk_len=300, pool_chunks=6, tail_len=40,
                     tail_cap=100)
    if paged:
        w = W.paginate(w, paged, seed=1)
    cfg = ops.config_of(w, **({"key_positions": ops.KEYS_LOCAL} if local else {}))
    return w, cfg, ops.shared_decode_plan(cfg, w.chunks, w.chunk_start, 0)


@pytest.mark.parametrize("local,paged", [(False, 0), (True, 0), (False, 64), (True, 32)])
def test_shared_plan_validator_accepts_planner_output(ops, local, paged):
    w, cfg, plan = _plan_case(ops, local, paged)
    code, bad, why = ops.validate_shared_plan(cfg, plan, w.q_pos0, w.pool.size, w.pool.size)
    assert code == ops.LAZY_OK, (bad, why)


def _mut(field, idx, value, table="items"):
    def f(plan):
        getattr(plan, table)[field][idx] = value
    return f


SHARED_PLAN_MUTATIONS = [
    (_mut("num_users", 0, 5), "num_users"),            # G = 4: at most 4 users per item
    (_mut("num_users", 0, 0), "num_users"),
    (_mut("num_ranges", 0, 0), "num_ranges"),
    (_mut("num_ranges", 0, 65), "num_ranges"),
    (_mut("range_begin", 0, -1), "ranges outside"),
    (_mut("user_begin", 0, 10 ** 6), "users outside"),
    (_mut("reserved", 0, 1), "reserved"),
    (_mut("range_keys", 0, 0), "range_keys"),
    (_mut("k_offset", 0, 3, "ranges"), "multiples of 8"),
    (_mut("key_end", 0, 10 ** 6, "ranges"), "stride"),
    (_mut("key_begin", 0, -2, "ranges"), "non-empty"),
    (_mut("request", 0, 99, "users"), "request out of range"),
    (_mut("slot", 0, 50, "users"), "slot out of range"),
    (_mut("pos_offset", 0, -5, "users"), "positions out of range"),
]


@pytest.mark.parametrize("mutate,reason", SHARED_PLAN_MUTATIONS)
def test_shared_plan_validator_rejects_contract_violations(ops, mutate, reason):
    w, cfg, plan = _plan_case(ops)
    mutate(plan)
    code, bad, why = ops.validate_shared_plan(cfg, plan, w.q_pos0, w.pool.size, w.pool.size)
    assert code == ops.LAZY_EDATA and reason in why, (code, why)


def test_shared_plan_validator_slot_coverage_pools_and_args(ops):
    w, cfg, plan = _plan_case(ops)
    # a slot written twice (and another never): two users of different items pointed at one slot
    p2 = ops.SharedPlan(plan.items.copy(), plan.ranges.copy(), plan.users.copy(), plan.slot_start.copy())
    r = int(p2.users["request"][0])
    same = np.nonzero(p2.users["request"] == r)[0]
    p2.users["slot"][same[1]] = p2.users["slot"][same[0]]
    code, _, why = ops.validate_shared_plan(cfg, p2, w.q_pos0, w.pool.size, w.pool.size)
    assert code == ops.LAZY_EDATA and "exactly once" in why
    # pools too small, too few slots allowed, a local-position store with multi-range items, bad query position
    assert ops.validate_shared_plan(cfg, plan, w.q_pos0, 1024, w.pool.size)[2] == "range K outside the pool"
    assert ops.validate_shared_plan(cfg, plan, w.q_pos0, w.pool.size, 1024)[2] == "range V outside the pool"
    assert "max_slots" in ops.validate_shared_plan(cfg, plan, w.q_pos0, w.pool.size, w.pool.size, max_slots=1)[2]
    wp, cp, pp = _plan_case(ops, False, 64)
    assert pp.items["num_ranges"].max() > 1
    local = ops.config_of(wp, key_positions=ops.KEYS_LOCAL)
    assert "single ranges" in ops.validate_shared_plan(local, pp, wp.q_pos0, wp.pool.size, wp.pool.size)[2]
    qp = np.array(w.q_pos0, dtype=np.int32)
    qp[2] = -1
    assert "query position" in ops.validate_shared_plan(cfg, plan, qp, w.pool.size, w.pool.size)[2]
    # G = 17 is outside what the shared decode takes; a null parameter block is an argument error
    assert ops.validate_shared_plan(ops.Config(34, 2, 128, 1e4), plan, None, w.pool.size,
                                    w.pool.size)[0] == ops.LAZY_EUNSUPPORTED
    L = ops.lib()
    assert L.lazy_shared_decode_validate(None, None, 0, None, 0, None, 0, plan.slot_start.ctypes.data, 0, 0, None,
                                         0, 0, None, None) == ops.LAZY_EINVAL


@pytest.mark.parametrize("make", ["icl", "rag_decode", "paged", "repeated"])
def test_storage_order_is_a_stable_sort_per_request(ops, make):
    if make == "icl":
        w = W.icl_prefill(seed=7, batch=3, hq=4, hkv=2, d=64, n_chunks=9, chunk_len=40, q_len=5, decode_steps=2)
    elif make == "rag_decode":
        w = W.rag_decode(seed=8, batch=5, hq=8, hkv=2, n_chunks=4, chunk_len=100, pool_chunks=6, tail_len=3,
                         tail_cap=8)
    elif make == "paged":
        w = W.paginate(W.rag_decode(seed=9, batch=3, hq=8, hkv=2, n_chunks=3, chunk_len=130, pool_chunks=4,
                                    tail_len=5, tail_cap=8), 32, seed=2)
    else:  # one request reading the same stored chunk twice, at two offsets (equal keys keep their order)
        w = W.icl_prefill(seed=10, batch=2, hq=4, hkv=2, d=64, n_chunks=4, chunk_len=32, q_len=3, decode_steps=1)
        ch = w.chunks.copy()
        ch[2]["k_offset"], ch[2]["v_offset"] = ch[0]["k_offset"], ch[0]["v_offset"]
        w.chunks[:] = ch
    out = ops.storage_order(w.chunks, w.chunk_start)
    for r in range(w.batch):
        a, b = int(w.chunk_start[r]), int(w.chunk_start[r + 1])
        src, got = w.chunks[a:b], out[a:b]
        order = np.argsort(src["k_offset"], kind="stable")
        assert np.array_equal(got.view(np.uint8), src[order].view(np.uint8)), r
        assert np.all(np.diff(got["k_offset"]) >= 0)
    # in place (out aliases the input) gives the same table
    inplace = np.ascontiguousarray(w.chunks).copy()
    cs = np.ascontiguousarray(w.chunk_start, dtype=np.int32)
    L = ops.lib()
    assert L.lazy_chunk_table_storage_order(inplace.ctypes.data, cs.ctypes.data, cs.size - 1,
                                            inplace.ctypes.data) == ops.LAZY_OK
    assert np.array_equal(inplace.view(np.uint8), out.view(np.uint8))


def test_storage_order_errors(ops):
    L = ops.lib()
    ch = np.zeros(3, dtype=ops.CHUNK_DTYPE)
    out = np.zeros_like(ch)
    good = np.array([0, 1, 3], dtype=np.int32)
    assert L.lazy_chunk_table_storage_order(ch.ctypes.data, good.ctypes.data, 2, out.ctypes.data) == ops.LAZY_OK
    for bad in ([1, 1, 3], [0, 2, 1]):
        cs = np.array(bad, dtype=np.int32)
        assert L.lazy_chunk_table_storage_order(ch.ctypes.data, cs.ctypes.data, 2, out.ctypes.data) == ops.LAZY_EINVAL
    assert L.lazy_chunk_table_storage_order(ch.ctypes.data, good.ctypes.data, -1, out.ctypes.data) == ops.LAZY_EINVAL
    assert L.lazy_chunk_table_storage_order(None, good.ctypes.data, 2, out.ctypes.data) == ops.LAZY_EINVAL
    assert L.lazy_chunk_table_storage_order(ch.ctypes.data, None, 2, out.ctypes.data) == ops.LAZY_EINVAL
    empty = np.zeros(1, dtype=np.int32)
    assert L.lazy_chunk_table_storage_order(None, empty.ctypes.data, 0, None) == ops.LAZY_OK
