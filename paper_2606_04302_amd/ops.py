"""Thin ctypes binding of ``liblazyattn.so`` (C ABI in ``include/lazy_attn.h``) over torch tensors.

Argument marshalling only: torch supplies device memory and the current stream, every step of the attention runs
in the HIP library.  There is no fallback: if the library is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np
import torch

from .workloads import CHUNK_DTYPE, Workload, bf16_bits

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblazyattn.so")

LAZY_OK, LAZY_EINVAL, LAZY_EUNSUPPORTED, LAZY_EWORKSPACE, LAZY_EHIP, LAZY_EDATA = 0, -1, -2, -3, -4, -5
KEYS_NOPE, KEYS_LOCAL = 0, 1  # key-store conventions (lazy_attn_params_t.key_positions)
ROPE_HALF, ROPE_INTERLEAVED, ALIBI = 0, 1, 2  # positional method (lazy_attn_params_t.rope_style)
CACHE_DEFAULT, CACHE_STREAM = 0, 1  # K / V cache hint (lazy_attn_params_t.cache_hint)

_c_i32, _c_i64, _c_f32, _c_p, _c_sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t


class LazyAttnParams(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", _c_i32),
        ("num_kv_heads", _c_i32),
        ("head_dim", _c_i32),
        ("causal", _c_i32),
        ("rope_base", _c_f32),
        ("softmax_scale", _c_f32),
        ("inv_freq", _c_p),
        ("num_splits", _c_i32),
        ("key_positions", _c_i32),
        ("rope_style", _c_i32),
        ("q_prerotated", _c_i32),
        ("cache_hint", _c_i32),
    ]


class LazyChunk(ctypes.Structure):
    _fields_ = [("k_offset", _c_i64), ("v_offset", _c_i64), ("len", _c_i32), ("pos_offset", _c_i32),
                ("k_stride", _c_i32), ("v_stride", _c_i32)]


assert ctypes.sizeof(LazyChunk) == CHUNK_DTYPE.itemsize == 32

# Plan records of the chunk-major shared decode (lazy_shared_item_t, lazy_shared_user_t).
RANGE_DTYPE = np.dtype([("k_offset", "<i8"), ("v_offset", "<i8"), ("k_stride", "<i4"), ("v_stride", "<i4"),
                        ("key_begin", "<i4"), ("key_end", "<i4")])
ITEM_DTYPE = np.dtype([("range_begin", "<i4"), ("num_ranges", "<i4"), ("range_keys", "<i4"), ("user_begin", "<i4"),
                       ("num_users", "<i4"), ("reserved", "<i4")])
USER_DTYPE = np.dtype([("request", "<i4"), ("pos_offset", "<i4"), ("slot", "<i4"), ("reserved", "<i4")])
assert RANGE_DTYPE.itemsize == 32 and ITEM_DTYPE.itemsize == 24 and USER_DTYPE.itemsize == 16
SHARED_MAX_RANGES = 64  # LAZY_SHARED_MAX_RANGES

_ATTN_PREFILL = [ctypes.POINTER(LazyAttnParams), _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i32, _c_i32, _c_i32,
                 _c_i32, _c_p, _c_p, _c_p, _c_sz, _c_p]
_ATTN_DECODE = [ctypes.POINTER(LazyAttnParams), _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i32, _c_i32, _c_p, _c_p,
                _c_p, _c_sz, _c_p]
SIGNATURES = {
    "lazy_attn_prefill": (_c_i32, _ATTN_PREFILL),
    "lazy_plain_attn_prefill": (_c_i32, _ATTN_PREFILL),
    "lazy_attn_prefill_workspace_size": (_c_sz, [ctypes.POINTER(LazyAttnParams), _c_i32, _c_i32, _c_i32, _c_i32]),
    "lazy_attn_decode": (_c_i32, _ATTN_DECODE),
    "lazy_plain_attn_decode": (_c_i32, _ATTN_DECODE),
    "lazy_attn_decode_workspace_size": (_c_sz, [ctypes.POINTER(LazyAttnParams), _c_i32, _c_i32]),
    "lazy_attn_decode_noalloc": (_c_i32, [ctypes.POINTER(LazyAttnParams), _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i32,
                                          _c_i32, _c_p, _c_p, _c_p]),
    "lazy_attn_combine": (_c_i32, [_c_p, _c_p, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p]),
    "lazy_materialize_k": (_c_i32, [ctypes.POINTER(LazyAttnParams), _c_p, _c_p, _c_i32, _c_i32, _c_i64, _c_p, _c_p,
                                    _c_p]),
    "lazy_attn_validate": (_c_i32, [ctypes.POINTER(LazyAttnParams), _c_p, _c_p, _c_p, _c_p, _c_i32, _c_i64, _c_i64,
                                    ctypes.POINTER(_c_i64), ctypes.POINTER(ctypes.c_char_p)]),
    "lazy_shared_decode_plan": (_c_i32, [ctypes.POINTER(LazyAttnParams), _c_p, _c_p, _c_i32, _c_i32, _c_p, _c_i32,
                                         _c_p, _c_i32, _c_p, _c_i32, ctypes.POINTER(_c_i32), ctypes.POINTER(_c_i32),
                                         ctypes.POINTER(_c_i32), _c_p]),
    "lazy_attn_decode_shared": (_c_i32, [ctypes.POINTER(LazyAttnParams), _c_p, _c_p, _c_p, _c_p, _c_p, _c_i32, _c_p,
                                         _c_p, _c_p, _c_i32, _c_i32, _c_p, _c_p, _c_p, _c_sz, _c_p]),
    "lazy_attn_decode_shared_workspace_size": (_c_sz, [ctypes.POINTER(LazyAttnParams), _c_i32, _c_i32]),
    "lazy_chunk_table_storage_order": (_c_i32, [_c_p, _c_p, _c_i32, _c_p]),
    "lazy_shared_decode_validate": (_c_i32, [ctypes.POINTER(LazyAttnParams), _c_p, _c_i32, _c_p, _c_i32, _c_p,
                                             _c_i32, _c_p, _c_i32, _c_i32, _c_p, _c_i64, _c_i64,
                                             ctypes.POINTER(_c_i64), ctypes.POINTER(ctypes.c_char_p)]),
    "lazy_pool_create": (_c_p, [_c_i32]),
    "lazy_pool_destroy": (None, [_c_p]),
    "lazy_pool_acquire": (_c_i32, [_c_p, ctypes.c_uint64, ctypes.POINTER(_c_i32), ctypes.POINTER(_c_i32),
                                   ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(_c_i32)]),
    "lazy_pool_stats": (_c_i32, [_c_p, ctypes.POINTER(_c_i64), ctypes.POINTER(_c_i64), ctypes.POINTER(_c_i64),
                                 ctypes.POINTER(_c_i32)]),
    "lazy_attn_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "lazy_attn_version": (ctypes.c_int, []),
}

_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_04302_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


class LazyAttnError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {strerror(code)} (code {code})")
        self.code = code


def strerror(code: int) -> str:
    return lib().lazy_attn_strerror(code).decode()


def _check(code: int, what: str):
    if code != LAZY_OK:
        raise LazyAttnError(code, what)


@dataclass
class Config:
    """Head layout and positional-encoding parameters of one launch."""

    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    rope_base: float
    causal: bool = True
    softmax_scale: float = 0.0
    inv_freq: torch.Tensor | None = None  # device fp32 [D/2]
    num_splits: int = 0
    key_positions: int = 0  # KEYS_NOPE or KEYS_LOCAL
    rope_style: int = 0  # ROPE_HALF, ROPE_INTERLEAVED or ALIBI (then inv_freq optionally holds the Hq slopes)
    q_prerotated: bool = False  # q already holds R(q_pos) q
    cache_hint: int = 0  # CACHE_DEFAULT or CACHE_STREAM (decode: non-temporal K / V loads)

    def c(self) -> LazyAttnParams:
        return LazyAttnParams(self.num_q_heads, self.num_kv_heads, self.head_dim, int(bool(self.causal)),
                              float(self.rope_base), float(self.softmax_scale),
                              None if self.inv_freq is None else self.inv_freq.data_ptr(), int(self.num_splits),
                              int(self.key_positions), int(self.rope_style), int(bool(self.q_prerotated)),
                              int(self.cache_hint))


def config_of(w: Workload, **kw) -> Config:
    return Config(w.num_q_heads, w.num_kv_heads, w.head_dim, w.rope_base, w.causal, **kw)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _need(cond, msg):
    if not cond:
        raise ValueError(msg)


def _dev(t, dtype, name):
    _need(t.is_cuda, f"{name} must be a device tensor")
    _need(t.dtype == dtype, f"{name} must be {dtype}, got {t.dtype}")
    _need(t.is_contiguous(), f"{name} must be contiguous")


def _chunks(t):
    _need(t.is_cuda and t.dtype == torch.uint8 and t.is_contiguous() and t.numel() % 32 == 0,
          "chunks must be a contiguous device uint8 tensor of 32-byte lazy_chunk_t records")


def prefill_workspace_size(cfg: Config, batch: int, total_q: int, max_q_len: int, max_kv_len: int) -> int:
    p = cfg.c()
    return int(lib().lazy_attn_prefill_workspace_size(ctypes.byref(p), batch, total_q, max_q_len, max_kv_len))


def decode_workspace_size(cfg: Config, batch: int, max_kv_len: int) -> int:
    p = cfg.c()
    return int(lib().lazy_attn_decode_workspace_size(ctypes.byref(p), batch, max_kv_len))


def _workspace(nbytes, device, workspace):
    if nbytes == 0:
        return None
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return workspace


def prefill(cfg: Config, q, q_start, q_pos0, k_pool, v_pool, chunks, chunk_start, max_q_len: int, max_kv_len: int,
            out=None, lse=None, workspace=None, stream=None, plain: bool = False):
    """lazy_attn_prefill (or lazy_plain_attn_prefill with plain=True).  Returns (out, lse)."""
    _dev(q, torch.bfloat16, "q")
    _dev(k_pool, torch.bfloat16, "k_pool")
    _dev(v_pool, torch.bfloat16, "v_pool")
    _dev(q_start, torch.int32, "q_start")
    _dev(q_pos0, torch.int32, "q_pos0")
    _dev(chunk_start, torch.int32, "chunk_start")
    _chunks(chunks)
    _need(q.dim() == 3 and q.shape[1] == cfg.num_q_heads and q.shape[2] == cfg.head_dim, "q must be [T, Hq, D]")
    batch = q_start.numel() - 1
    _need(chunk_start.numel() == batch + 1 and q_pos0.numel() == batch, "table sizes disagree with the batch")
    total_q = q.shape[0]
    if out is None:
        out = torch.empty_like(q)
    _dev(out, torch.bfloat16, "out")
    _need(out.shape == q.shape, "out must have the shape of q")
    if lse is not None:
        _dev(lse, torch.float32, "lse")
        _need(lse.shape == (total_q, cfg.num_q_heads), "lse must be [T, Hq]")
    nbytes = prefill_workspace_size(cfg, batch, total_q, max_q_len, max_kv_len)
    workspace = _workspace(nbytes, q.device, workspace)
    p = cfg.c()
    fn = lib().lazy_plain_attn_prefill if plain else lib().lazy_attn_prefill
    _check(fn(ctypes.byref(p), q.data_ptr(), q_start.data_ptr(), q_pos0.data_ptr(), k_pool.data_ptr(),
              v_pool.data_ptr(), chunks.data_ptr(), chunk_start.data_ptr(), batch, total_q, max_q_len, max_kv_len,
              out.data_ptr(), _ptr(lse), _ptr(workspace), nbytes, _stream(stream)),
           "lazy_plain_attn_prefill" if plain else "lazy_attn_prefill")
    return out, lse


def decode(cfg: Config, q, q_pos, k_pool, v_pool, chunks, chunk_start, max_kv_len: int, out=None, lse=None,
           workspace=None, stream=None, plain: bool = False):
    """lazy_attn_decode (or lazy_plain_attn_decode with plain=True).  q is [B, Hq, D].  Returns (out, lse)."""
    _dev(q, torch.bfloat16, "q")
    _dev(k_pool, torch.bfloat16, "k_pool")
    _dev(v_pool, torch.bfloat16, "v_pool")
    _dev(q_pos, torch.int32, "q_pos")
    _dev(chunk_start, torch.int32, "chunk_start")
    _chunks(chunks)
    _need(q.dim() == 3 and q.shape[1] == cfg.num_q_heads and q.shape[2] == cfg.head_dim, "q must be [B, Hq, D]")
    batch = q.shape[0]
    _need(chunk_start.numel() == batch + 1 and q_pos.numel() == batch, "table sizes disagree with the batch")
    if out is None:
        out = torch.empty_like(q)
    _dev(out, torch.bfloat16, "out")
    if lse is not None:
        _dev(lse, torch.float32, "lse")
        _need(lse.shape == (batch, cfg.num_q_heads), "lse must be [B, Hq]")
    nbytes = decode_workspace_size(cfg, batch, max_kv_len)
    workspace = _workspace(nbytes, q.device, workspace)
    p = cfg.c()
    fn = lib().lazy_plain_attn_decode if plain else lib().lazy_attn_decode
    _check(fn(ctypes.byref(p), q.data_ptr(), q_pos.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(),
              chunks.data_ptr(), chunk_start.data_ptr(), batch, max_kv_len, out.data_ptr(), _ptr(lse),
              _ptr(workspace), nbytes, _stream(stream)),
           "lazy_plain_attn_decode" if plain else "lazy_attn_decode")
    return out, lse


NOALLOC_SCRATCH_BYTES = 8 << 20  # LAZY_NOALLOC_SCRATCH_BYTES


def decode_noalloc(cfg: Config, q, q_pos, k_pool, v_pool, chunks, chunk_start, max_kv_len: int, out, lse=None,
                   stream=None):
    """lazy_attn_decode_noalloc: lazy_attn_decode with the split partials in the library's fixed device array.
    The caller passes the output (nothing is allocated here either).  Returns (out, lse)."""
    _dev(q, torch.bfloat16, "q")
    _dev(k_pool, torch.bfloat16, "k_pool")
    _dev(v_pool, torch.bfloat16, "v_pool")
    _dev(q_pos, torch.int32, "q_pos")
    _dev(chunk_start, torch.int32, "chunk_start")
    _chunks(chunks)
    _need(q.dim() == 3 and q.shape[1] == cfg.num_q_heads and q.shape[2] == cfg.head_dim, "q must be [B, Hq, D]")
    batch = q.shape[0]
    _need(chunk_start.numel() == batch + 1 and q_pos.numel() == batch, "table sizes disagree with the batch")
    _dev(out, torch.bfloat16, "out")
    _need(out.shape == q.shape, "out must have the shape of q")
    if lse is not None:
        _dev(lse, torch.float32, "lse")
        _need(lse.shape == (batch, cfg.num_q_heads), "lse must be [B, Hq]")
    p = cfg.c()
    _check(lib().lazy_attn_decode_noalloc(ctypes.byref(p), q.data_ptr(), q_pos.data_ptr(), k_pool.data_ptr(),
                                          v_pool.data_ptr(), chunks.data_ptr(), chunk_start.data_ptr(), batch,
                                          max_kv_len, out.data_ptr(), _ptr(lse), _stream(stream)),
           "lazy_attn_decode_noalloc")
    return out, lse


def combine(part_o, part_lse, out=None, lse=None, stream=None):
    """lazy_attn_combine: part_o [S, rows, D] bf16 (normalised partial outputs), part_lse [S, rows] fp32
    -> out [rows, D] bf16, lse [rows] fp32 (optional)."""
    _dev(part_o, torch.bfloat16, "part_o")
    _dev(part_lse, torch.float32, "part_lse")
    s, rows, d = part_o.shape
    _need(part_lse.shape == (s, rows), "part_lse must be [S, rows]")
    if out is None:
        out = torch.empty((rows, d), dtype=torch.bfloat16, device=part_o.device)
    _dev(out, torch.bfloat16, "out")
    if lse is not None:
        _dev(lse, torch.float32, "lse")
    _check(lib().lazy_attn_combine(part_o.data_ptr(), part_lse.data_ptr(), s, rows, d, out.data_ptr(), _ptr(lse),
                                   _stream(stream)), "lazy_attn_combine")
    return out, lse


def split_views(workspace, rows: int, head_dim: int):
    """The split-KV partial results inside a prefill / decode workspace: (part_o [S, rows, D] bf16,
    part_lse [S, rows] fp32), S = the number of splits the workspace was sized for (0 if it is empty)."""
    per = rows * (2 * head_dim + 4)
    s = workspace.numel() // per if per else 0
    if s <= 1:
        return None, None
    po = workspace[: s * rows * head_dim * 2].view(torch.bfloat16).view(s, rows, head_dim)
    pl = workspace[s * rows * head_dim * 2: s * per].view(torch.float32).view(s, rows)
    return po, pl


def materialize_k(cfg: Config, k_pool, chunks, max_chunk_len: int, total_kv: int, k_out=None, chunks_out=None,
                  stream=None):
    """lazy_materialize_k: rotated, request-contiguous copy of every record's keys.  Returns (k_out, chunks_out)."""
    _dev(k_pool, torch.bfloat16, "k_pool")
    _chunks(chunks)
    n = chunks.numel() // 32
    if k_out is None:
        k_out = torch.empty(max(1, cfg.num_kv_heads * total_kv * cfg.head_dim), dtype=torch.bfloat16,
                            device=k_pool.device)
    if chunks_out is None:
        chunks_out = torch.empty_like(chunks)
    _dev(k_out, torch.bfloat16, "k_out")
    _chunks(chunks_out)
    _need(k_out.numel() >= cfg.num_kv_heads * total_kv * cfg.head_dim, "k_out too small")
    p = cfg.c()
    _check(lib().lazy_materialize_k(ctypes.byref(p), k_pool.data_ptr(), chunks.data_ptr(), n, max_chunk_len, total_kv,
                                    k_out.data_ptr(), chunks_out.data_ptr(), _stream(stream)), "lazy_materialize_k")
    return k_out, chunks_out


def validate(cfg: Config, q_start, q_pos0, chunks: np.ndarray, chunk_start, k_pool_elems: int, v_pool_elems: int):
    """lazy_attn_validate on host (numpy) tables.  Returns (code, bad_index, reason)."""
    chunks = np.ascontiguousarray(chunks, dtype=CHUNK_DTYPE)
    cs = np.ascontiguousarray(chunk_start, dtype=np.int32)
    qs = None if q_start is None else np.ascontiguousarray(q_start, dtype=np.int32)
    qp = None if q_pos0 is None else np.ascontiguousarray(q_pos0, dtype=np.int32)
    bad = _c_i64(-1)
    why = ctypes.c_char_p()
    p = cfg.c()
    code = lib().lazy_attn_validate(ctypes.byref(p), None if qs is None else qs.ctypes.data,
                                    None if qp is None else qp.ctypes.data, chunks.ctypes.data if chunks.size else None,
                                    cs.ctypes.data, cs.size - 1, k_pool_elems, v_pool_elems, ctypes.byref(bad),
                                    ctypes.byref(why))
    return code, int(bad.value), (why.value or b"").decode()


@dataclass
class SharedPlan:
    """A chunk-major shared-decode plan (host arrays from lazy_shared_decode_plan)."""

    items: np.ndarray       # ITEM_DTYPE
    ranges: np.ndarray      # RANGE_DTYPE
    users: np.ndarray       # USER_DTYPE
    slot_start: np.ndarray  # int32 [batch+1]

    @property
    def max_slots(self) -> int:
        return int(np.diff(self.slot_start).max()) if self.slot_start.size > 1 else 0

    def item_keys(self) -> np.ndarray:
        """Keys of every item's run."""
        last = self.ranges[self.items["range_begin"] + self.items["num_ranges"] - 1]
        return ((self.items["num_ranges"].astype(np.int64) - 1) * self.items["range_keys"]
                + (last["key_end"] - last["key_begin"]))

    def read_keys(self) -> int:
        """Keys read per KV head by one shared-decode launch: every item reads its run once."""
        return int(self.item_keys().sum()) if self.items.size else 0


def shared_decode_plan(cfg: Config, chunks: np.ndarray, chunk_start, max_keys_per_item: int = 0) -> SharedPlan:
    """lazy_shared_decode_plan on host tables (grows the output arrays if the first guess is too small)."""
    chunks = np.ascontiguousarray(chunks, dtype=CHUNK_DTYPE)
    cs = np.ascontiguousarray(chunk_start, dtype=np.int32)
    batch = cs.size - 1
    step = max_keys_per_item or 1024
    cap = max(1, int(np.sum((chunks["len"].astype(np.int64) + step - 1) // step)) if chunks.size else 1)
    p = cfg.c()
    n_items, n_ranges, n_users = _c_i32(0), _c_i32(0), _c_i32(0)
    slot_start = np.zeros(batch + 1, dtype=np.int32)
    for _ in range(2):
        items = np.zeros(cap, dtype=ITEM_DTYPE)
        ranges = np.zeros(cap, dtype=RANGE_DTYPE)
        users = np.zeros(cap, dtype=USER_DTYPE)
        code = lib().lazy_shared_decode_plan(ctypes.byref(p), chunks.ctypes.data if chunks.size else None,
                                             cs.ctypes.data, batch, max_keys_per_item, items.ctypes.data, cap,
                                             ranges.ctypes.data, cap, users.ctypes.data, cap, ctypes.byref(n_items),
                                             ctypes.byref(n_ranges), ctypes.byref(n_users), slot_start.ctypes.data)
        need = max(n_items.value, n_ranges.value, n_users.value)
        if code == LAZY_EINVAL and need > cap:
            cap = need
            continue
        _check(code, "lazy_shared_decode_plan")
        return SharedPlan(items[: n_items.value].copy(), ranges[: n_ranges.value].copy(), users[: n_users.value].copy(),
                          slot_start)
    raise RuntimeError("lazy_shared_decode_plan: capacity did not converge")


def storage_order(chunks: np.ndarray, chunk_start) -> np.ndarray:
    """lazy_chunk_table_storage_order on host tables: a copy with each request's records sorted by k_offset."""
    chunks = np.ascontiguousarray(chunks, dtype=CHUNK_DTYPE)
    cs = np.ascontiguousarray(chunk_start, dtype=np.int32)
    out = np.empty_like(chunks)
    _check(lib().lazy_chunk_table_storage_order(chunks.ctypes.data if chunks.size else None, cs.ctypes.data,
                                                cs.size - 1, out.ctypes.data if out.size else None),
           "lazy_chunk_table_storage_order")
    return out


def validate_shared_plan(cfg: Config, plan: SharedPlan, q_pos, k_pool_elems: int, v_pool_elems: int,
                         max_slots: int | None = None):
    """lazy_shared_decode_validate on a host plan.  Returns (code, bad_index, reason)."""
    items = np.ascontiguousarray(plan.items, dtype=ITEM_DTYPE)
    ranges = np.ascontiguousarray(plan.ranges, dtype=RANGE_DTYPE)
    users = np.ascontiguousarray(plan.users, dtype=USER_DTYPE)
    ss = np.ascontiguousarray(plan.slot_start, dtype=np.int32)
    qp = None if q_pos is None else np.ascontiguousarray(q_pos, dtype=np.int32)
    bad = _c_i64(-1)
    why = ctypes.c_char_p()
    p = cfg.c()
    ptr = lambda a: a.ctypes.data if a.size else None
    code = lib().lazy_shared_decode_validate(ctypes.byref(p), ptr(items), items.size, ptr(ranges), ranges.size,
                                             ptr(users), users.size, ss.ctypes.data, ss.size - 1,
                                             plan.max_slots if max_slots is None else max_slots,
                                             None if qp is None else qp.ctypes.data, k_pool_elems, v_pool_elems,
                                             ctypes.byref(bad), ctypes.byref(why))
    return code, int(bad.value), (why.value or b"").decode()


@dataclass
class DevicePlan:
    items: torch.Tensor
    ranges: torch.Tensor
    users: torch.Tensor
    slot_start: torch.Tensor
    num_items: int
    max_slots: int


def upload_plan(plan: SharedPlan, device="cuda") -> DevicePlan:
    def raw(a):
        b = np.ascontiguousarray(a).view(np.uint8).reshape(-1)
        return torch.from_numpy(b.copy() if b.size else np.zeros(16, np.uint8)).to(device)
    return DevicePlan(raw(plan.items), raw(plan.ranges), raw(plan.users),
                      torch.from_numpy(plan.slot_start.copy()).to(device), int(plan.items.size), plan.max_slots)


def decode_shared_workspace_size(cfg: Config, batch: int, max_slots: int) -> int:
    p = cfg.c()
    return int(lib().lazy_attn_decode_shared_workspace_size(ctypes.byref(p), batch, max_slots))


def decode_shared(cfg: Config, q, q_pos, k_pool, v_pool, plan: DevicePlan, out=None, lse=None, workspace=None,
                  stream=None):
    """lazy_attn_decode_shared over an uploaded plan.  q is [B, Hq, D].  Returns (out, lse)."""
    _dev(q, torch.bfloat16, "q")
    _dev(k_pool, torch.bfloat16, "k_pool")
    _dev(v_pool, torch.bfloat16, "v_pool")
    _dev(q_pos, torch.int32, "q_pos")
    _dev(plan.slot_start, torch.int32, "slot_start")
    _need(q.dim() == 3 and q.shape[1] == cfg.num_q_heads and q.shape[2] == cfg.head_dim, "q must be [B, Hq, D]")
    batch = q.shape[0]
    _need(q_pos.numel() == batch and plan.slot_start.numel() == batch + 1, "table sizes disagree with the batch")
    if out is None:
        out = torch.empty_like(q)
    _dev(out, torch.bfloat16, "out")
    if lse is not None:
        _dev(lse, torch.float32, "lse")
        _need(lse.shape == (batch, cfg.num_q_heads), "lse must be [B, Hq]")
    nbytes = decode_shared_workspace_size(cfg, batch, plan.max_slots)
    workspace = _workspace(nbytes, q.device, workspace)
    p = cfg.c()
    _check(lib().lazy_attn_decode_shared(ctypes.byref(p), q.data_ptr(), q_pos.data_ptr(), k_pool.data_ptr(),
                                         v_pool.data_ptr(), plan.items.data_ptr(), plan.num_items,
                                         plan.ranges.data_ptr(), plan.users.data_ptr(), plan.slot_start.data_ptr(),
                                         batch, plan.max_slots,
                                         out.data_ptr(), _ptr(lse), _ptr(workspace), nbytes, _stream(stream)),
           "lazy_attn_decode_shared")
    return out, lse


# ---------------------------------------------------------------------------------------------------------------
# Host -> device marshalling of a seeded workload.
# ---------------------------------------------------------------------------------------------------------------


def bf16_tensor(x: np.ndarray, device) -> torch.Tensor:
    """float32 array holding exact bf16 values -> bf16 device tensor (bit copy, no rounding)."""
    bits = bf16_bits(x)
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(device)


def chunks_tensor(chunks: np.ndarray, device) -> torch.Tensor:
    raw = np.ascontiguousarray(chunks, dtype=CHUNK_DTYPE).view(np.uint8).reshape(-1)
    return torch.from_numpy(raw.copy()).to(device)


def chunks_from_tensor(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(CHUNK_DTYPE)


@dataclass
class DeviceWorkload:
    w: Workload
    q: torch.Tensor
    q_start: torch.Tensor
    q_pos0: torch.Tensor
    pool: torch.Tensor
    chunks: torch.Tensor
    chunk_start: torch.Tensor

    @property
    def cfg(self) -> Config:
        return config_of(self.w)


def upload(w: Workload, device="cuda") -> DeviceWorkload:
    return DeviceWorkload(
        w=w,
        q=bf16_tensor(w.q, device),
        q_start=torch.from_numpy(w.q_start.astype(np.int32)).to(device),
        q_pos0=torch.from_numpy(w.q_pos0.astype(np.int32)).to(device),
        pool=bf16_tensor(w.pool, device),
        chunks=chunks_tensor(w.chunks, device),
        chunk_start=torch.from_numpy(w.chunk_start.astype(np.int32)).to(device),
    )


def run_lazy(dw: DeviceWorkload, cfg: Config | None = None, with_lse: bool = True, plain_k=None, plain_chunks=None,
             **kw):
    """Run the workload's hot path through the library: prefill or decode by its kind.  With plain_k /
    plain_chunks (from materialize_k) the plain (no K rotation) entry points run over the materialised keys."""
    w = dw.w
    cfg = cfg or dw.cfg
    lse = torch.empty((w.total_q, w.num_q_heads), dtype=torch.float32, device=dw.q.device) if with_lse else None
    plain = plain_k is not None
    kp = plain_k if plain else dw.pool
    ch = plain_chunks if plain else dw.chunks
    if w.kind == "decode":
        return decode(cfg, dw.q, dw.q_pos0, kp, dw.pool, ch, dw.chunk_start, max(1, w.max_kv_len), lse=lse,
                      plain=plain, **kw)
    return prefill(cfg, dw.q, dw.q_start, dw.q_pos0, kp, dw.pool, ch, dw.chunk_start, max(1, w.max_q_len),
                   max(1, w.max_kv_len), lse=lse, plain=plain, **kw)


def run_materialized(dw: DeviceWorkload, cfg: Config | None = None, **kw):
    """Materialise-then-attend baseline: rotate-and-copy K, then plain attention over the copy."""
    w = dw.w
    cfg = cfg or dw.cfg
    total_kv = int(w.chunks["len"].astype(np.int64).sum())
    k_out, ch_out = materialize_k(cfg, dw.pool, dw.chunks, int(w.chunks["len"].max()) if len(w.chunks) else 0,
                                  total_kv)
    return run_lazy(dw, cfg, plain_k=k_out, plain_chunks=ch_out, **kw), (k_out, ch_out)
