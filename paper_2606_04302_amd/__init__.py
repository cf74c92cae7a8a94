"""LazyAttention hot path for MI355X (gfx950): causal / GQA softmax attention over a position-free chunk KV store,
with RoPE applied inside the kernels at each chunk's offset in the current request.

The compute lives in the HIP library ``liblazyattn.so`` (C ABI declared in ``include/lazy_attn.h``); ``ops``
is the thin ctypes binding over torch tensors.  Importing this package does not load the library: the first
call into ``ops`` does, and it raises if the library is missing.
"""

__all__ = ["workloads", "accounting", "ops"]
