// Host-only check of chunk / query tables against the layout contract of lazy_attn.h.  Pure C++ with no HIP
// dependency so that it can be built and sanitised on a machine without a GPU.
#include <stdint.h>

#include "lazy_attn.h"

namespace {

int fail(int64_t idx, const char* why, int64_t* bad_index, const char** reason) {
  if (bad_index) *bad_index = idx;
  if (reason) *reason = why;
  return LAZY_EDATA;
}

}  // namespace

extern "C" int lazy_attn_validate(const lazy_attn_params_t* p, const int32_t* q_start, const int32_t* q_pos0,
                                  const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch,
                                  int64_t k_pool_elems, int64_t v_pool_elems, int64_t* bad_index,
                                  const char** reason) {
  if (bad_index) *bad_index = -1;
  if (reason) *reason = "";
  if (!p || batch < 0 || !chunk_start || k_pool_elems < 0 || v_pool_elems < 0) return LAZY_EINVAL;
  if (p->num_q_heads <= 0 || p->num_kv_heads <= 0 || p->num_q_heads % p->num_kv_heads != 0) return LAZY_EINVAL;
  if (p->head_dim != 64 && p->head_dim != 128) return LAZY_EUNSUPPORTED;
  const int64_t d = p->head_dim, hkv = p->num_kv_heads;
  if (chunk_start[0] != 0) return fail(0, "chunk_start[0] must be 0", bad_index, reason);
  for (int32_t r = 0; r < batch; ++r)
    if (chunk_start[r + 1] < chunk_start[r]) return fail(r, "chunk_start must be non-decreasing", bad_index, reason);
  const int64_t n = chunk_start[batch];
  if (n > 0 && !chunks) return LAZY_EINVAL;
  for (int64_t i = 0; i < n; ++i) {
    const lazy_chunk_t& c = chunks[i];
    if (c.len < 1) return fail(i, "record len must be >= 1", bad_index, reason);
    if (c.pos_offset < 0) return fail(i, "record pos_offset must be >= 0", bad_index, reason);
    if ((int64_t)c.pos_offset + c.len > LAZY_MAX_POS) return fail(i, "key position beyond LAZY_MAX_POS", bad_index, reason);
    if (c.k_stride < c.len || c.v_stride < c.len) return fail(i, "stride must be >= len", bad_index, reason);
    if (c.k_offset < 0 || c.v_offset < 0) return fail(i, "offsets must be >= 0", bad_index, reason);
    if ((c.k_offset & 7) || (c.v_offset & 7)) return fail(i, "offsets must be multiples of 8 elements", bad_index, reason);
    const int64_t kend = c.k_offset + ((hkv - 1) * c.k_stride + c.len) * d;
    const int64_t vend = c.v_offset + ((hkv - 1) * c.v_stride + c.len) * d;
    if (kend > k_pool_elems) return fail(i, "K range outside the pool", bad_index, reason);
    if (vend > v_pool_elems) return fail(i, "V range outside the pool", bad_index, reason);
  }
  if (!q_pos0) return LAZY_OK;
  if (q_start && q_start[0] != 0) return fail(0, "q_start[0] must be 0", bad_index, reason);
  for (int32_t r = 0; r < batch; ++r) {
    const int64_t lq = q_start ? (int64_t)q_start[r + 1] - q_start[r] : 1;
    if (lq < 0) return fail(r, "q_start must be non-decreasing", bad_index, reason);
    if (q_pos0[r] < 0 || (int64_t)q_pos0[r] + lq > LAZY_MAX_POS)
      return fail(r, "query position out of range", bad_index, reason);
    if (p->causal && lq > 0) {
      // The request's earliest query must see at least one key (then every later one does).
      bool seen = false;
      for (int32_t i = chunk_start[r]; i < chunk_start[r + 1] && !seen; ++i) seen = chunks[i].pos_offset <= q_pos0[r];
      if (!seen) return fail(r, "a query sees no key under the causal rule", bad_index, reason);
    } else if (lq > 0 && chunk_start[r + 1] == chunk_start[r]) {
      return fail(r, "request has queries but no keys", bad_index, reason);
    }
  }
  return LAZY_OK;
}
