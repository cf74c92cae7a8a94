// Host-only checks of chunk / query tables and of shared-decode plans against the layout contract of lazy_attn.h.
// Pure C++ with no HIP dependency so that it can be built and sanitised on a machine without a GPU.
#include <stdint.h>

#include <vector>

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

extern "C" int lazy_shared_decode_validate(const lazy_attn_params_t* p, const lazy_shared_item_t* items,
                                           int32_t num_items, const lazy_shared_range_t* ranges, int32_t num_ranges,
                                           const lazy_shared_user_t* users, int32_t num_users,
                                           const int32_t* slot_start, int32_t batch, int32_t max_slots,
                                           const int32_t* q_pos, int64_t k_pool_elems, int64_t v_pool_elems,
                                           int64_t* bad_index, const char** reason) {
  if (bad_index) *bad_index = -1;
  if (reason) *reason = "";
  if (!p || batch < 0 || num_items < 0 || num_ranges < 0 || num_users < 0 || max_slots < 0 || !slot_start ||
      k_pool_elems < 0 || v_pool_elems < 0)
    return LAZY_EINVAL;
  if ((num_items > 0 && !items) || (num_ranges > 0 && !ranges) || (num_users > 0 && !users)) return LAZY_EINVAL;
  if (p->num_q_heads <= 0 || p->num_kv_heads <= 0 || p->num_q_heads % p->num_kv_heads != 0) return LAZY_EINVAL;
  if (p->head_dim != 64 && p->head_dim != 128) return LAZY_EUNSUPPORTED;
  const int32_t g = p->num_q_heads / p->num_kv_heads;
  if (g > 16) return LAZY_EUNSUPPORTED;
  const int64_t d = p->head_dim, hkv = p->num_kv_heads;
  const bool local = p->key_positions == LAZY_KEYS_LOCAL;

  if (slot_start[0] != 0) return fail(0, "slot_start[0] must be 0", bad_index, reason);
  for (int32_t r = 0; r < batch; ++r) {
    const int64_t n = (int64_t)slot_start[r + 1] - slot_start[r];
    if (n < 0) return fail(r, "slot_start must be non-decreasing", bad_index, reason);
    if (n > max_slots) return fail(r, "a request has more slots than max_slots", bad_index, reason);
    if (q_pos && (q_pos[r] < 0 || q_pos[r] >= LAZY_MAX_POS)) return fail(r, "query position out of range", bad_index, reason);
  }
  for (int32_t i = 0; i < num_ranges; ++i) {
    const lazy_shared_range_t& rg = ranges[i];
    if (rg.k_offset < 0 || rg.v_offset < 0) return fail(i, "range offsets must be >= 0", bad_index, reason);
    if ((rg.k_offset & 7) || (rg.v_offset & 7))
      return fail(i, "range offsets must be multiples of 8 elements", bad_index, reason);
    if (rg.key_begin < 0 || rg.key_end <= rg.key_begin) return fail(i, "range keys must be non-empty", bad_index, reason);
    if (rg.key_end > rg.k_stride || rg.key_end > rg.v_stride) return fail(i, "range keys beyond the stride", bad_index, reason);
    if (rg.k_offset + ((hkv - 1) * rg.k_stride + rg.key_end) * d > k_pool_elems)
      return fail(i, "range K outside the pool", bad_index, reason);
    if (rg.v_offset + ((hkv - 1) * rg.v_stride + rg.key_end) * d > v_pool_elems)
      return fail(i, "range V outside the pool", bad_index, reason);
  }
  // Every slot of every request must be written by exactly one (item, user) pair: the merge reads all of them.
  const int64_t total_slots = slot_start[batch];
  std::vector<int32_t> writes((size_t)(total_slots > 0 ? total_slots : 0), 0);
  for (int32_t i = 0; i < num_items; ++i) {
    const lazy_shared_item_t& it = items[i];
    if (it.num_ranges < 1 || it.num_ranges > LAZY_SHARED_MAX_RANGES)
      return fail(i, "item num_ranges must be 1..LAZY_SHARED_MAX_RANGES", bad_index, reason);
    if (local && it.num_ranges != 1) return fail(i, "local-position items must be single ranges", bad_index, reason);
    if (it.range_begin < 0 || (int64_t)it.range_begin + it.num_ranges > num_ranges)
      return fail(i, "item ranges outside the range table", bad_index, reason);
    if (it.range_keys < 1) return fail(i, "item range_keys must be >= 1", bad_index, reason);
    if (it.num_ranges > 1 && it.range_keys % 32) return fail(i, "multi-range items need range_keys % 32 == 0", bad_index, reason);
    int64_t keys = 0;
    for (int32_t k = 0; k < it.num_ranges; ++k) {
      const lazy_shared_range_t& rg = ranges[it.range_begin + k];
      const int32_t n = rg.key_end - rg.key_begin;
      if (k + 1 < it.num_ranges ? n != it.range_keys : n > it.range_keys)
        return fail(i, "item range lengths disagree with range_keys", bad_index, reason);
      keys += n;
    }
    if (it.num_users < 1 || it.num_users > 16 / g) return fail(i, "item num_users must be 1..floor(16 / G)", bad_index, reason);
    if (it.user_begin < 0 || (int64_t)it.user_begin + it.num_users > num_users)
      return fail(i, "item users outside the user table", bad_index, reason);
    if (it.reserved != 0) return fail(i, "item reserved field must be 0", bad_index, reason);
    for (int32_t u = it.user_begin; u < it.user_begin + it.num_users; ++u) {
      const lazy_shared_user_t& us = users[u];
      if (us.request < 0 || us.request >= batch) return fail(i, "item user request out of range", bad_index, reason);
      if (us.slot < 0 || us.slot >= slot_start[us.request + 1] - slot_start[us.request])
        return fail(i, "item user slot out of range", bad_index, reason);
      if (us.pos_offset < 0 || us.pos_offset + keys > LAZY_MAX_POS)
        return fail(i, "item user key positions out of range", bad_index, reason);
      ++writes[(size_t)(slot_start[us.request] + us.slot)];
    }
  }
  for (int32_t r = 0; r < batch; ++r)
    for (int32_t s = slot_start[r]; s < slot_start[r + 1]; ++s)
      if (writes[(size_t)s] != 1) return fail(r, "a request slot is not written exactly once", bad_index, reason);
  return LAZY_OK;
}
