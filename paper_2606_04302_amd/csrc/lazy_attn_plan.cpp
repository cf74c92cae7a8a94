// Host planner of the chunk-major shared decode: groups the decode batch's records by the stored keys they read
// and lays out work items (one key range of one stored chunk, up to 16 / G users each) and per-request result slots.
// Pure C++ with no HIP dependency: it runs on host copies of the tables and is testable without a GPU.
#include <stdint.h>

#include <algorithm>
#include <map>
#include <tuple>
#include <vector>

#include "lazy_attn.h"

namespace {

constexpr int kColumns = 16;          // MFMA columns of one decode workgroup: (user, query head) pairs
constexpr int kDefaultItemKeys = 1024;

struct Piece {
  int32_t request, pos_offset, slot;
};

}  // namespace

extern "C" int lazy_shared_decode_plan(const lazy_attn_params_t* p, const lazy_chunk_t* chunks,
                                       const int32_t* chunk_start, int32_t batch, int32_t max_keys_per_item,
                                       lazy_shared_item_t* items, int32_t item_capacity, lazy_shared_user_t* users,
                                       int32_t user_capacity, int32_t* num_items, int32_t* num_users,
                                       int32_t* slot_start) {
  if (num_items) *num_items = 0;
  if (num_users) *num_users = 0;
  if (!p || !chunk_start || !num_items || !num_users || !slot_start || batch < 0 || max_keys_per_item < 0 ||
      item_capacity < 0 || user_capacity < 0)
    return LAZY_EINVAL;
  if (p->num_q_heads <= 0 || p->num_kv_heads <= 0 || p->num_q_heads % p->num_kv_heads != 0) return LAZY_EINVAL;
  const int g = p->num_q_heads / p->num_kv_heads;
  if (g > kColumns) return LAZY_EUNSUPPORTED;
  const int per_item = kColumns / g;
  const int32_t step = max_keys_per_item > 0 ? max_keys_per_item : kDefaultItemKeys;
  if (chunk_start[0] != 0) return LAZY_EINVAL;
  for (int32_t r = 0; r < batch; ++r)
    if (chunk_start[r + 1] < chunk_start[r]) return LAZY_EINVAL;
  if (chunk_start[batch] > 0 && !chunks) return LAZY_EINVAL;

  // Stored key range (k_offset, v_offset, k_stride, v_stride, key_begin, key_end) -> its users, in first-use order.
  using Key = std::tuple<int64_t, int64_t, int32_t, int32_t, int32_t, int32_t>;
  std::map<Key, int32_t> index;
  std::vector<Key> keys;
  std::vector<std::vector<Piece>> groups;
  slot_start[0] = 0;
  for (int32_t r = 0; r < batch; ++r) {
    int32_t slot = 0;
    for (int32_t i = chunk_start[r]; i < chunk_start[r + 1]; ++i) {
      const lazy_chunk_t& c = chunks[i];
      if (c.len < 0) return LAZY_EDATA;
      for (int32_t kb = 0; kb < c.len; kb += step) {
        const Key key{c.k_offset, c.v_offset, c.k_stride, c.v_stride, kb, std::min<int32_t>(c.len, kb + step)};
        auto it = index.find(key);
        if (it == index.end()) {
          it = index.emplace(key, (int32_t)groups.size()).first;
          keys.push_back(key);
          groups.emplace_back();
        }
        groups[it->second].push_back(Piece{r, c.pos_offset, slot++});
      }
    }
    slot_start[r + 1] = slot_start[r] + slot;
  }

  // Longest ranges first, so that the dispatcher starts the heaviest workgroups early.
  std::vector<int32_t> order(groups.size());
  for (size_t k = 0; k < order.size(); ++k) order[k] = (int32_t)k;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return std::get<5>(keys[a]) - std::get<4>(keys[a]) > std::get<5>(keys[b]) - std::get<4>(keys[b]);
  });
  int64_t n_items = 0, n_users = 0;
  for (int32_t k : order) n_items += ((int64_t)groups[k].size() + per_item - 1) / per_item;
  for (const auto& grp : groups) n_users += (int64_t)grp.size();
  if (n_items > INT32_MAX || n_users > INT32_MAX) return LAZY_EUNSUPPORTED;
  *num_items = (int32_t)n_items;
  *num_users = (int32_t)n_users;
  if (n_items > item_capacity || n_users > user_capacity || (n_items > 0 && (!items || !users)))
    return LAZY_EINVAL;

  int32_t it_out = 0, us_out = 0;
  for (int32_t k : order) {
    const Key& key = keys[k];
    const auto& grp = groups[k];
    for (size_t u0 = 0; u0 < grp.size(); u0 += per_item) {
      const int32_t n = (int32_t)std::min<size_t>(per_item, grp.size() - u0);
      lazy_shared_item_t& item = items[it_out++];
      item.k_offset = std::get<0>(key);
      item.v_offset = std::get<1>(key);
      item.k_stride = std::get<2>(key);
      item.v_stride = std::get<3>(key);
      item.key_begin = std::get<4>(key);
      item.key_end = std::get<5>(key);
      item.user_begin = us_out;
      item.num_users = n;
      for (int32_t u = 0; u < n; ++u) {
        const Piece& pc = grp[u0 + u];
        users[us_out++] = lazy_shared_user_t{pc.request, pc.pos_offset, pc.slot, 0};
      }
    }
  }
  return LAZY_OK;
}
