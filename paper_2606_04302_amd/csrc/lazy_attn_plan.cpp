// Host planner of the chunk-major shared decode: groups the decode batch's records by the stored keys they read,
// chains groups that all of their users read back to back (the blocks of one chunk in a paged store) into runs, and
// lays out work items (one run, up to 16 / G users each), their key ranges and per-request result slots.
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
constexpr int kTileKeys = 32;         // decode tile: every range of a run but the last holds whole tiles

// One use of a piece: request, record index in the flat table, position of the piece's first key.
struct Use {
  int32_t request, record, pos;
};
// Stored key range: k_offset, v_offset, k_stride, v_stride, key_begin, key_end.
using Key = std::tuple<int64_t, int64_t, int32_t, int32_t, int32_t, int32_t>;
struct Group {
  Key key;
  std::vector<Use> uses;  // in table order (request, then record)
  bool whole = true;      // every use covers its whole record
  int32_t keys() const { return std::get<5>(key) - std::get<4>(key); }
};
struct Run {
  std::vector<int32_t> groups;
  int64_t keys = 0;
};

}  // namespace

extern "C" int lazy_shared_decode_plan(const lazy_attn_params_t* p, const lazy_chunk_t* chunks,
                                       const int32_t* chunk_start, int32_t batch, int32_t max_keys_per_item,
                                       lazy_shared_item_t* items, int32_t item_capacity, lazy_shared_range_t* ranges,
                                       int32_t range_capacity, lazy_shared_user_t* users, int32_t user_capacity,
                                       int32_t* num_items, int32_t* num_ranges, int32_t* num_users,
                                       int32_t* slot_start) {
  if (num_items) *num_items = 0;
  if (num_ranges) *num_ranges = 0;
  if (num_users) *num_users = 0;
  if (!p || !chunk_start || !num_items || !num_ranges || !num_users || !slot_start || batch < 0 ||
      max_keys_per_item < 0 || item_capacity < 0 || range_capacity < 0 || user_capacity < 0)
    return LAZY_EINVAL;
  if (p->num_q_heads <= 0 || p->num_kv_heads <= 0 || p->num_q_heads % p->num_kv_heads != 0) return LAZY_EINVAL;
  const int g = p->num_q_heads / p->num_kv_heads;
  if (g > kColumns) return LAZY_EUNSUPPORTED;
  const int per_item = kColumns / g;
  const int32_t step = max_keys_per_item > 0 ? max_keys_per_item : kDefaultItemKeys;
  if (chunk_start[0] != 0) return LAZY_EINVAL;
  for (int32_t r = 0; r < batch; ++r)
    if (chunk_start[r + 1] < chunk_start[r]) return LAZY_EINVAL;
  const int32_t n_records = chunk_start[batch];
  if (n_records > 0 && !chunks) return LAZY_EINVAL;

  // 1. Pieces of at most `step` keys, grouped by the stored keys they read.
  std::map<Key, int32_t> index;
  std::vector<Group> groups;
  std::vector<int32_t> first_piece(n_records, -1);  // group of each record's first piece
  for (int32_t r = 0; r < batch; ++r) {
    for (int32_t i = chunk_start[r]; i < chunk_start[r + 1]; ++i) {
      const lazy_chunk_t& c = chunks[i];
      if (c.len < 0) return LAZY_EDATA;
      for (int32_t kb = 0; kb < c.len; kb += step) {
        const int32_t ke = std::min<int32_t>(c.len, kb + step);
        const Key key{c.k_offset, c.v_offset, c.k_stride, c.v_stride, kb, ke};
        auto it = index.find(key);
        if (it == index.end()) {
          it = index.emplace(key, (int32_t)groups.size()).first;
          groups.emplace_back();
          groups.back().key = key;
        }
        Group& grp = groups[it->second];
        grp.uses.push_back(Use{r, i, c.pos_offset + kb});
        if (kb > 0 || ke < c.len) grp.whole = false;
        if (kb == 0) first_piece[i] = it->second;
      }
    }
  }

  // 2. Successor of each group: the group every one of its users reads next, at the next position.  Only for a NoPE
  //    store (keys rotated by their index in the run); a local-position store encodes keys per record.
  std::vector<int32_t> succ(groups.size(), -1);
  if (p->key_positions == LAZY_KEYS_NOPE) {
    for (size_t a = 0; a < groups.size(); ++a) {
      const Group& A = groups[a];
      const int32_t la = A.keys();
      if (!A.whole || la % kTileKeys != 0) continue;
      const Use& u0 = A.uses[0];
      if (u0.record + 1 >= chunk_start[u0.request + 1]) continue;
      const int32_t b = first_piece[u0.record + 1];
      if (b < 0 || b == (int32_t)a) continue;
      const Group& B = groups[b];
      if (!B.whole || B.keys() > la || B.uses.size() != A.uses.size()) continue;
      bool ok = true;
      for (size_t k = 0; ok && k < A.uses.size(); ++k)
        ok = B.uses[k].request == A.uses[k].request && B.uses[k].record == A.uses[k].record + 1 &&
             (int64_t)B.uses[k].pos == (int64_t)A.uses[k].pos + la;
      if (ok) succ[a] = b;
    }
  }
  // Runs: follow successors from every group not yet taken (a group's successor is created after it, so scanning in
  // creation order meets every run at its start); all ranges but the last have the first one's length.
  std::vector<int32_t> run_of(groups.size(), -1);
  std::vector<Run> runs;
  for (size_t g0 = 0; g0 < groups.size(); ++g0) {
    if (run_of[g0] >= 0) continue;
    Run run;
    const int32_t rk = groups[g0].keys();
    for (int32_t cur = (int32_t)g0; cur >= 0 && run_of[cur] < 0; cur = succ[cur]) {
      const int32_t len = groups[cur].keys();
      if (!run.groups.empty() &&
          (len > rk || run.keys + len > step || (int)run.groups.size() >= LAZY_SHARED_MAX_RANGES))
        break;
      run.groups.push_back(cur);
      run_of[cur] = (int32_t)runs.size();
      run.keys += len;
      if (len != rk) break;
    }
    runs.push_back(std::move(run));
  }

  // 3. One slot per (request, run).
  std::vector<int32_t> nslots(batch, 0);
  std::vector<std::vector<int32_t>> run_slots(runs.size());
  for (size_t k = 0; k < runs.size(); ++k)
    for (const Use& u : groups[runs[k].groups[0]].uses) run_slots[k].push_back(nslots[u.request]++);
  slot_start[0] = 0;
  for (int32_t r = 0; r < batch; ++r) slot_start[r + 1] = slot_start[r] + nslots[r];

  // 4. Items, longest run first (the dispatcher starts the heaviest workgroups early).
  std::vector<int32_t> order(runs.size());
  for (size_t k = 0; k < order.size(); ++k) order[k] = (int32_t)k;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return runs[a].keys > runs[b].keys; });
  int64_t n_items = 0, n_ranges = 0, n_users = 0;
  for (const Run& run : runs) {
    const int64_t nu = (int64_t)groups[run.groups[0]].uses.size();
    n_items += (nu + per_item - 1) / per_item;
    n_ranges += (int64_t)run.groups.size();
    n_users += nu;
  }
  if (n_items > INT32_MAX || n_ranges > INT32_MAX || n_users > INT32_MAX) return LAZY_EUNSUPPORTED;
  *num_items = (int32_t)n_items;
  *num_ranges = (int32_t)n_ranges;
  *num_users = (int32_t)n_users;
  if (n_items > item_capacity || n_ranges > range_capacity || n_users > user_capacity ||
      (n_items > 0 && (!items || !ranges || !users)))
    return LAZY_EINVAL;

  int32_t it_out = 0, rg_out = 0, us_out = 0;
  for (int32_t k : order) {
    const Run& run = runs[k];
    const int32_t range_begin = rg_out;
    for (int32_t gi : run.groups) {
      const Key& key = groups[gi].key;
      ranges[rg_out++] = lazy_shared_range_t{std::get<0>(key), std::get<1>(key), std::get<2>(key),
                                             std::get<3>(key), std::get<4>(key), std::get<5>(key)};
    }
    const std::vector<Use>& uses = groups[run.groups[0]].uses;
    for (size_t u0 = 0; u0 < uses.size(); u0 += per_item) {
      const int32_t n = (int32_t)std::min<size_t>(per_item, uses.size() - u0);
      items[it_out++] = lazy_shared_item_t{range_begin, (int32_t)run.groups.size(), groups[run.groups[0]].keys(),
                                           us_out, n, 0};
      for (int32_t u = 0; u < n; ++u) {
        const Use& use = uses[u0 + u];
        users[us_out++] = lazy_shared_user_t{use.request, use.pos, run_slots[k][u0 + u], 0};
      }
    }
  }
  return LAZY_OK;
}

// Chunk table in storage order: each request's records, stably sorted by k_offset.  The attention a request gets is
// fixed by its records' positions, not by their order in the table, so only the traversal order changes.
extern "C" int lazy_chunk_table_storage_order(const lazy_chunk_t* chunks, const int32_t* chunk_start, int32_t batch,
                                              lazy_chunk_t* out) {
  if (!chunk_start || batch < 0 || chunk_start[0] != 0) return LAZY_EINVAL;
  for (int32_t r = 0; r < batch; ++r)
    if (chunk_start[r + 1] < chunk_start[r]) return LAZY_EINVAL;
  const int32_t n = chunk_start[batch];
  if (n == 0) return LAZY_OK;
  if (!chunks || !out) return LAZY_EINVAL;
  if (out != chunks) std::copy(chunks, chunks + n, out);
  for (int32_t r = 0; r < batch; ++r)
    std::stable_sort(out + chunk_start[r], out + chunk_start[r + 1],
                     [](const lazy_chunk_t& a, const lazy_chunk_t& b) { return a.k_offset < b.k_offset; });
  return LAZY_OK;
}
