// Position-agnostic chunk pool: a host-side LRU directory over a fixed number of equal-size slots of a device KV
// region.  Entries are keyed by a 64-bit id; with position-free storage the id is the document alone, so one slot
// serves every request and every offset (the position-agnostic cache of Sec. 2 "Hit-ratio impact under limited
// cache capacity"); a position-aware cache would have to key by (document, position).  Pure C++, no HIP.
#include <stdint.h>

#include <new>
#include <unordered_map>
#include <vector>

#include "lazy_attn.h"

struct lazy_pool {
  struct Node {
    uint64_t key;
    int32_t prev, next;  // LRU list (most recent at head), -1 = none
    bool used;
  };
  std::vector<Node> nodes;                    // one per slot
  std::unordered_map<uint64_t, int32_t> map;  // key -> slot
  std::vector<int32_t> free_slots;
  int32_t head = -1, tail = -1;
  int64_t lookups = 0, hits = 0, evictions = 0;

  void unlink(int32_t s) {
    Node& n = nodes[s];
    if (n.prev >= 0) nodes[n.prev].next = n.next; else head = n.next;
    if (n.next >= 0) nodes[n.next].prev = n.prev; else tail = n.prev;
    n.prev = n.next = -1;
  }
  void push_front(int32_t s) {
    Node& n = nodes[s];
    n.prev = -1;
    n.next = head;
    if (head >= 0) nodes[head].prev = s;
    head = s;
    if (tail < 0) tail = s;
  }
};

extern "C" {

lazy_pool_t* lazy_pool_create(int32_t capacity_slots) {
  if (capacity_slots <= 0) return nullptr;
  lazy_pool_t* p = new (std::nothrow) lazy_pool_t();
  if (!p) return nullptr;
  try {
    p->nodes.assign(capacity_slots, lazy_pool::Node{0, -1, -1, false});
    p->free_slots.reserve(capacity_slots);
    for (int32_t s = capacity_slots - 1; s >= 0; --s) p->free_slots.push_back(s);
    p->map.reserve((size_t)capacity_slots * 2);
  } catch (...) {
    delete p;
    return nullptr;
  }
  return p;
}

void lazy_pool_destroy(lazy_pool_t* p) { delete p; }

int lazy_pool_acquire(lazy_pool_t* p, uint64_t key, int32_t* slot, int32_t* hit, uint64_t* evicted_key,
                      int32_t* evicted) {
  if (!p || !slot || !hit) return LAZY_EINVAL;
  ++p->lookups;
  if (evicted) *evicted = 0;
  auto it = p->map.find(key);
  if (it != p->map.end()) {
    ++p->hits;
    *hit = 1;
    *slot = it->second;
    p->unlink(it->second);
    p->push_front(it->second);
    return LAZY_OK;
  }
  *hit = 0;
  int32_t s;
  if (!p->free_slots.empty()) {
    s = p->free_slots.back();
    p->free_slots.pop_back();
  } else {
    s = p->tail;  // least recently used
    p->unlink(s);
    p->map.erase(p->nodes[s].key);
    ++p->evictions;
    if (evicted) *evicted = 1;
    if (evicted_key) *evicted_key = p->nodes[s].key;
  }
  p->nodes[s].key = key;
  p->nodes[s].used = true;
  p->push_front(s);
  try {
    p->map.emplace(key, s);
  } catch (...) {
    return LAZY_EINVAL;
  }
  *slot = s;
  return LAZY_OK;
}

int lazy_pool_stats(const lazy_pool_t* p, int64_t* lookups, int64_t* hits, int64_t* evictions, int32_t* resident) {
  if (!p) return LAZY_EINVAL;
  if (lookups) *lookups = p->lookups;
  if (hits) *hits = p->hits;
  if (evictions) *evictions = p->evictions;
  if (resident) *resident = (int32_t)p->map.size();
  return LAZY_OK;
}

}  // extern "C"
