// Session-consistent prefix cache of the paged KV pool (host side; prefix caching in the
// serving engine, paper Sec. 4.1 and Sec. 5.3; the cache-hit re-prefill of an agent's
// growing context, Sec. 5.4; a request reuses keys/values only for a prefix whose token IDs
// are exactly the recorded ones, Sec. 4.2).
//
// Blocks of 16 positions. A cached full block is identified by its parent (the cached block
// of the preceding 16 tokens, or none) and its own 16 token IDs, so a chain of matches is
// an exact match of the whole prefix. Cached blocks form a tree; dropping a block's entry
// drops the entries of its subtree. Allocation takes the lowest free block id; when none is
// free, the least recently released cached block without references is evicted. The pool
// owns no device memory: it hands out block ids for the caller's block tables.
#include <array>
#include <cstdint>
#include <cstring>
#include <list>
#include <set>
#include <unordered_map>
#include <vector>

#include "internal.h"

namespace {

constexpr int kBS = 16;

struct Key {
  int parent;
  std::array<int32_t, kBS> t;
  bool operator==(const Key& o) const { return parent == o.parent && t == o.t; }
};

struct KeyHash {
  size_t operator()(const Key& k) const {
    uint64_t h = 1469598103934665603ull ^ uint64_t(uint32_t(k.parent));
    h *= 1099511628211ull;
    for (int32_t v : k.t) {
      h ^= uint64_t(uint32_t(v));
      h *= 1099511628211ull;
    }
    return size_t(h);
  }
};

Key make_key(int parent, const int32_t* toks) {
  Key k;
  k.parent = parent;
  std::memcpy(k.t.data(), toks, sizeof(int32_t) * kBS);
  return k;
}

}  // namespace

struct molt_prefix_cache {
  int n = 0;
  std::vector<int> ref;
  std::vector<char> cached;
  std::vector<Key> key;                       // of each cached block
  std::vector<std::vector<int>> children;     // cached blocks whose parent is this block
  std::unordered_map<Key, int, KeyHash> map;
  std::set<int> free;
  std::list<int> lru;                         // cached, no references; least recent first
  std::vector<std::list<int>::iterator> lru_at;
  std::vector<char> in_lru;
  long long lookup_tokens = 0, hit_tokens = 0, evictions = 0;

  explicit molt_prefix_cache(int nb)
      : n(nb), ref(nb, 0), cached(nb, 0), key(nb), children(nb), lru_at(nb), in_lru(nb, 0) {
    for (int b = 0; b < nb; ++b) free.insert(b);
  }

  void lru_remove(int b) {
    if (in_lru[b]) {
      lru.erase(lru_at[b]);
      in_lru[b] = 0;
    }
  }

  // drops the entry of block v and of every block cached under it
  void drop(int v) {
    std::vector<int> stack{v}, sub;
    while (!stack.empty()) {
      const int b = stack.back();
      stack.pop_back();
      sub.push_back(b);
      for (int c : children[b]) stack.push_back(c);
    }
    const int p = key[v].parent;
    if (p >= 0) {
      auto& ch = children[p];
      for (size_t i = 0; i < ch.size(); ++i)
        if (ch[i] == v) { ch.erase(ch.begin() + long(i)); break; }
    }
    for (int b : sub) {
      map.erase(key[b]);
      cached[b] = 0;
      children[b].clear();
      if (ref[b] == 0) {
        lru_remove(b);
        free.insert(b);
      }
    }
  }

  void release_row(const int32_t* row, int nb) {
    for (int i = nb - 1; i >= 0; --i) {
      const int b = row[i];
      if (--ref[b] == 0) {
        if (cached[b]) {
          lru.push_back(b);
          lru_at[b] = std::prev(lru.end());
          in_lru[b] = 1;
        } else {
          free.insert(b);
        }
      }
    }
  }
};

extern "C" {

molt_prefix_cache* molt_prefix_cache_create(int num_blocks) {
  if (num_blocks < 1) return nullptr;
  return new molt_prefix_cache(num_blocks);
}

void molt_prefix_cache_destroy(molt_prefix_cache* c) { delete c; }

int molt_prefix_cache_acquire(molt_prefix_cache* c, const int32_t* tokens, int n, int extra_tokens,
                              int32_t* block_table, int max_blocks, int* n_cached) {
  if (!c || !tokens || !block_table || !n_cached || n < 1 || extra_tokens < 0 || max_blocks < 1)
    return MOLT_ERR_INVALID_ARG;
  const long need = (long(n) + extra_tokens + kBS - 1) / kBS;
  if (need > max_blocks) return MOLT_ERR_INVALID_ARG;
  std::vector<int32_t> row;
  int parent = -1;
  for (int i = 0; i < (n - 1) / kBS; ++i) {   // at least one position is left to compute
    auto it = c->map.find(make_key(parent, tokens + long(i) * kBS));
    if (it == c->map.end()) break;
    row.push_back(it->second);
    parent = it->second;
  }
  const int hits = int(row.size());
  for (int b : row) {
    if (c->ref[b] == 0) c->lru_remove(b);
    ++c->ref[b];
  }
  // Only free blocks and unreferenced cached blocks can be handed out; when they cannot
  // cover the request, fail before evicting anything, so no cached prefix is lost.
  if (need - hits > long(c->free.size() + c->lru.size())) {
    c->release_row(row.data(), hits);
    return MOLT_ERR_CAPACITY;
  }
  while (long(row.size()) < need) {
    if (c->free.empty()) {                    // the evicted block itself becomes free
      ++c->evictions;
      c->drop(c->lru.front());
    }
    const int b = *c->free.begin();
    c->free.erase(c->free.begin());
    ++c->ref[b];
    row.push_back(b);
  }
  for (int i = 0; i < max_blocks; ++i) block_table[i] = i < need ? row[i] : -1;
  *n_cached = kBS * hits;
  c->lookup_tokens += n;
  c->hit_tokens += kBS * hits;
  return int(need);
}

int molt_prefix_cache_commit(molt_prefix_cache* c, const int32_t* tokens, int n,
                             const int32_t* block_table, int n_blocks) {
  if (!c || !tokens || !block_table || n < 0 || n_blocks < 0) return MOLT_ERR_INVALID_ARG;
  const int full = n / kBS < n_blocks ? n / kBS : n_blocks;
  for (int i = 0; i < full; ++i)
    if (block_table[i] < 0 || block_table[i] >= c->n || c->ref[block_table[i]] == 0)
      return MOLT_ERR_INVALID_ARG;
  int parent = -1;
  for (int i = 0; i < full; ++i) {
    const Key k = make_key(parent, tokens + long(i) * kBS);
    auto it = c->map.find(k);
    if (it != c->map.end()) {                 // this prefix is cached already (maybe elsewhere)
      parent = it->second;
      continue;
    }
    const int b = block_table[i];
    if (c->cached[b]) break;                  // held under another prefix: stop the chain
    c->cached[b] = 1;
    c->key[b] = k;
    c->map.emplace(k, b);
    if (parent >= 0) c->children[parent].push_back(b);
    parent = b;
  }
  return MOLT_OK;
}

int molt_prefix_cache_release(molt_prefix_cache* c, const int32_t* block_table, int n_blocks) {
  if (!c || !block_table || n_blocks < 0) return MOLT_ERR_INVALID_ARG;
  for (int i = 0; i < n_blocks; ++i)
    if (block_table[i] < 0 || block_table[i] >= c->n || c->ref[block_table[i]] == 0)
      return MOLT_ERR_INVALID_ARG;
  c->release_row(block_table, n_blocks);
  return MOLT_OK;
}

int molt_prefix_cache_stats(const molt_prefix_cache* c, long long* out) {
  if (!c || !out) return MOLT_ERR_INVALID_ARG;
  long long referenced = 0;
  for (int b = 0; b < c->n; ++b) referenced += c->ref[b] > 0;
  out[0] = static_cast<long long>(c->free.size());
  out[1] = static_cast<long long>(c->map.size());
  out[2] = referenced;
  out[3] = static_cast<long long>(c->lru.size());
  out[4] = c->lookup_tokens;
  out[5] = c->hit_tokens;
  out[6] = c->evictions;
  return MOLT_OK;
}

}  // extern "C"
