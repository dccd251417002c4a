// Host radix cache: radix tree over token ids, reference counters, LRU leaf
// eviction and the shared FIFO slot pool (section 3 of the SGLang paper and
// Algorithm 1).  Semantics, including where the paper is silent:
//  * match_prefix and insert each advance a logical clock once and stamp
//    every node they walk ("used" for LRU);
//  * eviction takes the unreferenced leaf with the smallest (stamp, id),
//    frees whole leaves, and re-examines a parent that becomes a leaf;
//  * a match ending inside an edge splits it; a split keeps the old id for
//    the lower part, gives the upper part the next id, the old counter and
//    the old stamp;
//  * a reference lock covers the whole root-to-node path;
//  * insert keeps cached slots and frees caller slots that differ from them;
//  * the pool is a FIFO queue with a caller-given initial order.
//
// Data layout for large trees (hundreds of thousands of operations over
// millions of tokens, where requests that end inside shared text cut the
// shared edges into runs of a few tokens, so a walk crosses hundreds of
// edges): nodes live in a vector indexed by id, one cache line each, with
// the edge's tokens and slots in one buffer; the child edge index is one
// open-addressing table keyed by (parent id, first token), whose entry for
// the next edge is fetched while the current edge is compared; the free map
// is one bit per slot; the evictable leaves are an ordered set keyed by
// (stamp, id), kept current on every change, so eviction never scans the
// tree.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <deque>
#include <memory>
#include <set>
#include <string>
#include <vector>

#include "radixattn.h"
#include "ra_error.h"

namespace {

struct alignas(64) Node {
  int64_t parent = -1;
  uint64_t stamp = 0;
  uint64_t lru_stamp = 0;  // stamp it was filed under
  int64_t ref = 0;
  int32_t len = 0;         // tokens on the edge into this node
  int32_t n_children = 0;
  bool alive = false;
  bool in_lru = false;     // present in the evictable-leaf set
  std::unique_ptr<int32_t[]> kv;  // the edge's tokens, then their slots
  const int32_t* key() const { return kv.get(); }
  const int32_t* slots() const { return kv.get() + len; }
  void assign(const int32_t* k, const int32_t* s, int64_t n) {
    std::unique_ptr<int32_t[]> b(new int32_t[2 * n]);
    std::memcpy(b.get(), k, n * sizeof(int32_t));
    std::memcpy(b.get() + n, s, n * sizeof(int32_t));
    kv = std::move(b);
    len = static_cast<int32_t>(n);
  }
};

inline uint64_t edge_key(int64_t parent, int32_t tok) {
  return (static_cast<uint64_t>(parent) << 32) ^ static_cast<uint32_t>(tok);
}

// Open-addressing map from edge key to child id: linear probing over a
// power-of-two table at most 3/4 full, deletion by backward shift (no
// tombstones).  The slot hash is the first xor-shift-multiply round of
// MurmurHash3's 64-bit finalizer.  Keys are below 2^63 (node ids < 2^31), so
// the all-ones word marks an empty entry.
class EdgeMap {
 public:
  EdgeMap() { rehash(1024); }
  int64_t find(uint64_t k) const {
    size_t i = slot(k);
    for (;;) {
      const Entry& e = tab_[i];
      if (e.key == k) return e.val;
      if (e.key == kEmpty) return -1;
      i = (i + 1) & mask_;
    }
  }
  void set(uint64_t k, int64_t v) {
    if ((size_ + 1) * 4 > tab_.size() * 3) rehash(tab_.size() * 2);
    size_t i = slot(k);
    for (;;) {
      Entry& e = tab_[i];
      if (e.key == k) { e.val = v; return; }
      if (e.key == kEmpty) { e.key = k; e.val = v; ++size_; return; }
      i = (i + 1) & mask_;
    }
  }
  void erase(uint64_t k) {
    size_t i = slot(k);
    for (;;) {
      if (tab_[i].key == kEmpty) return;
      if (tab_[i].key == k) break;
      i = (i + 1) & mask_;
    }
    // shift later members of the probe run back into the hole
    size_t hole = i;
    for (size_t j = (i + 1) & mask_;; j = (j + 1) & mask_) {
      if (tab_[j].key == kEmpty) break;
      size_t home = slot(tab_[j].key);
      // j's entry may fill the hole if its home is not in (hole, j]
      bool movable = hole <= j ? (home <= hole || home > j) : (home <= hole && home > j);
      if (movable) { tab_[hole] = tab_[j]; hole = j; }
    }
    tab_[hole].key = kEmpty;
    --size_;
  }
  // starts fetching the probe run of k (a lookup that follows soon)
  void prefetch(uint64_t k) const { __builtin_prefetch(&tab_[slot(k)]); }
 private:
  static constexpr uint64_t kEmpty = ~0ull;
  struct Entry { uint64_t key; int64_t val; };
  size_t slot(uint64_t k) const {
    k ^= k >> 33; k *= 0xff51afd7ed558ccdull; k ^= k >> 33;
    return static_cast<size_t>(k) & mask_;
  }
  void rehash(size_t cap) {
    std::vector<Entry> old;
    old.swap(tab_);
    tab_.assign(cap, Entry{kEmpty, 0});
    mask_ = cap - 1;
    size_ = 0;
    for (const Entry& e : old)
      if (e.key != kEmpty) set(e.key, e.val);
  }
  std::vector<Entry> tab_;
  size_t mask_ = 0, size_ = 0;
};

// One bit per pool slot: set while the slot is in the free queue.
class SlotBits {
 public:
  void reset(size_t n) { w_.assign((n + 63) / 64, 0); }
  bool get(int32_t s) const { return (w_[static_cast<uint32_t>(s) >> 6] >> (s & 63)) & 1; }
  void set(int32_t s) { w_[static_cast<uint32_t>(s) >> 6] |= 1ull << (s & 63); }
  void clr(int32_t s) { w_[static_cast<uint32_t>(s) >> 6] &= ~(1ull << (s & 63)); }
 private:
  std::vector<uint64_t> w_;
};

}  // namespace

struct ra_cache {
  int64_t pool_slots = 0;
  // FIFO free queue as a ring buffer of capacity pool_slots
  std::vector<int32_t> ring;
  int64_t head = 0, count = 0;
  SlotBits is_free;

  std::vector<Node> nodes;
  EdgeMap children;  // (parent, first token) -> child
  std::set<std::pair<uint64_t, int64_t>> lru;      // evictable leaves
  uint64_t clock = 0;
  int64_t live = 1;
  int64_t evictable = 0;  // tokens in unreferenced live nodes
  int64_t cached = 0;     // tokens in live nodes

  // Optional eviction log (for a data-parallel router that mirrors this
  // tree): per evicted leaf, its root-to-leaf tokens and its own length.
  struct Evicted {
    std::vector<int32_t> path;
    int64_t len;
  };
  bool log_evictions = false;
  std::deque<Evicted> eviction_log;

  bool evictable_leaf(int64_t id) const {
    const Node& n = nodes[id];
    return id != 0 && n.alive && n.ref == 0 && n.n_children == 0;
  }
  void refresh(int64_t id) {
    Node& n = nodes[id];
    bool want = evictable_leaf(id);
    if (n.in_lru && (!want || n.lru_stamp != n.stamp)) {
      lru.erase({n.lru_stamp, id});
      n.in_lru = false;
    }
    if (want && !n.in_lru) {
      lru.insert({n.stamp, id});
      n.in_lru = true;
      n.lru_stamp = n.stamp;
    }
  }

  // ---- pool ----
  // (head and count stay in [0, pool_slots]: wrap by one comparison, no
  // division per slot)
  void push_free(int32_t s) {
    int64_t at = head + count;
    if (at >= pool_slots) at -= pool_slots;
    ring[at] = s;
    ++count;
    is_free.set(s);
  }
  int32_t pop_free() {
    int32_t s = ring[head];
    if (++head == pool_slots) head = 0;
    --count;
    is_free.clr(s);
    return s;
  }

  // ---- tree ----
  // Appends a node.  key and slots are taken by value: callers may pass
  // views into another node, which the vector growth below would invalidate.
  int64_t new_node(int64_t parent, const int32_t* key, const int32_t* slots, int64_t len,
                   int64_t ref, uint64_t stamp) {
    int64_t id = static_cast<int64_t>(nodes.size());
    nodes.emplace_back();
    Node& n = nodes.back();
    n.parent = parent;
    n.assign(key, slots, len);
    n.ref = ref;
    n.stamp = stamp;
    n.alive = true;
    ++live;
    return id;
  }

  // Splits node x after c tokens; returns the new upper node.
  int64_t split(int64_t x, int64_t c) {
    int64_t par = nodes[x].parent;
    int32_t first = nodes[x].key()[0];
    int64_t y = new_node(par, nodes[x].key(), nodes[x].slots(), c, nodes[x].ref, nodes[x].stamp);
    Node& X = nodes[x];
    Node& Y = nodes[y];
    X.assign(X.key() + c, X.slots() + c, X.len - c);
    X.parent = y;
    Y.n_children = 1;
    children.set(edge_key(par, first), y);
    children.set(edge_key(y, X.key()[0]), x);
    refresh(x);
    refresh(y);
    return y;
  }

  // Walks tokens from the root; calls visit(node, pos) on every matched node.
  template <class F>
  int64_t walk(const int32_t* tok, int64_t n, int64_t* out_pos, F&& visit) {
    ++clock;
    int64_t node = 0, pos = 0;
    while (pos < n) {
      int64_t ch = children.find(edge_key(node, tok[pos]));
      if (ch < 0) break;
      const Node& cn = nodes[ch];
      const int32_t* key = cn.key();
      const int64_t klen = cn.len;
      if (pos + klen < n) children.prefetch(edge_key(ch, tok[pos + klen]));
      __builtin_prefetch(key);
      int64_t lim = std::min<int64_t>(klen, n - pos);
      int64_t c = 0;
      while (c < lim && key[c] == tok[pos + c]) ++c;
      if (c < klen) ch = split(ch, c);
      nodes[ch].stamp = clock;
      refresh(ch);
      visit(ch, pos);
      pos += c;
      node = ch;
    }
    *out_pos = pos;
    return node;
  }
};

extern "C" {

int ra_cache_create(int64_t pool_slots, const int32_t* order, ra_cache** out) {
  return ra_guard("ra_cache_create", [&]() -> int {
    if (!out) return ra_fail(RA_EINVAL, "ra_cache_create: out is NULL");
    if (pool_slots < 0 || pool_slots > INT32_MAX)
      return ra_fail(RA_EINVAL, "ra_cache_create: pool_slots out of range");
    std::unique_ptr<ra_cache> c(new ra_cache());
    c->pool_slots = pool_slots;
    c->ring.resize(static_cast<size_t>(pool_slots));
    c->is_free.reset(static_cast<size_t>(pool_slots));
    for (int64_t i = 0; i < pool_slots; ++i) {
      int32_t s = order ? order[i] : static_cast<int32_t>(i);
      if (s < 0 || s >= pool_slots || c->is_free.get(s))
        return ra_fail(RA_EINVAL, "ra_cache_create: initial order is not a permutation");
      c->push_free(s);
    }
    c->nodes.emplace_back();  // root
    c->nodes[0].alive = true;
    *out = c.release();
    return ra_ok();
  });
}

void ra_cache_destroy(ra_cache* c) { delete c; }

// A match creates at most one node (a split) and an insert at most two (a
// split and the new leaf); ids stay below 2^31, which the child table's keys
// rely on.
static bool ids_left(const ra_cache* c, int64_t need) {
  return static_cast<int64_t>(c->nodes.size()) + need <= INT32_MAX;
}

int ra_match_prefix(ra_cache* c, const int32_t* tokens, int64_t n, int32_t* out_slots,
                    int64_t* out_len, int64_t* out_node) {
  return ra_guard("ra_match_prefix", [&]() -> int {
    if (!c || n < 0 || (n > 0 && !tokens)) return ra_fail(RA_EINVAL, "ra_match_prefix: bad argument");
    if (!ids_left(c, 1)) return ra_fail(RA_ENOMEM, "ra_match_prefix: node ids exhausted (2^31 created)");
    int64_t pos = 0;
    int64_t node = c->walk(tokens, n, &pos, [&](int64_t ch, int64_t p) {
      if (out_slots) {
        const Node& nd = c->nodes[ch];
        std::memcpy(out_slots + p, nd.slots(), nd.len * sizeof(int32_t));
      }
    });
    if (out_len) *out_len = pos;
    if (out_node) *out_node = node;
    return ra_ok();
  });
}

static bool valid_node(const ra_cache* c, int64_t node) {
  return node >= 0 && node < static_cast<int64_t>(c->nodes.size()) && c->nodes[node].alive;
}

int ra_inc_ref(ra_cache* c, int64_t node, int64_t* out_delta) {
  return ra_guard("ra_inc_ref", [&]() -> int {
    if (!c || !valid_node(c, node)) return ra_fail(RA_EINVAL, "ra_inc_ref: unknown node");
    int64_t delta = 0;
    for (int64_t x = node; x != 0; x = c->nodes[x].parent) {
      Node& n = c->nodes[x];
      if (n.ref == 0) {
        delta -= n.len;
      }
      ++n.ref;
      c->refresh(x);
    }
    c->evictable += delta;
    if (out_delta) *out_delta = delta;
    return ra_ok();
  });
}

int ra_dec_ref(ra_cache* c, int64_t node, int64_t* out_delta) {
  return ra_guard("ra_dec_ref", [&]() -> int {
    if (!c || !valid_node(c, node)) return ra_fail(RA_EINVAL, "ra_dec_ref: unknown node");
    for (int64_t x = node; x != 0; x = c->nodes[x].parent)
      if (c->nodes[x].ref == 0) return ra_fail(RA_EINVAL, "ra_dec_ref: reference counter underflow");
    int64_t delta = 0;
    for (int64_t x = node; x != 0; x = c->nodes[x].parent) {
      Node& n = c->nodes[x];
      if (--n.ref == 0) delta += n.len;
      c->refresh(x);
    }
    c->evictable += delta;
    if (out_delta) *out_delta = delta;
    return ra_ok();
  });
}

int ra_alloc_slots(ra_cache* c, int64_t n, int32_t* out_slots) {
  return ra_guard("ra_alloc_slots", [&]() -> int {
    if (!c || n < 0 || (n > 0 && !out_slots)) return ra_fail(RA_EINVAL, "ra_alloc_slots: bad argument");
    if (n > c->count) return ra_fail(RA_ENOMEM, "ra_alloc_slots: not enough free slots");
    // the front n entries of the ring, in at most two runs
    const int64_t first = std::min<int64_t>(n, c->pool_slots - c->head);
    std::memcpy(out_slots, c->ring.data() + c->head, static_cast<size_t>(first) * sizeof(int32_t));
    std::memcpy(out_slots + first, c->ring.data(), static_cast<size_t>(n - first) * sizeof(int32_t));
    for (int64_t i = 0; i < n; ++i) c->is_free.clr(out_slots[i]);
    c->head += n;
    if (c->head >= c->pool_slots) c->head -= c->pool_slots;
    c->count -= n;
    return ra_ok();
  });
}

static int check_freeable(ra_cache* c, const int32_t* slots, int64_t n, const char* who) {
  // every slot in range, currently allocated, and not repeated
  for (int64_t i = 0; i < n; ++i) {
    int32_t s = slots[i];
    if (s < 0 || s >= c->pool_slots || c->is_free.get(s))
      return ra_fail(RA_EINVAL, std::string(who) + ": slot out of range or already free");
  }
  // Repeats: mark each slot in the free map (all are allocated, so unmarked)
  // and find a mark already set; the marks are cleared again either way.
  int64_t i = 0;
  for (; i < n; ++i) {
    if (c->is_free.get(slots[i])) break;
    c->is_free.set(slots[i]);
  }
  for (int64_t j = 0; j < i; ++j) c->is_free.clr(slots[j]);
  if (i < n) return ra_fail(RA_EINVAL, std::string(who) + ": repeated slot");
  return RA_OK;
}

int ra_free_slots(ra_cache* c, const int32_t* slots, int64_t n) {
  return ra_guard("ra_free_slots", [&]() -> int {
    if (!c || n < 0 || (n > 0 && !slots)) return ra_fail(RA_EINVAL, "ra_free_slots: bad argument");
    int st = check_freeable(c, slots, n, "ra_free_slots");
    if (st != RA_OK) return st;
    for (int64_t i = 0; i < n; ++i) c->push_free(slots[i]);
    return ra_ok();
  });
}

int ra_insert(ra_cache* c, const int32_t* tokens, const int32_t* slots, int64_t n,
              int64_t* out_cached, int64_t* out_node) {
  return ra_guard("ra_insert", [&]() -> int {
    if (!c || n < 0 || (n > 0 && (!tokens || !slots))) return ra_fail(RA_EINVAL, "ra_insert: bad argument");
    if (n > INT32_MAX) return ra_fail(RA_EINVAL, "ra_insert: sequence longer than 2^31 - 1 tokens");
    if (!ids_left(c, 2)) return ra_fail(RA_ENOMEM, "ra_insert: node ids exhausted (2^31 created)");
    // One read-only walk records the path and the caller slots that differ
    // from cached ones, and everything is validated before the tree changes;
    // then the recorded path is stamped (and split where the match ends
    // inside an edge) without walking again.
    struct Step {
      int64_t child, matched;
    };
    std::vector<Step> path;
    std::vector<int32_t> dup;
    int64_t pos = 0;
    {
      int64_t node = 0;
      while (pos < n) {
        const int64_t chid = c->children.find(edge_key(node, tokens[pos]));
        if (chid < 0) break;
        const Node& ch = c->nodes[chid];
        if (pos + ch.len < n) c->children.prefetch(edge_key(chid, tokens[pos + ch.len]));
        const int32_t* key = ch.key();
        const int32_t* cs = ch.slots();
        int64_t lim = std::min<int64_t>(ch.len, n - pos);
        int64_t k = 0;
        while (k < lim && key[k] == tokens[pos + k]) {
          if (slots[pos + k] != cs[k]) dup.push_back(slots[pos + k]);
          ++k;
        }
        path.push_back({chid, k});
        pos += k;
        if (k < ch.len) break;
        node = chid;
      }
      if (!dup.empty()) {
        int st = check_freeable(c, dup.data(), static_cast<int64_t>(dup.size()), "ra_insert");
        if (st != RA_OK) return st;
      }
      // slots that will enter the tree must be allocated pool slots
      for (int64_t i = pos; i < n; ++i)
        if (slots[i] < 0 || slots[i] >= c->pool_slots || c->is_free.get(slots[i]))
          return ra_fail(RA_EINVAL, "ra_insert: new slot out of range or free");
    }
    ++c->clock;
    int64_t node = 0;
    for (const Step& st : path) {
      int64_t ch = st.child;
      if (st.matched < c->nodes[ch].len) ch = c->split(ch, st.matched);
      c->nodes[ch].stamp = c->clock;
      c->refresh(ch);
      node = ch;
    }
    for (int32_t s : dup) c->push_free(s);
    int64_t cached = pos;
    if (pos < n) {
      int64_t leaf = c->new_node(node, tokens + pos, slots + pos, n - pos, 0, c->clock);
      c->children.set(edge_key(node, tokens[pos]), leaf);
      c->nodes[node].n_children += 1;
      c->evictable += n - pos;
      c->cached += n - pos;
      c->refresh(node);
      c->refresh(leaf);
      node = leaf;
    }
    if (out_cached) *out_cached = cached;
    if (out_node) *out_node = node;
    return ra_ok();
  });
}

int ra_evict(ra_cache* c, int64_t n_tokens, int64_t* out_freed) {
  return ra_guard("ra_evict", [&]() -> int {
    if (!c) return ra_fail(RA_EINVAL, "ra_evict: cache is NULL");
    int64_t freed = 0;
    while (freed < n_tokens && !c->lru.empty()) {
      int64_t x = c->lru.begin()->second;
      c->lru.erase(c->lru.begin());
      Node& n = c->nodes[x];
      n.in_lru = false;
      if (c->log_evictions) {
        ra_cache::Evicted e;
        e.len = n.len;
        std::vector<int64_t> chain;
        for (int64_t y = x; y != 0; y = c->nodes[y].parent) chain.push_back(y);
        for (auto it = chain.rbegin(); it != chain.rend(); ++it) {
          const Node& a = c->nodes[*it];
          e.path.insert(e.path.end(), a.key(), a.key() + a.len);
        }
        c->eviction_log.push_back(std::move(e));
      }
      const int32_t* ns = n.slots();
      int64_t len = n.len;
      for (int64_t i = 0; i < len; ++i) c->push_free(ns[i]);
      freed += len;
      c->evictable -= len;
      c->cached -= len;
      c->children.erase(edge_key(n.parent, n.key()[0]));
      int64_t par = n.parent;
      n.alive = false;
      n.kv.reset();
      n.len = 0;
      --c->live;
      c->nodes[par].n_children -= 1;
      c->refresh(par);
    }
    if (out_freed) *out_freed = freed;
    return ra_ok();
  });
}

int ra_cache_log_evictions(ra_cache* c, int32_t enable) {
  if (!c) return ra_fail(RA_EINVAL, "ra_cache_log_evictions: cache is NULL");
  c->log_evictions = enable != 0;
  if (!c->log_evictions) c->eviction_log.clear();
  return ra_ok();
}

int ra_eviction_log_pop(ra_cache* c, int32_t* tokens, int64_t cap, int64_t* out_path_len, int64_t* out_evicted_len) {
  return ra_guard("ra_eviction_log_pop", [&]() -> int {
    if (!c || !out_path_len) return ra_fail(RA_EINVAL, "ra_eviction_log_pop: NULL argument");
    if (c->eviction_log.empty()) {
      *out_path_len = -1;
      if (out_evicted_len) *out_evicted_len = 0;
      return ra_ok();
    }
    const auto& e = c->eviction_log.front();
    const int64_t n = static_cast<int64_t>(e.path.size());
    *out_path_len = n;
    if (out_evicted_len) *out_evicted_len = e.len;
    if (!tokens || cap < n) return ra_fail(RA_EINVAL, "ra_eviction_log_pop: token buffer too small");
    std::memcpy(tokens, e.path.data(), sizeof(int32_t) * n);
    c->eviction_log.pop_front();
    return ra_ok();
  });
}

int64_t ra_evictable_size(const ra_cache* c) { return c ? c->evictable : 0; }
int64_t ra_available_size(const ra_cache* c) { return c ? c->count : 0; }
int64_t ra_cached_tokens(const ra_cache* c) { return c ? c->cached : 0; }
int64_t ra_num_nodes(const ra_cache* c) { return c ? c->live : 0; }

int ra_snapshot(const ra_cache* c, int64_t* buf, int64_t cap, int64_t* out_len) {
  return ra_guard("ra_snapshot", [&]() -> int {
    if (!c) return ra_fail(RA_EINVAL, "ra_snapshot: cache is NULL");
    int64_t need = 3 + c->count;
    for (const Node& n : c->nodes)
      if (n.alive) need += 5 + 2 * static_cast<int64_t>(n.len);
    if (out_len) *out_len = need;
    if (!buf) return ra_ok();
    if (cap < need) return ra_fail(RA_EINVAL, "ra_snapshot: buffer too small");
    int64_t* w = buf;
    *w++ = static_cast<int64_t>(c->clock);
    *w++ = c->live;
    *w++ = c->count;
    for (size_t id = 0; id < c->nodes.size(); ++id) {
      const Node& n = c->nodes[id];
      if (!n.alive) continue;
      *w++ = static_cast<int64_t>(id);
      *w++ = n.parent;
      *w++ = n.ref;
      *w++ = static_cast<int64_t>(n.stamp);
      *w++ = n.len;
      for (int64_t i = 0; i < 2 * static_cast<int64_t>(n.len); ++i) *w++ = n.kv[i];  // tokens, then slots
    }
    for (int64_t i = 0; i < c->count; ++i) *w++ = c->ring[(c->head + i) % c->pool_slots];
    return ra_ok();
  });
}

}  // extern "C"
