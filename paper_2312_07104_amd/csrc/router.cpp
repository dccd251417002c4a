// Router meta-tree for data-parallel RadixAttention (Appendix A.4 of the SGLang
// paper): each replica worker keeps its own radix tree; the router keeps one
// trie over the token sequences of all workers in which every node records
// the set of workers that hold that prefix.  Dispatch matches a request in the
// meta-tree to find, per worker, how much of its prompt that worker has
// cached.  Workers report evictions through a queue that the router applies
// when it is idle, so its view is weakly consistent: between commits it may
// still credit a worker with a prefix the worker has already dropped.
//
// Layout: nodes in a vector indexed by id, the child index one hash map keyed
// by (parent id, first token) plus a child list per node (for subtree walks),
// a 64-bit worker mask per node (at most 64 workers).  A node whose mask
// becomes empty and that has no children is removed, and so is its parent
// when that leaves it empty and childless.
#include <cstdint>
#include <memory>
#include <string>
#include <unordered_map>
#include <vector>

#include "radixattn.h"
#include "ra_error.h"

namespace {

struct MNode {
  int64_t parent = -1;
  std::vector<int32_t> key;
  uint64_t mask = 0;
  std::vector<int64_t> kids;
  bool alive = false;
};

void drop(std::vector<int64_t>& v, int64_t x) {
  for (size_t i = 0; i < v.size(); ++i)
    if (v[i] == x) {
      v[i] = v.back();
      v.pop_back();
      return;
    }
}

inline uint64_t edge(int64_t parent, int32_t tok) {
  return (static_cast<uint64_t>(parent) << 32) ^ static_cast<uint32_t>(tok);
}

}  // namespace

struct ra_router {
  int32_t n_workers = 0;
  std::vector<MNode> nodes;
  std::vector<int64_t> free_ids;
  std::unordered_map<uint64_t, int64_t> children;
  std::vector<int64_t> held;  // tokens per worker in the router's view
  int64_t live = 1;

  int64_t new_node() {
    int64_t id;
    if (!free_ids.empty()) {
      id = free_ids.back();
      free_ids.pop_back();
      nodes[id] = MNode();
    } else {
      id = static_cast<int64_t>(nodes.size());
      nodes.emplace_back();
    }
    nodes[id].alive = true;
    ++live;
    return id;
  }

  // Splits node x so that its first j tokens form a new upper node, which is
  // returned; x keeps the rest.  Both carry x's mask.
  int64_t split(int64_t x, int64_t j) {
    const int64_t y = new_node();
    MNode& X = nodes[x];
    MNode& Y = nodes[y];
    Y.parent = X.parent;
    Y.key.assign(X.key.begin(), X.key.begin() + j);
    Y.mask = X.mask;
    Y.kids.push_back(x);
    children[edge(Y.parent, Y.key[0])] = y;
    for (int64_t& k : nodes[Y.parent].kids)
      if (k == x) k = y;
    X.key.erase(X.key.begin(), X.key.begin() + j);
    X.parent = y;
    children[edge(y, X.key[0])] = x;
    return y;
  }

  void remove_if_empty(int64_t x) {
    while (x != 0 && nodes[x].alive && nodes[x].mask == 0 && nodes[x].kids.empty()) {
      MNode& n = nodes[x];
      const int64_t par = n.parent;
      children.erase(edge(par, n.key[0]));
      n.alive = false;
      std::vector<int32_t>().swap(n.key);
      free_ids.push_back(x);
      --live;
      drop(nodes[par].kids, x);
      x = par;
    }
  }

  // Clears worker bit b in the subtree rooted at x (x included).
  void clear_subtree(int64_t x, uint64_t b, int32_t w) {
    std::vector<int64_t> stack{x};
    std::vector<int64_t> order;
    while (!stack.empty()) {
      const int64_t y = stack.back();
      stack.pop_back();
      order.push_back(y);
      for (int64_t k : nodes[y].kids) stack.push_back(k);
    }
    for (auto it = order.rbegin(); it != order.rend(); ++it) {
      MNode& n = nodes[*it];
      if (n.mask & b) {
        n.mask &= ~b;
        held[w] -= static_cast<int64_t>(n.key.size());
      }
      remove_if_empty(*it);
    }
  }
};

extern "C" {

int ra_router_create(int32_t n_workers, ra_router** out) {
  return ra_guard("ra_router_create", [&]() -> int {
    if (!out) return ra_fail(RA_EINVAL, "ra_router_create: out is NULL");
    *out = nullptr;
    if (n_workers < 1 || n_workers > 64) return ra_fail(RA_EINVAL, "ra_router_create: n_workers must be in [1, 64]");
    std::unique_ptr<ra_router> r(new ra_router);
    r->n_workers = n_workers;
    r->nodes.emplace_back();
    r->nodes[0].alive = true;
    r->nodes[0].mask = n_workers == 64 ? ~0ull : ((1ull << n_workers) - 1);  // every worker holds the empty prefix
    r->held.assign(n_workers, 0);
    *out = r.release();
    return ra_ok();
  });
}

void ra_router_destroy(ra_router* r) { delete r; }

int ra_router_match(const ra_router* r, const int32_t* tokens, int64_t n, int64_t* out_len) {
  return ra_guard("ra_router_match", [&]() -> int {
    if (!r || !out_len || (n > 0 && !tokens) || n < 0) return ra_fail(RA_EINVAL, "ra_router_match: bad argument");
    for (int32_t w = 0; w < r->n_workers; ++w) out_len[w] = 0;
    int64_t node = 0, pos = 0;
    while (pos < n) {
      auto it = r->children.find(edge(node, tokens[pos]));
      if (it == r->children.end()) break;
      const MNode& x = r->nodes[it->second];
      int64_t j = 0;
      const int64_t kl = static_cast<int64_t>(x.key.size());
      while (j < kl && pos + j < n && x.key[j] == tokens[pos + j]) ++j;
      pos += j;
      for (uint64_t m = x.mask; m; m &= m - 1) out_len[__builtin_ctzll(m)] = pos;
      if (j < kl || x.mask == 0) break;
      node = it->second;
    }
    return ra_ok();
  });
}

int ra_router_insert(ra_router* r, int32_t worker, const int32_t* tokens, int64_t n) {
  return ra_guard("ra_router_insert", [&]() -> int {
    if (!r || worker < 0 || worker >= r->n_workers || n < 0 || (n > 0 && !tokens))
      return ra_fail(RA_EINVAL, "ra_router_insert: bad argument");
    const uint64_t b = 1ull << worker;
    int64_t node = 0, pos = 0;
    while (pos < n) {
      auto it = r->children.find(edge(node, tokens[pos]));
      if (it == r->children.end()) {
        const int64_t leaf = r->new_node();
        MNode& L = r->nodes[leaf];
        L.parent = node;
        L.key.assign(tokens + pos, tokens + n);
        L.mask = b;
        r->children[edge(node, tokens[pos])] = leaf;
        r->nodes[node].kids.push_back(leaf);
        r->held[worker] += n - pos;
        return ra_ok();
      }
      int64_t x = it->second;
      int64_t j = 0;
      const int64_t kl = static_cast<int64_t>(r->nodes[x].key.size());
      while (j < kl && pos + j < n && r->nodes[x].key[j] == tokens[pos + j]) ++j;
      if (j < kl) x = r->split(x, j);
      MNode& X = r->nodes[x];
      if (!(X.mask & b)) {
        X.mask |= b;
        r->held[worker] += static_cast<int64_t>(X.key.size());
      }
      pos += j;
      node = x;
    }
    return ra_ok();
  });
}

int ra_router_evict(ra_router* r, int32_t worker, const int32_t* tokens, int64_t path_len, int64_t evicted_len) {
  return ra_guard("ra_router_evict", [&]() -> int {
    if (!r || worker < 0 || worker >= r->n_workers || path_len < 0 || evicted_len < 0 || evicted_len > path_len ||
        (path_len > 0 && !tokens))
      return ra_fail(RA_EINVAL, "ra_router_evict: bad argument");
    if (evicted_len == 0) return ra_ok();
    const uint64_t b = 1ull << worker;
    const int64_t start = path_len - evicted_len;
    // Walk the path to position `start`, splitting the node that straddles it,
    // so that the evicted range begins on a node boundary.
    int64_t node = 0, pos = 0;
    while (pos < start) {
      auto it = r->children.find(edge(node, tokens[pos]));
      if (it == r->children.end()) return ra_ok();  // the router never saw this range
      const int64_t x = it->second;
      const int64_t kl = static_cast<int64_t>(r->nodes[x].key.size());
      int64_t j = 0;
      while (j < kl && pos + j < start && r->nodes[x].key[j] == tokens[pos + j]) ++j;
      if (pos + kl <= start) {
        if (j < kl) return ra_ok();
        pos += kl;
        node = x;
        continue;
      }
      if (j < start - pos) return ra_ok();  // the path leaves the tree before the evicted range
      node = r->split(x, start - pos);      // the upper part ends at `start`
      pos = start;
    }
    // The node that continues the path at `start` heads the evicted range; the
    // worker held nothing below the evicted leaf, so its bit goes from that
    // node's whole subtree.
    auto it = r->children.find(edge(node, tokens[start]));
    if (it == r->children.end()) return ra_ok();
    r->clear_subtree(it->second, b, worker);
    return ra_ok();
  });
}

int64_t ra_router_num_nodes(const ra_router* r) { return r ? r->live : 0; }

int64_t ra_router_held_tokens(const ra_router* r, int32_t worker) {
  if (!r || worker < 0 || worker >= r->n_workers) return -1;
  return r->held[worker];
}

}  // extern "C"
