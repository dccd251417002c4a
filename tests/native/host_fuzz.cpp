// Host-side stress driver for the radix cache, its eviction log and the
// router meta-tree, built with AddressSanitizer and UndefinedBehaviorSanitizer
// by tests/test_native_sanitizers.py.  Seeded random request streams over a
// small vocabulary (so sequences share prefixes): match, lock, allocate
// (evicting on shortage, as Algorithm 1 does), insert, unlock, drain the
// eviction log into the router, and check that every slot is either free or
// held by the tree.  Exits non-zero on the first failed check.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <numeric>
#include <random>
#include <vector>

#include "radixattn.h"

#define CHECK(cond)                                                                 \
  do {                                                                              \
    if (!(cond)) {                                                                  \
      std::fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__, #cond, \
                   ra_last_error());                                                \
      return 1;                                                                     \
    }                                                                               \
  } while (0)

static int run_seed(int seed) {
  std::mt19937_64 rng(static_cast<uint64_t>(seed));
  const int64_t S = 64 + static_cast<int64_t>(rng() % 512);
  std::vector<int32_t> perm(static_cast<size_t>(S));
  std::iota(perm.begin(), perm.end(), 0);
  std::shuffle(perm.begin(), perm.end(), rng);
  ra_cache* c = nullptr;
  CHECK(ra_cache_create(S, perm.data(), &c) == RA_OK);
  CHECK(ra_cache_log_evictions(c, 1) == RA_OK);
  const int32_t n_workers = 1 + static_cast<int32_t>(rng() % 6);
  ra_router* r = nullptr;
  CHECK(ra_router_create(n_workers, &r) == RA_OK);
  std::vector<int32_t> path(8);
  for (int op = 0; op < 400; ++op) {
    const int n = 1 + static_cast<int>(rng() % 48);
    std::vector<int32_t> t(static_cast<size_t>(n));
    for (auto& x : t) x = static_cast<int32_t>(rng() % 4);
    std::vector<int32_t> slots(static_cast<size_t>(n));
    int64_t len = -1, node = -1, delta = 0;
    CHECK(ra_match_prefix(c, t.data(), n, slots.data(), &len, &node) == RA_OK);
    CHECK(len >= 0 && len <= n && node >= 0);
    CHECK(ra_inc_ref(c, node, &delta) == RA_OK && delta <= 0);
    const int64_t need = n - len;
    if (ra_available_size(c) < need) {
      int64_t freed = 0;
      CHECK(ra_evict(c, need, &freed) == RA_OK && freed >= 0);
    }
    if (ra_available_size(c) >= need) {
      CHECK(ra_alloc_slots(c, need, slots.data() + len) == RA_OK);
      int64_t cached = -1, leaf = -1;
      CHECK(ra_insert(c, t.data(), slots.data(), n, &cached, &leaf) == RA_OK);
      CHECK(cached >= len && cached <= n);
      CHECK(ra_router_insert(r, static_cast<int32_t>(rng() % n_workers), t.data(), n) == RA_OK);
    } else {
      CHECK(ra_alloc_slots(c, need, slots.data() + len) == RA_ENOMEM);
    }
    CHECK(ra_dec_ref(c, node, &delta) == RA_OK && delta >= 0);
    for (;;) {
      int64_t pl = 0, el = 0;
      const int st = ra_eviction_log_pop(c, path.data(), static_cast<int64_t>(path.size()), &pl, &el);
      if (st != RA_OK) {
        CHECK(pl > static_cast<int64_t>(path.size()));
        path.resize(static_cast<size_t>(pl));
        continue;
      }
      if (pl < 0) break;
      CHECK(el >= 1 && el <= pl);
      CHECK(ra_router_evict(r, static_cast<int32_t>(rng() % n_workers), path.data(), pl, el) == RA_OK);
    }
    CHECK(ra_available_size(c) + ra_cached_tokens(c) == S);
    CHECK(ra_evictable_size(c) == ra_cached_tokens(c));  // nothing stays locked between requests
    std::vector<int64_t> held(static_cast<size_t>(n_workers));
    CHECK(ra_router_match(r, t.data(), n, held.data()) == RA_OK);
    for (int64_t h : held) CHECK(h >= 0 && h <= n);
    if (op % 64 == 0) {
      int64_t words = 0;
      CHECK(ra_snapshot(c, nullptr, 0, &words) == RA_OK && words >= 3);
      std::vector<int64_t> buf(static_cast<size_t>(words));
      CHECK(ra_snapshot(c, buf.data(), words, &words) == RA_OK);
      CHECK(ra_snapshot(c, buf.data(), words - 1, &words) == RA_EINVAL);
    }
  }
  // Error paths change nothing.
  const int64_t avail = ra_available_size(c);
  CHECK(ra_dec_ref(c, 0x7fffffff, nullptr) == RA_EINVAL);
  CHECK(ra_alloc_slots(c, S + 1, perm.data()) == RA_ENOMEM);
  CHECK(ra_insert(c, nullptr, nullptr, 3, nullptr, nullptr) == RA_EINVAL);
  CHECK(ra_router_insert(r, n_workers, path.data(), 1) == RA_EINVAL);
  CHECK(ra_available_size(c) == avail);
  int64_t freed = 0;
  CHECK(ra_evict(c, S, &freed) == RA_OK);
  CHECK(ra_available_size(c) == S && ra_cached_tokens(c) == 0 && ra_num_nodes(c) >= 1);
  ra_router_destroy(r);
  ra_cache_destroy(c);
  return 0;
}

int main(int argc, char** argv) {
  const int seeds = argc > 1 ? std::atoi(argv[1]) : 20;
  for (int s = 0; s < seeds; ++s)
    if (run_seed(s) != 0) {
      std::fprintf(stderr, "seed %d failed\n", s);
      return 1;
    }
  std::printf("ok %d seeds\n", seeds);
  return 0;
}
