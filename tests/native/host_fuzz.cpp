// Host-side stress driver for the radix cache, its eviction log and the
// router meta-tree, built with AddressSanitizer and UndefinedBehaviorSanitizer
// by tests/test_native_sanitizers.py.  Seeded random request streams over a
// small vocabulary (so sequences share prefixes): match, lock, allocate
// (evicting on shortage, as Algorithm 1 does), insert, unlock, drain the
// eviction log into the router, and check that every slot is either free or
// held by the tree; then plan random batches of slot rows for the
// shared-prefix decode and check the plans' coverage.  Exits non-zero on the
// first failed check.
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

// The shared-prefix decode planner on a batch of slot rows drawn from a
// random tree of slot runs (shared runs, identical rows, rows that are
// prefixes of others, empty contexts, permuted table rows): every request's
// positions covered exactly once, members' rows equal over their items,
// partial indices consecutive per request; a short buffer is rejected.
static int plan_seed(int seed) {
  std::mt19937_64 rng(0x5eed0000u + static_cast<uint64_t>(seed));
  const int32_t B = 1 + static_cast<int32_t>(rng() % 40);
  std::vector<std::vector<int32_t>> runs;  // node k's slot run; parent of k is k / 3 (k > 0)
  int32_t next = 100;
  for (int k = 0; k < 40; ++k) {
    std::vector<int32_t> r(1 + rng() % 30);
    for (auto& x : r) x = next++;
    runs.push_back(r);
  }
  std::vector<std::vector<int32_t>> rows(static_cast<size_t>(B));
  for (int32_t b = 0; b < B; ++b) {
    int node = static_cast<int>(rng() % runs.size());
    std::vector<int> path;
    for (; node > 0; node /= 3) path.push_back(node);
    for (auto it = path.rbegin(); it != path.rend(); ++it) rows[b].insert(rows[b].end(), runs[*it].begin(), runs[*it].end());
    if (b > 0 && rng() % 8 == 0) rows[b] = rows[rng() % b];                      // identical row
    if (rng() % 5 == 0) rows[b].resize(rng() % (rows[b].size() + 1));          // cut (maybe empty)
    for (int k = static_cast<int>(rng() % 6); k > 0; --k) rows[b].push_back(next++);  // private tail
  }
  size_t stride = 1;
  for (auto& r : rows) stride = std::max(stride, r.size() + 2);
  const int64_t R = B + 3;
  std::vector<int32_t> rtt(static_cast<size_t>(R) * stride, -9), rpi(B), lens(B);
  for (int32_t b = 0; b < B; ++b) {
    rpi[b] = (b * 7 + 2) % static_cast<int32_t>(R);
    while (std::count(rpi.begin(), rpi.begin() + b, rpi[b])) rpi[b] = (rpi[b] + 1) % static_cast<int32_t>(R);
    std::copy(rows[b].begin(), rows[b].end(), rtt.begin() + static_cast<int64_t>(rpi[b]) * stride);
    lens[b] = static_cast<int32_t>(rows[b].size());
  }
  const int32_t mpb = 1 + static_cast<int32_t>(rng() % 16), min_shared = 1 + static_cast<int32_t>(rng() % 20);
  const int32_t chunk = static_cast<int32_t>(rng() % 3 == 0 ? 0 : 1 + rng() % 40);
  int64_t need = 0;
  CHECK(ra_decode_share_plan(rtt.data(), R, static_cast<int64_t>(stride), rpi.data(), lens.data(), B, mpb, min_shared,
                             chunk, 8, nullptr, 0, &need) == RA_OK);
  std::vector<int32_t> plan(static_cast<size_t>(need));
  if (need > 1)
    CHECK(ra_decode_share_plan(rtt.data(), R, static_cast<int64_t>(stride), rpi.data(), lens.data(), B, mpb,
                               min_shared, chunk, 8, plan.data(), need - 1, &need) == RA_EINVAL);
  CHECK(ra_decode_share_plan(rtt.data(), R, static_cast<int64_t>(stride), rpi.data(), lens.data(), B, mpb, min_shared,
                             chunk, 8, plan.data(), need, &need) == RA_OK);
  const int32_t n_items = plan[0], n_mem = plan[1], n_parts = plan[2];
  CHECK(plan[3] == B && plan[4] == mpb && need == 16 + 8 * int64_t{n_items} + 2 * int64_t{n_mem} + B + 1);
  const int32_t* items = plan.data() + 16;
  const int32_t* mem = items + 8 * static_cast<int64_t>(n_items);
  const int32_t* part_off = mem + 2 * static_cast<int64_t>(n_mem);
  std::vector<std::vector<int>> cover(static_cast<size_t>(B));
  std::vector<std::vector<int32_t>> parts(static_cast<size_t>(B));
  for (int32_t b = 0; b < B; ++b) cover[b].assign(static_cast<size_t>(lens[b]), 0);
  for (int32_t i = 0; i < n_items; ++i) {
    const int32_t* it = items + 8 * i;
    CHECK(it[0] >= 0 && it[0] < R && 0 <= it[1] && it[1] < it[2] && it[4] >= 1 && it[4] <= mpb);
    CHECK(it[3] >= 0 && it[3] + it[4] <= n_mem);
    for (int32_t m = 0; m < it[4]; ++m) {
      const int32_t b = mem[2 * (it[3] + m)];
      CHECK(b >= 0 && b < B && it[2] <= lens[b]);
      for (int32_t t = it[1]; t < it[2]; ++t) {
        CHECK(rtt[static_cast<size_t>(rpi[b]) * stride + t] == rtt[static_cast<size_t>(it[0]) * stride + t]);
        ++cover[b][t];
      }
      parts[b].push_back(mem[2 * (it[3] + m) + 1]);
    }
  }
  CHECK(part_off[0] == 0 && part_off[B] == n_parts);
  for (int32_t b = 0; b < B; ++b) {
    for (int c : cover[b]) CHECK(c == 1);
    const int32_t lo = part_off[b], hi = part_off[b + 1];
    if (parts[b].size() == 1) {
      CHECK(parts[b][0] == -1 && hi == lo);
    } else {
      std::sort(parts[b].begin(), parts[b].end());
      CHECK(static_cast<int32_t>(parts[b].size()) == hi - lo);
      for (size_t k = 0; k < parts[b].size(); ++k) CHECK(parts[b][k] == lo + static_cast<int32_t>(k));
    }
  }
  return 0;
}

int main(int argc, char** argv) {
  const int seeds = argc > 1 ? std::atoi(argv[1]) : 20;
  for (int s = 0; s < seeds; ++s)
    if (run_seed(s) != 0 || plan_seed(s) != 0) {
      std::fprintf(stderr, "seed %d failed\n", s);
      return 1;
    }
  std::printf("ok %d seeds\n", seeds);
  return 0;
}
