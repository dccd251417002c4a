// Host plan of a shared-prefix decode batch (ra_decode_share_plan).
//
// RadixAttention keeps one copy of every cached prefix (section 3): requests
// whose contexts start with the same tokens hold the same pool slots for those
// positions.  A decode batch in which many requests sit on the same branches
// of the radix tree therefore asks for the same K/V rows many times.  This
// planner finds those shared runs from the requests' slot rows and cuts the
// batch into work items, each a run of positions of one table row read once
// for up to `members_per_item` requests.
//
//   1. Requests with a context are sorted by their slot rows (lexicographic
//      over positions 0 .. L-1 with the bytes of each slot number compared as
//      memcmp does, which is as good a total order as numeric order; a row
//      that is a prefix of another sorts first).  Any lexicographic order
//      puts the requests that share a prefix next to each other, so
//      neighbours share the longest common prefixes, and the
//      common-prefix lengths of neighbours (lcp) define a tree of intervals:
//      an interval [lb, rb] with value l is a maximal run of sorted requests
//      that all agree on positions 0 .. l-1 (the radix tree of the batch).
//   2. Walking that tree from the root with the first position not yet
//      covered (ps): a node whose members number at least two and whose run
//      l - ps is at least min_shared tokens becomes a shared segment
//      [ps, l); its subtree then starts at l.  A shorter run is left to the
//      node's children (their segments start at ps).  Each request's rest,
//      [ps, L), is its private segment.
//   3. Segments are cut into chunks of at most chunk_len positions and their
//      members into blocks of at most members_per_item; every (chunk, block)
//      is a work item.  chunk_len = 0 takes the longest of 4096, 2048, 1024,
//      512 and 256 positions that still gives at least min_items items (the
//      shortest if none does).  Items are ordered longest first.
//   4. Every (item, member) pair is one partial result of that request.  A
//      request with several partials gets consecutive partial indices
//      (part_off); a request with one writes its output directly (index -1).
//
// Plan layout (int32): a 16-word header {n_items, n_member_entries, n_parts,
// batch, members_per_item, rows_per_kv_head (sum of item lengths, capped at
// INT32_MAX), chunk length, 0 ...}, then n_items items of 8 words {table row, first
// position, end position, first member entry, member count, 0, 0, 0}, then
// n_member_entries pairs {request, partial index or -1}, then part_off
// [batch + 1] (request b's partials are part_off[b] .. part_off[b+1]-1).
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

#include "radixattn.h"
#include "ra_error.h"

namespace {

struct Interval {
  int32_t lcp;
  int32_t lb, rb;
  std::vector<int32_t> kids;  // indices into the interval vector
};

struct Item {
  int32_t row, t0, t1;
  std::vector<int32_t> members;  // requests
};

// A segment before chunking: positions [t0, t1) of request rep's row, shared
// by the sorted requests mem[0 .. nm).
struct Segment {
  int32_t rep, t0, t1;
  const int32_t* mem;
  int32_t nm;
};

// Length of the common prefix of two slot rows over their first n entries
// (compared 64 entries at a time with memcmp, then entry by entry).
int32_t common_prefix(const int32_t* a, const int32_t* b, int32_t n) {
  int32_t k = 0;
  while (k + 64 <= n && std::memcmp(a + k, b + k, 64 * sizeof(int32_t)) == 0) k += 64;
  while (k < n && a[k] == b[k]) ++k;
  return k;
}

}  // namespace

extern "C" int ra_decode_share_plan(const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                    const int32_t* req_pool_idx, const int32_t* seq_lens, int32_t batch,
                                    int32_t members_per_item, int32_t min_shared, int32_t chunk_len,
                                    int32_t min_items, int32_t* plan, int64_t plan_capacity, int64_t* plan_len) {
  return ra_guard("ra_decode_share_plan", [&]() -> int {
    if (batch < 0 || rtt_rows <= 0 || rtt_stride <= 0 || members_per_item < 1 || members_per_item > 16 ||
        min_shared < 1 || chunk_len < 0 || min_items < 0 || !plan_len)
      return ra_fail(RA_EINVAL, "ra_decode_share_plan: bad sizes");
    if (batch > 0 && (!req_to_token || !req_pool_idx || !seq_lens))
      return ra_fail(RA_EINVAL, "ra_decode_share_plan: NULL pointer");
    std::vector<int32_t> len(batch, 0);
    std::vector<int32_t> reqs;
    for (int32_t b = 0; b < batch; ++b) {
      const int64_t r = req_pool_idx[b];
      if (r < 0 || r >= rtt_rows) return ra_fail(RA_EINVAL, "ra_decode_share_plan: table row out of range");
      len[b] = static_cast<int32_t>(std::min<int64_t>(std::max(seq_lens[b], 0), rtt_stride));
      if (len[b] > 0) reqs.push_back(b);
    }
    auto row = [&](int32_t b) { return req_to_token + static_cast<int64_t>(req_pool_idx[b]) * rtt_stride; };
    // 1. sort by slot row; lcp of neighbours
    std::stable_sort(reqs.begin(), reqs.end(), [&](int32_t a, int32_t b) {
      const int32_t n = std::min(len[a], len[b]);
      const int c = std::memcmp(row(a), row(b), static_cast<size_t>(n) * sizeof(int32_t));
      return c != 0 ? c < 0 : len[a] < len[b];
    });
    const int32_t n = static_cast<int32_t>(reqs.size());
    std::vector<int32_t> lcp(n + 1, 0);
    for (int32_t i = 1; i < n; ++i) {
      const int32_t a = reqs[i - 1], b = reqs[i];
      lcp[i] = common_prefix(row(a), row(b), std::min(len[a], len[b]));
    }
    // interval tree, bottom-up over the lcp array (lcp[n] = 0 closes all
    // intervals but the root)
    std::vector<Interval> iv;
    std::vector<int32_t> st;
    iv.push_back({0, 0, n - 1, {}});
    st.push_back(0);
    for (int32_t i = 1; i <= n; ++i) {
      const int32_t l = i < n ? lcp[i] : 0;
      int32_t lb = i - 1;
      int32_t last = -1;
      while (l < iv[st.back()].lcp) {
        const int32_t top = st.back();
        st.pop_back();
        iv[top].rb = i - 1;
        lb = iv[top].lb;
        last = top;
        if (l <= iv[st.back()].lcp) {
          iv[st.back()].kids.push_back(last);
          last = -1;
        }
      }
      if (l > iv[st.back()].lcp) {
        Interval node{l, lb, -1, {}};
        if (last >= 0) node.kids.push_back(last);
        iv.push_back(std::move(node));
        st.push_back(static_cast<int32_t>(iv.size()) - 1);
      }
    }
    // 2. walk (explicit stack: the tree can be as deep as the batch)
    std::vector<Segment> segs;
    auto emit = [&](int32_t rep, int32_t t0, int32_t t1, const int32_t* mem, int32_t nm) {
      segs.push_back({rep, t0, t1, mem, nm});
    };
    if (n > 0) {
      struct Frame {
        int32_t node, ps;
      };
      std::vector<Frame> todo{{0, 0}};
      std::vector<char> covered;
      while (!todo.empty()) {
        const Frame f = todo.back();
        todo.pop_back();
        const Interval& v = iv[f.node];
        int32_t ps = f.ps;
        const int32_t nm = v.rb - v.lb + 1;
        if (nm >= 2 && v.lcp - ps >= min_shared) {
          emit(reqs[v.lb], ps, v.lcp, &reqs[v.lb], nm);
          ps = v.lcp;
        }
        covered.assign(nm, 0);
        for (int32_t k : v.kids) {
          for (int32_t i = iv[k].lb; i <= iv[k].rb; ++i) covered[i - v.lb] = 1;
          todo.push_back({k, ps});
        }
        for (int32_t i = v.lb; i <= v.rb; ++i) {
          const int32_t b = reqs[i];
          if (!covered[i - v.lb] && len[b] > ps) emit(b, ps, len[b], &reqs[i], 1);
        }
      }
    }
    // 3. chunks and member blocks
    auto count_items = [&](int32_t ch) {
      int64_t k = 0;
      for (const Segment& g : segs)
        k += ((static_cast<int64_t>(g.t1) - g.t0 + ch - 1) / ch) * ((g.nm + members_per_item - 1) / members_per_item);
      return k;
    };
    int32_t chunk = chunk_len;
    if (chunk == 0) {
      static const int32_t kChunks[] = {4096, 2048, 1024, 512, 256};
      for (int32_t ch : kChunks) {
        chunk = ch;
        if (count_items(ch) >= min_items) break;
      }
    }
    std::vector<Item> items;
    items.reserve(static_cast<size_t>(count_items(chunk)));
    for (const Segment& g : segs) {
      for (int32_t c0 = g.t0; c0 < g.t1; c0 += chunk) {
        const int32_t c1 = static_cast<int32_t>(std::min<int64_t>(g.t1, static_cast<int64_t>(c0) + chunk));
        for (int32_t m0 = 0; m0 < g.nm; m0 += members_per_item) {
          Item it{req_pool_idx[g.rep], c0, c1, {}};
          it.members.assign(g.mem + m0, g.mem + std::min(g.nm, m0 + members_per_item));
          items.push_back(std::move(it));
        }
        if (c1 >= g.t1) break;
      }
    }
    std::stable_sort(items.begin(), items.end(),
                     [](const Item& a, const Item& b) { return a.t1 - a.t0 > b.t1 - b.t0; });
    // 4. partial indices
    std::vector<int32_t> nparts(batch, 0);
    int64_t n_mem = 0, rows = 0;
    for (const Item& it : items) {
      n_mem += static_cast<int64_t>(it.members.size());
      rows += it.t1 - it.t0;
      for (int32_t b : it.members) ++nparts[b];
    }
    std::vector<int32_t> part_off(static_cast<size_t>(batch) + 1, 0);
    for (int32_t b = 0; b < batch; ++b) part_off[b + 1] = part_off[b] + (nparts[b] > 1 ? nparts[b] : 0);
    const int64_t need = 16 + 8 * static_cast<int64_t>(items.size()) + 2 * n_mem + batch + 1;
    if (need > INT32_MAX || part_off[batch] < 0) return ra_fail(RA_EINVAL, "ra_decode_share_plan: plan too large");
    *plan_len = need;
    if (!plan || plan_capacity < need) {
      if (!plan) return ra_ok();  // size query
      return ra_fail(RA_EINVAL, "ra_decode_share_plan: plan buffer too small");
    }
    std::fill(plan, plan + 16, 0);
    plan[0] = static_cast<int32_t>(items.size());
    plan[1] = static_cast<int32_t>(n_mem);
    plan[2] = part_off[batch];
    plan[3] = batch;
    plan[4] = members_per_item;
    plan[5] = static_cast<int32_t>(std::min<int64_t>(rows, INT32_MAX));
    plan[6] = chunk;
    int32_t* ip = plan + 16;
    int32_t* mp = ip + 8 * items.size();
    int32_t* po = mp + 2 * n_mem;
    std::vector<int32_t> next(part_off.begin(), part_off.end() - 1);
    int32_t e = 0;
    for (size_t i = 0; i < items.size(); ++i) {
      const Item& it = items[i];
      int32_t* d = ip + 8 * i;
      d[0] = it.row, d[1] = it.t0, d[2] = it.t1, d[3] = e, d[4] = static_cast<int32_t>(it.members.size());
      d[5] = d[6] = d[7] = 0;
      for (int32_t b : it.members) {
        mp[2 * e] = b;
        mp[2 * e + 1] = nparts[b] > 1 ? next[b]++ : -1;
        ++e;
      }
    }
    std::copy(part_off.begin(), part_off.end(), po);
    return ra_ok();
  });
}
