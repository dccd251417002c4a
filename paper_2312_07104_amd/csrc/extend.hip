// Extend attention (ra_extend_attention): prefill of a request's new tokens
// over its cached prefix (the work that remains once RadixAttention reuses the
// prefix's KV cache; section 3, Appendix A.1) plus causal attention among the
// new tokens.  A dense contraction, so QK^T and PV run on bf16 MFMA
// (v_mfma_f32_16x16x32_bf16) with fp32 accumulation.
//
// Work item = (request, kv head, query tile).  A tile packs query rows as
// (new token, query head of the kv head's group), so the G heads sharing a kv
// head share every K/V tile.  Waves of 32 query rows (two 16-column MFMA
// blocks), two waves per SIMD: eight waves and 256 rows per work-group with
// 64-key tiles (one work-group per CU), or four waves and 128 rows with
// 32-key tiles (two per CU) for requests with fewer rows.  Work items start
// longest first (ra_lpt_item), so batches that fill the chip only a few
// times over do not end on their longest items.
//   * K/V tiles arrive by direct-to-LDS copies (global_load_lds_dwordx4: a
//     prefix row is gathered through the request's slot-table row, a new
//     token's row read from k_new / v_new) into a four-stage ring, two tiles
//     of lead.  The slot indices travel by copy four tiles ahead into their
//     own ring and are read into registers a tile before use.  A tile is
//     row-major (a key's D values contiguous, 16-byte slots swizzled by
//     ext_swz), so one copy instruction moves whole rows.
//   * The loop runs over 32-key halves, software pipelined in one issue
//     order that sched_barrier fences hold: the S^T = K Q^T MFMAs of the next
//     half, each followed by one probability of the current half (fma +
//     exp2, bf16 pack every second), then the current half's PV MFMAs with
//     the next half's maxima between them.  About 1.5 VALU instructions per
//     MFMA, which one wave can issue under the matrix core's pace.
//   * At a tile's top (one barrier) the wave computes the addresses of the
//     copies two tiles ahead; the copies themselves are issued one every two
//     PV MFMA steps of the next fused step, so the waves never queue their
//     copies at the address unit all at once.
//   * Q^T and the O^T accumulators live in AGPRs (inline-assembly MFMAs with
//     "a" operands); S^T stays in VGPRs, where the softmax reads it.  The
//     compiler does not track hazards of inline assembly, so the code keeps
//     the wait states itself: two after the VALU writes P^T, several MFMAs
//     between an S^T MFMA and the VALU reading its result, and a long s_nop
//     run before the VALU touches O (rare rescale, epilogue).
//   * Online softmax in the base-2 domain.  The running maximum moves only
//     when some score exceeds it by more than 2^24 after exponentiation, so
//     after the first half of a query tile the rescale path is practically
//     never taken; the test is on each lane's partial maximum, so the common
//     path has no cross-lane reduction.  Probabilities up to 2^24 cannot
//     overflow the fp32 accumulators (2^24 times 2^22 keys times |v|).  Row
//     sums come from an MFMA against a ones operand, so numerator and
//     denominator see the same bf16 P.

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "device_common.h"
#include "lds_dma.h"

namespace {

constexpr int kStages = 4;   // K/V tiles resident in LDS
template <int V>
using ic = std::integral_constant<int, V>;
constexpr int kRing = 4;     // slot-index ring (tiles)
constexpr int kQB = 2;       // 16-query column blocks per wave (32 query rows)
// exp2 argument ceiling of the lazy maximum: p <= 2^kLazyLog2
constexpr float kLazyLog2 = 24.f;

// O^T block += A B on AGPR accumulators (the compiler inserts no wait states
// for it: callers keep VALU writes of A and B at least two wait states away).
__device__ __forceinline__ void pv_mfma(f32x4_t& o, const bf16x8_t& a, const bf16x8_t& b) {
  asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(o) : "v"(a), "v"(b));
}

// S^T block (+)= K Q^T with the Q^T operand in AGPRs and S^T in VGPRs.  The
// compiler inserts no wait states for it: VALU reads of S^T must come at
// least 11 wait states after the last MFMA writing it (callers keep several
// MFMAs in between, or an s_nop run).
__device__ __forceinline__ void s_mfma_first(f32x4_t& s, const bf16x8_t& a, const bf16x8_t& qa) {
  asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(s) : "v"(a), "a"(qa));
}
__device__ __forceinline__ void s_mfma_acc(f32x4_t& s, const bf16x8_t& a, const bf16x8_t& qa) {
  asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(s) : "v"(a), "a"(qa));
}

// Layout of a K or V tile: row-major, row r = RB = 2 D bytes; its 16-byte
// slot s (head-dimension values 8 s .. 8 s + 7) sits at slot s ^ ext_swz(r).
// One direct-to-LDS copy instruction (1 KB) then fills 1024 / RB whole rows,
// each read from one contiguous run of global memory (the 64-byte runs of a
// piece-group layout touch twice as many cache lines per instruction).  The
// swizzles were found by an exhaustive search over XOR masks of the row
// bits against the gfx950 LDS bank model (64 banks of 4 bytes; ds_read_b128
// in four cycles of the 16-lane groups {0-7, 24-31}, {8-15, 16-23},
// {32-39, 56-63}, {40-47, 48-55}; ds_read_b64_tr_b16 in two cycles of 32
// lanes): the K operand reads (rows 8 (c >> 2) + (c & 3) + const, slot
// 4 ks + (lane >> 4)) and the transposed V reads (rows 8 (lane >> 4) +
// (c >> 2) + const) then touch 64 distinct banks per cycle.  The masks ignore
// row bits 2, 4 and 5, which the loops add as constants, so every operand
// read is one per-lane offset plus an immediate.
template <int D>
__device__ __forceinline__ int ext_swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 1) | (r & 8);
  else return (r & 2) | ((r & 8) >> 1);
}

// Key splits: an item whose keys are cut into splits takes at least this many
// tiles per split (fewer splits for shorter items; the rest stay empty), and
// at most kMaxSplits splits.
constexpr int kMinSplitTiles = 8;
constexpr int kMaxSplits = 16;

// Requests above this batch size keep the static item order: the ranking
// below is quadratic in the batch, and its scratch (8 * batch + 8 words)
// lives in the K/V ring, whose smallest configuration (D = 64, 128 rows) has
// 32 KB.
constexpr int kLptMaxBatch = 1016;

// Work item of block k in longest-first order.  A unit is (request, query
// tile, key split).  Units are ordered by their request's key count P + E,
// longest first (ties by request index), and within a request by query tile,
// the last (longest) tile first, then by split.  Block k takes unit k / hkv of kv head
// k % hkv.  The dispatcher starts blocks in index order and deals them to
// the XCDs round-robin, so every XCD runs its share longest-first, and with
// 8 | hkv each XCD keeps whole kv heads (its L2 sees their rows only).  A
// static order would leave the longest items for the end when a batch fills
// the chip only a few times over (short extends, head shards).  Every
// thread of the work-group takes part; `scratch` holds 8 * batch + 8 words
// of LDS.  The request's own arguments (start, E, P and table row, as passed)
// come back through `req_args`, read once for the whole batch.  The LDS loops
// read four words per instruction so that their latencies overlap.  Returns
// false when block k has no unit.
template <bool UNIFORM>
__device__ bool ra_lpt_item(int32_t* scratch, int64_t k, int32_t hkv, int32_t batch, int32_t tpb,
                            const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ prefix_lens,
                            const int32_t* __restrict__ extend_lens, const int32_t* __restrict__ extend_start,
                            int64_t total_tokens, int64_t rtt_stride, int32_t nsplit, int& g, int& b, int& qt,
                            int& sp, int32_t (&req_args)[4], int nthreads) {
  const int bp = (batch + 3) & ~3;         // batch padded to whole int4 reads
  int32_t* args = scratch;                 // [batch][4] start, E, P, table row as passed (16-byte entries)
  int32_t* cost = scratch + 4 * batch;     // [bp] key count of the request's units, -1 if none, -2 padding
  int32_t* nun = cost + bp;                // [batch] units of the request
  int32_t* nrank = nun + batch;            // [bp] units by rank (0 padding)
  int32_t* ord = nrank + bp;               // [batch] request at each rank
  int32_t* found = ord + batch;            // [2] request and unit offset of this block
  const int tid = static_cast<int>(UNIFORM ? __builtin_amdgcn_workitem_id_x() : threadIdx.x), nt = nthreads;
  if (tid == 0) found[0] = -1;
  for (int t = tid; t < bp; t += nt) {
    if (t >= batch) {
      cost[t] = -2;
      nrank[t] = 0;
      continue;
    }
    const int32_t st = extend_start[t], el = extend_lens[t], pl = prefix_lens[t], rp = req_pool_idx[t];
    *reinterpret_cast<int4*>(&args[4 * t]) = make_int4(st, el, pl, rp);
    const int64_t e = (st < 0 || st > total_tokens) ? 0 : min<int64_t>(el, total_tokens - st);
    const int64_t p = min<int64_t>(max(pl, 0), rtt_stride);
    const int64_t nu = e > 0 ? (e + tpb - 1) / tpb * nsplit : 0;
    nun[t] = static_cast<int32_t>(nu);
    cost[t] = nu > 0 ? static_cast<int32_t>(min<int64_t>(p + e, INT32_MAX)) : -1;
  }
  __syncthreads();
  // rank = requests with a larger key count, or an equal one and a smaller
  // index (cost is only read here; ord and nrank are other words)
  for (int t = tid; t < batch; t += nt) {
    const int32_t c = cost[t];
    int rank = 0;
    for (int s4 = 0; s4 < bp; s4 += 4) {
      const int4 cs = *reinterpret_cast<const int4*>(&cost[s4]);
      rank += (cs.x > c) | ((cs.x == c) & (s4 < t));
      rank += (cs.y > c) | ((cs.y == c) & (s4 + 1 < t));
      rank += (cs.z > c) | ((cs.z == c) & (s4 + 2 < t));
      rank += (cs.w > c) | ((cs.w == c) & (s4 + 3 < t));
    }
    ord[rank] = t;
    nrank[rank] = nun[t];
  }
  __syncthreads();
  // Wave 0 scans the unit counts in rank order, 64 ranks at a time, and
  // finds the rank whose units hold unit r.
  const int64_t r = k / hkv;
  if (tid < 64) {
    int64_t carry = 0;
    for (int base = 0; base < batch; base += 64) {
      const int j = base + tid;
      const int32_t v = j < batch ? nrank[j] : 0;
      int64_t incl = v;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int64_t up = __shfl_up(incl, d, 64);
        if (tid >= d) incl += up;
      }
      const int64_t excl = carry + incl - v;
      if (j < batch && r >= excl && r < excl + v) {
        found[0] = ord[j];
        found[1] = static_cast<int32_t>(v - 1 - (r - excl));
      }
      carry += __shfl(incl, 63, 64);
    }
  }
  __syncthreads();
  // Every lane reads the same words.  UNIFORM makes that known to the
  // compiler, so the item's sizes, loops and branches stay scalar.
  auto uni = [](int32_t v) { return UNIFORM ? __builtin_amdgcn_readfirstlane(v) : v; };
  const int req = uni(found[0]);
  const int tile = uni(found[1]);
  if (req >= 0) {
    const int4 a = *reinterpret_cast<const int4*>(&args[4 * req]);
    req_args[0] = uni(a.x), req_args[1] = uni(a.y), req_args[2] = uni(a.z), req_args[3] = uni(a.w);
  }
  // the scratch is the K/V ring, which the copies overwrite next
  __syncthreads();
  if (req < 0) return false;
  g = static_cast<int>(k % hkv);
  b = req;
  qt = tile / nsplit;
  sp = tile % nsplit;
  return true;
}

// WAVES waves of 32 query rows per work-group, BN keys per K/V tile (64:
// two 32-key halves per tile; 32: one).  <D, 8, 64>: 256 rows, one
// work-group per CU; <D, 4, 32>: 128 rows, two work-groups per CU (65 KB of
// LDS each).  Either way two waves share each SIMD.
// nsplit > 1: the keys of each (request, kv head, query tile) are cut into
// up to nsplit runs of whole tiles, one work item each; an item writes its
// rows' output normalised over its own keys (fp32, ws_o [nsplit][rows][D],
// row = token * Hq + head) and their log2-sum-exp of scaled scores (ws_lse
// [nsplit][rows], -inf where the item saw no key of the row), and
// extend_combine_kernel merges them.
template <int D, int WAVES, int BN>
__global__ __launch_bounds__(WAVES * 64, 8 / WAVES) void extend_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k_new, const __bf16* __restrict__ v_new,
    int64_t total_tokens, const __bf16* __restrict__ k_pool, const __bf16* __restrict__ v_pool,
    int64_t pool_slots, const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride,
    const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ prefix_lens,
    const int32_t* __restrict__ extend_lens, const int32_t* __restrict__ extend_start, int32_t batch,
    int32_t hkv, int32_t grp, int32_t n_qtiles, int32_t lpt, float scale_log2, int32_t nsplit,
    float* __restrict__ ws_o, float* __restrict__ ws_lse, __bf16* __restrict__ out) {
  constexpr int kWaves = WAVES;
  constexpr int kBN = BN;
  constexpr int kBM = 32 * WAVES;             // query rows per work-group
  static_assert(BN == 32 || BN == 64, "tile of one or two 32-key halves");
  constexpr int KS = D / 32;                  // MFMA k-steps over the head dimension
  constexpr int DB = D / 16;                  // 16-row blocks of O^T
  constexpr int RB = 2 * D;                   // bytes of one K (or V) row
  constexpr int NSL = RB / 16;                // 16-byte slots of a row
  constexpr int RPI = 1024 / RB;              // rows per 1 KB copy instruction
  constexpr int TILE_B = kBN * RB;            // bytes per K (or V) tile
  constexpr int KRING_B = kStages * TILE_B;   // K ring, then the V ring
  // (a ring position is then an immediate offset of at most 48 KB, within
  // the 16-bit LDS offset field, once the loops unroll over the stages)
  constexpr int LOADS = TILE_B / (kWaves * 64 * 16);  // DMA instructions per wave per tile per tensor
  constexpr int ROW_STEP = kBN / LOADS;       // a DMA lane covers rows u0 + it * ROW_STEP
  static_assert(LOADS == 1 || LOADS == 2, "index vector width");
  static_assert(LOADS == 1 || RPI * kWaves == ROW_STEP, "a lane's rows are ROW_STEP apart");
  __shared__ __align__(16) unsigned char kv_lds[2 * KRING_B];
  static_assert((8 * kLptMaxBatch + 8) * 4 <= 2 * KRING_B, "ranking scratch exceeds the K/V rings");
  // one index copy moves 64 words (rows beyond the tile are never read)
  __shared__ __align__(16) int32_t idx_lds[kRing][64];

  // Work-groups go to the 8 XCDs round-robin (block i -> XCD i % 8).  Either
  // order below keeps the blocks of one kv head together on an XCD where it
  // can, so they share K/V rows through its L2.
  // The 256-row shape reads its ids through the intrinsics rather than
  // blockIdx / threadIdx: in a kernel this large the helper calls behind
  // those are not always inlined, and their results then look per-lane to
  // the compiler, which turns the item's loops and branches into divergent
  // ones (ten more VALU instructions per fused step).  The 128-row shape
  // keeps the helpers: with scalar loops its register allocation moves O^T
  // accumulators next to the inline-assembly MFMAs, which the wait-state
  // check on its assembly rejects.
  constexpr bool kUniform = WAVES == 8;
  const int64_t blk = kUniform ? static_cast<int64_t>(__builtin_amdgcn_workgroup_id_x()) : blockIdx.x;
  const int tpb = kBM / grp;  // new tokens per tile
  const int64_t n_items = static_cast<int64_t>(hkv) * batch * n_qtiles * nsplit;
  int g, b, qt, sp;
  int32_t req_args[4];  // extend_start, extend_lens, prefix_lens, req_pool_idx of request b
  if (lpt) {
    if (!ra_lpt_item<kUniform>(reinterpret_cast<int32_t*>(kv_lds), blk, hkv, batch, tpb, req_pool_idx, prefix_lens,
                     extend_lens, extend_start, total_tokens, rtt_stride, nsplit, g, b, qt, sp, req_args, WAVES * 64))
      return;
  } else {
    // Static order: XCD i % 8 takes a contiguous eighth of the (kv head,
    // request, query tile, split) order.
    const int64_t per_xcd = (n_items + 7) / 8;
    const int64_t item = (blk % 8) * per_xcd + blk / 8;
    if (item >= n_items) return;
    const int64_t per_head = static_cast<int64_t>(batch) * n_qtiles * nsplit;
    g = static_cast<int>(item / per_head);
    const int64_t rem = item % per_head;
    b = static_cast<int>(rem / (static_cast<int64_t>(n_qtiles) * nsplit));
    const int rq = static_cast<int>(rem % (static_cast<int64_t>(n_qtiles) * nsplit));
    qt = n_qtiles - 1 - rq / nsplit;
    sp = rq % nsplit;
    req_args[0] = extend_start[b], req_args[1] = extend_lens[b], req_args[2] = prefix_lens[b];
    req_args[3] = req_pool_idx[b];
  }

  const int64_t start = req_args[0];
  int64_t E = req_args[1];
  if (qt < 0 || qt >= n_qtiles || start < 0 || start > total_tokens) return;
  E = min(E, total_tokens - start);
  const int tok0 = qt * tpb;
  if (E <= 0 || tok0 >= E) return;
  const int tok_end = static_cast<int>(min<int64_t>(E, tok0 + tpb));
  const int P = static_cast<int>(min<int64_t>(max(req_args[2], 0), rtt_stride));
  int64_t rrow = req_args[3];
  rrow = (rrow >= 0 && rrow < rtt_rows) ? rrow : 0;
  const int32_t* trow = rtt + rrow * rtt_stride;
  const int kend = P + tok_end;
  const int hq = hkv * grp;
  // This item's tiles: kt0 is its first key, n_tiles its tile count (all of
  // the keys unless they are split).
  const int nt_all = (kend + kBN - 1) / kBN;
  int t_lo = 0, n_tiles = nt_all;
  if (nsplit > 1) {
    const int ns = min(nsplit, max(1, nt_all / kMinSplitTiles));
    t_lo = sp < ns ? sp * nt_all / ns : 0;
    n_tiles = sp < ns ? (sp + 1) * nt_all / ns - t_lo : 0;
  }
  const int kt0 = t_lo * kBN;

  const int tid = static_cast<int>(kUniform ? __builtin_amdgcn_workitem_id_x() : threadIdx.x);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (SGPR)
  const int lane = tid & 63;
  const int c = lane & 15;
  const int g4 = lane >> 4;

  // ---- DMA lane mapping (fixed for the kernel) ----------------------------
  // Instruction ch = it * kWaves + wave fills rows RPI ch .. RPI ch + RPI - 1
  // (1 KB at ch * 1024): lane l lands in slot l % NSL of row RPI ch + l / NSL
  // and so carries that row's logical slot (l % NSL) ^ ext_swz(row).
  int dma_row[LOADS];
  uint32_t dma_lds[LOADS];   // byte offset inside a tile (uniform per wave)
  uint32_t dma_gofs[LOADS];  // byte offset inside the gathered global row
#pragma unroll
  for (int it = 0; it < LOADS; ++it) {
    const int ch = it * kWaves + wave;
    const int u = RPI * ch + lane / NSL;
    dma_row[it] = u;
    dma_lds[it] = ch * 1024;
    dma_gofs[it] = static_cast<uint32_t>(g * D * 2 + 16 * ((lane % NSL) ^ ext_swz<D>(u)));
  }
  const uint32_t row_bytes = static_cast<uint32_t>(hkv) * D * 2;
  const unsigned char* kpool_b = reinterpret_cast<const unsigned char*>(k_pool);
  const unsigned char* knew_b = reinterpret_cast<const unsigned char*>(k_new);
  const int64_t vpool_delta = reinterpret_cast<const unsigned char*>(v_pool) - kpool_b;
  const int64_t vnew_delta = reinterpret_cast<const unsigned char*>(v_new) - knew_b;
  const uint32_t smax = static_cast<uint32_t>(pool_slots - 1);
  uint64_t kpool_lane[LOADS], knew_lane[LOADS];
#pragma unroll
  for (int it = 0; it < LOADS; ++it) {
    kpool_lane[it] = reinterpret_cast<uint64_t>(kpool_b) + dma_gofs[it];
    knew_lane[it] = reinterpret_cast<uint64_t>(knew_b) + static_cast<uint64_t>(start - P) * row_bytes + dma_gofs[it];
  }
  const uint32_t lds_kv0 = ra_lds_addr(kv_lds);

  // The index ring stores tile row u at word LOADS * (u % ROW_STEP) +
  // u / ROW_STEP, so a lane's LOADS slot indices are one vector LDS read.
  const int u0 = dma_row[0];
  const int idx_pos = (lane % LOADS) * ROW_STEP + lane / LOADS;
  // Wave 0 copies the slot indices of one tile.  It issues the copy for every
  // tile (reading row position 0 where the tile has no cached rows) so that
  // each wave's count of outstanding loads per tile is fixed.
  auto issue_idx = [&](int tile) {
    if (wave != 0) return;
    const int pos = kt0 + tile * kBN + idx_pos;
    ra_dma4(trow + (tile < n_tiles && pos < P ? pos : 0), ra_lds_addr(&idx_lds[tile % kRing][0]));
  };
  // This lane's LOADS slot indices of a tile, read from the index ring (one
  // vector LDS read; the values are consumed a tile later).
  auto read_idx = [&](int tile, int32_t (&sl)[LOADS]) {
    const int32_t* w = &idx_lds[tile % kRing][LOADS * u0];
    if constexpr (LOADS == 2) {
      const int2 v = *reinterpret_cast<const int2*>(w);
      sl[0] = v.x, sl[1] = v.y;
    } else {
      sl[0] = w[0];
    }
  };
  // Copies of one tile's K and V rows into ring stage tile % kStages: 2 * LOADS
  // per wave (source address per lane, LDS base per wave), K then V for each
  // it.  sl = the tile's slot indices (read_idx).  A tile past the last one
  // gets dummy copies of slot 0's row (one cache line per copy) into its
  // stage, which no wave reads again, so every tile has the same number of
  // outstanding loads.
  struct KvCopies {
    uint64_t src[2 * LOADS];
    uint32_t lds[2 * LOADS];
  };
  auto prep_kv = [&](int tile, const int32_t (&sl)[LOADS], KvCopies& cp) {
    const int kb = kt0 + tile * kBN;
    const uint32_t kst = lds_kv0 + (tile % kStages) * TILE_B;
#pragma unroll
    for (int it = 0; it < LOADS; ++it) {
      cp.lds[2 * it] = kst + dma_lds[it];
      cp.lds[2 * it + 1] = kst + KRING_B + dma_lds[it];
    }
    if (tile >= n_tiles) {
#pragma unroll
      for (int it = 0; it < LOADS; ++it) {
        cp.src[2 * it] = kpool_lane[it];
        cp.src[2 * it + 1] = kpool_lane[it] + vpool_delta;
      }
    } else if (kb + kBN <= P) {
#pragma unroll
      for (int it = 0; it < LOADS; ++it) {
        const uint32_t slot = min(static_cast<uint32_t>(sl[it]), smax);  // negative -> clamped
        const uint64_t src = kpool_lane[it] + static_cast<uint64_t>(slot) * row_bytes;
        cp.src[2 * it] = src;
        cp.src[2 * it + 1] = src + vpool_delta;
      }
    } else {
#pragma unroll
      for (int it = 0; it < LOADS; ++it) {
        const int pos = min(kb + dma_row[it], kend - 1);  // padding rows repeat a real key
        uint64_t src;
        int64_t vdelta;
        if (pos < P) {
          const uint32_t slot = min(static_cast<uint32_t>(sl[it]), smax);
          src = kpool_lane[it] + static_cast<uint64_t>(slot) * row_bytes;
          vdelta = vpool_delta;
        } else {
          src = knew_lane[it] + static_cast<uint64_t>(pos) * row_bytes;
          vdelta = vnew_delta;
        }
        cp.src[2 * it] = src;
        cp.src[2 * it + 1] = src + vdelta;
      }
    }
  };
  auto issue_copy = [&](const KvCopies& cp, int i) {
    ra_dma16(reinterpret_cast<const void*>(cp.src[i]), cp.lds[i]);
  };
  // Top of tile u: K/V(u) is in LDS for every wave and stage (u + 2) %
  // kStages = (u - 2) % kStages is free.  Order of this wave's loads issued
  // since the top of u - 1: idx(u + 3) (wave 0 only), then the copies of
  // K/V(u + 1); the wait retires everything before those, so idx(u + 3) and
  // K/V(u) have landed, and the barrier makes them visible to all waves.
  // Then: the index copy of tile u + 4 (into the ring slot of tile u, whose
  // indices were read at the top of u - 3), the read of tile u + 3's indices
  // into registers (used at the top of u + 1, so no wait on it here), and the
  // addresses of tile u + 2's copies from the indices read at the top of
  // u - 1.  The copies themselves are issued by the next fused step, spread
  // over its PV MFMAs, so the eight waves do not queue their copies at the
  // address unit all at once after the barrier.
  int32_t sl_next[LOADS];  // slot indices of the tile whose copies are prepared next
  KvCopies cp;
  auto tile_top = [&](int u) {
    ra_wait_vmcnt<2 * LOADS>();
    __builtin_amdgcn_s_barrier();
    issue_idx(u + 4);
    int32_t sl[LOADS];
#pragma unroll
    for (int it = 0; it < LOADS; ++it) sl[it] = sl_next[it];
    read_idx(u + 3, sl_next);
    prep_kv(u + 2, sl, cp);
  };

  // Q^T operands of the wave's four 16-query column blocks.
  bf16x8_t qT[kQB][KS];
  int qlim[kQB];  // last key position each of this lane's query columns may see
  bool qok[kQB];
  int64_t qrow[kQB];
#pragma unroll
  for (int j = 0; j < kQB; ++j) {
    const int m = 32 * wave + 16 * j + c;
    const int it = tok0 + m / grp;
    qok[j] = it < tok_end;
    qlim[j] = P + min(it, tok_end - 1);
    qrow[j] = (start + min(it, tok_end - 1)) * hq + g * grp + m % grp;
  }
  const int64_t ws_row0 = static_cast<int64_t>(sp) * total_tokens * hq;  // this split's rows in the workspace
  if (n_tiles == 0) {
    // a split past the end of a short item's keys: its rows saw no key
    // (zero output, log2-sum-exp -inf, so the merge reads finite values only)
#pragma unroll
    for (int j = 0; j < kQB; ++j) {
      if (!qok[j]) continue;
      float* wp = ws_o + (ws_row0 + qrow[j]) * D + 4 * g4;
#pragma unroll
      for (int db = 0; db < DB; ++db) *reinterpret_cast<float4*>(wp + 16 * db) = make_float4(0.f, 0.f, 0.f, 0.f);
      if (g4 == 0) ws_lse[ws_row0 + qrow[j]] = -INFINITY;
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < kQB; ++j) {
    const __bf16* qp = q + qrow[j] * D + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qT[j][ks] = __builtin_bit_cast(bf16x8_t, ra_ld16(qp + 32 * ks));
  }

  // ---- prologue ------------------------------------------------------------
#pragma unroll
  for (int t = 0; t < kRing; ++t) issue_idx(t);
  ra_wait_vmcnt<0>();
  __syncthreads();
  {
    int32_t sl0[LOADS], sl1[LOADS];
    read_idx(0, sl0);
    read_idx(1, sl1);
    read_idx(2, sl_next);
    prep_kv(0, sl0, cp);
#pragma unroll
    for (int i = 0; i < 2 * LOADS; ++i) issue_copy(cp, i);
    prep_kv(1, sl1, cp);
#pragma unroll
    for (int i = 0; i < 2 * LOADS; ++i) issue_copy(cp, i);
  }

  f32x4_t o[DB + 1][kQB];  // O^T blocks; block DB holds the row sums (A operand = ones)
#pragma unroll
  for (int i = 0; i <= DB; ++i)
#pragma unroll
    for (int j = 0; j < kQB; ++j) o[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[kQB], thr[kQB], mb[kQB];  // running max (raw units), its lazy threshold, -m * scale_log2
#pragma unroll
  for (int j = 0; j < kQB; ++j) m_run[j] = thr[j] = -INFINITY, mb[j] = 0.f;
  const float lazy_raw = kLazyLog2 / scale_log2;
  // A operand of the row-sum MFMA.  It passes through the P^T wait-state asm
  // below on every half, so the compiler cannot rematerialise it with a VALU
  // move right in front of the MFMA.
  bf16x8_t ones = __builtin_bit_cast(bf16x8_t, make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));

  // Per-lane LDS offsets.  S^T block bb of half k2 feeds A-operand row c with
  // key r = 32 k2 + 4 bb + r0, r0 = 8 (c >> 2) + (c & 3): the accumulator's
  // row group g4 then holds keys 8 g4 .. 8 g4 + 7 of the half, P^T's
  // B-operand k slots in natural order.
  const int r0 = 8 * (c >> 2) + (c & 3);
  uint32_t koff[KS];  // per k-step: row r0, logical slot 4 ks + g4
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = r0 * RB + 16 * ((4 * ks + g4) ^ ext_swz<D>(r0));
  // V^T via transposed reads: lane supplies row 32 k2 + 4 h + (8 g4 + (c >> 2))
  // and logical piece 2 db + ((c & 3) >> 1), half (c & 1).
  const int vr = 8 * g4 + (c >> 2);
  uint32_t voff[DB];  // per 16-row block db of O^T: row vr, logical slot 2 db + ((c & 3) >> 1)
#pragma unroll
  for (int db = 0; db < DB; ++db)
    voff[db] = KRING_B + vr * RB + 16 * ((2 * db + ((c & 3) >> 1)) ^ ext_swz<D>(vr)) + 8 * (c & 1);

  // S^T of one 32-key half: s[bb][j], element i = key 32 k2 + 8 g4 + 4 bb + i.
  // (Prologue only; the main loop computes S^T inside the fused step.)
  auto compute_s = [&](f32x4_t (&s)[2][kQB], int tile, int k2) {
    const unsigned char* kst = kv_lds + (tile % kStages) * TILE_B;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb) {
        const bf16x8_t a = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const uint4*>(kst + koff[ks] + (32 * k2 + 4 * bb) * RB));
#pragma unroll
        for (int j = 0; j < kQB; ++j) {
          if (ks == 0) s_mfma_first(s[bb][j], a, qT[j][ks]);
          else s_mfma_acc(s[bb][j], a, qT[j][ks]);
        }
      }
    // let the last MFMAs retire before the VALU reads S^T (every block is an
    // operand, so no MFMA writing one can be scheduled past the nops)
    asm volatile("s_nop 7\n\ts_nop 7" : "+v"(s[0][0]), "+v"(s[0][1]), "+v"(s[1][0]), "+v"(s[1][1]));
  };

  // Maximum of one half's scores per query column (this lane's 8 keys).
  auto half_max = [&](f32x4_t (&s)[2][kQB], int j) {
    float m = __builtin_fmaxf(__builtin_fmaxf(s[0][j][0], s[0][j][1]), s[0][j][2]);
    m = __builtin_fmaxf(__builtin_fmaxf(m, s[0][j][3]), s[1][j][0]);
    m = __builtin_fmaxf(__builtin_fmaxf(m, s[1][j][1]), s[1][j][2]);
    return __builtin_fmaxf(m, s[1][j][3]);
  };

  // After a half's S^T is complete and its per-lane maxima mt are known:
  // causal mask (diagonal halves only, maxima recomputed), then the rare move
  // of the running maximum with its rescale of O^T.
  auto pre = [&](f32x4_t (&s)[2][kQB], int tile, int k2, float (&mt)[kQB]) {
    const int kh = kt0 + tile * kBN + 32 * k2;  // first key of the half
    if (kh + 31 > P + tok0) {
#pragma unroll
      for (int j = 0; j < kQB; ++j) {
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (kh + 8 * g4 + 4 * bb + i > qlim[j]) s[bb][j][i] = -INFINITY;
        mt[j] = half_max(s, j);
      }
    }
    bool up = false;
#pragma unroll
    for (int j = 0; j < kQB; ++j) up |= mt[j] > thr[j];
    if (__builtin_amdgcn_ballot_w64(up) != 0) {
      // Rare: some column's maximum passed its threshold.  Move those
      // columns' maxima and rescale their O^T.  The nops give the last
      // MFMAs that wrote O time to retire before the VALU reads the AGPRs.
#pragma unroll
      for (int j = 0; j < kQB; ++j) {
        const float mc = ra_max_across_rows(mt[j]);
        float alpha = 1.f;
        if (mc > thr[j]) {
          alpha = ra_exp2((m_run[j] - mc) * scale_log2);  // 0 while m_run = -inf (O is still 0)
          m_run[j] = mc;
          thr[j] = mc + lazy_raw;
          mb[j] = -mc * scale_log2;
        }
        if constexpr (DB == 8) {
          asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3"
                       : "+a"(o[0][j]), "+a"(o[1][j]), "+a"(o[2][j]), "+a"(o[3][j]), "+a"(o[4][j]),
                         "+a"(o[5][j]), "+a"(o[6][j]), "+a"(o[7][j]), "+a"(o[8][j]));
        } else {
          asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3"
                       : "+a"(o[0][j]), "+a"(o[1][j]), "+a"(o[2][j]), "+a"(o[3][j]), "+a"(o[4][j]));
        }
#pragma unroll
        for (int db = 0; db <= DB; ++db) o[db][j] *= alpha;
        // two wait states between the VALU writes of O and the next MFMA
        if constexpr (DB == 8) {
          asm volatile("s_nop 1"
                       : "+a"(o[0][j]), "+a"(o[1][j]), "+a"(o[2][j]), "+a"(o[3][j]), "+a"(o[4][j]),
                         "+a"(o[5][j]), "+a"(o[6][j]), "+a"(o[7][j]), "+a"(o[8][j]));
        } else {
          asm volatile("s_nop 1" : "+a"(o[0][j]), "+a"(o[1][j]), "+a"(o[2][j]), "+a"(o[3][j]), "+a"(o[4][j]));
        }
      }
    }
  };

  // One software-pipelined step over two halves, written in issue order:
  // the S^T MFMAs of the next half sn, each followed by one probability of
  // the current half sc (fma + exp, pack every second), with the K operand
  // reads two k-steps ahead and the V^T reads of the current half in the
  // second part; then the current half's PV MFMAs (AGPR accumulators, inline
  // assembly), the next half's per-lane maxima slotted between them.
  // sched_barrier(0) fences keep the scheduler from regrouping the MFMAs and
  // the VALU work, so the matrix core stays busy while the exponentials issue.
  // HAS_NEXT = false is the last half of the item (no S^T to compute).
  // kpre holds the K operands of sn's first two k-steps (read by the previous
  // step); at the end of the PV part the step reads those of the half after
  // sn, (tile_f, k2_f), when pf is set (its tile is resident by then).
  constexpr int KP = KS > 1 ? 2 : 1;  // k-steps prefetched across steps
  // with_copies: issue the copies prepared by the last tile_top, one every
  // DB / (2 LOADS) PV steps.  The ring stages of the halves (sk_n: K of sn,
  // sv_c: V of sc, sk_f: K of the half after sn) come as compile-time
  // constants in the steady loops, so every operand read is a per-lane
  // offset plus an immediate.
  auto fused = [&](auto has_next, auto with_copies, f32x4_t (&sn)[2][kQB], auto sk_n, int k2_n,
                   f32x4_t (&sc)[2][kQB], auto sv_c, int k2_c, float (&mt)[kQB], bf16x8_t (&kpre)[KP][2], bool pf,
                   auto sk_f, int k2_f) {
    constexpr bool HAS_NEXT = decltype(has_next)::value;
    constexpr bool COPIES = decltype(with_copies)::value;
    constexpr int CSTEP = DB / (2 * LOADS) > 0 ? DB / (2 * LOADS) : 1;
    constexpr int NS = 2 * KS * kQB;  // S^T MFMAs of one half
    constexpr int NP = 8 * kQB;       // probabilities per lane per half
    constexpr int VA = 3;             // V^T operands (16-row blocks) read ahead of their PV step
    const unsigned char* kst = kv_lds + static_cast<int>(sk_n) * TILE_B + 32 * k2_n * RB;
    const unsigned char* vst = kv_lds + static_cast<int>(sv_c) * TILE_B + 32 * k2_c * RB;
    bf16x8_t kf[KS][2];
    bf16x4_t vf[DB][2];
    float p[NP];
    uint32_t pw[NP / 2];
    auto read_k = [&](int ks) {
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
        kf[ks][bb] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(kst + koff[ks] + 4 * bb * RB));
    };
    auto read_v = [&](int db) {
      const unsigned char* vb = vst + voff[db];
#pragma unroll
      for (int h = 0; h < 2; ++h)
        vf[db][h] =
            __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4_t*)(vb + h * 4 * RB));
    };
    auto prob = [&](int v) {  // v = 8 j + 4 bb + i
      const int j = v >> 3, bb = (v >> 2) & 1, i = v & 3;
      p[v] = ra_exp2(__builtin_fmaf(sc[bb][j][i], scale_log2, mb[j]));
      if (v & 1) pw[v >> 1] = ra_pack_bf16x2(p[v - 1], p[v]);
    };
    // The same in three stages, so that the steps of one probability sit in
    // different MFMA groups and never wait on each other's latency.
    auto prob_fma = [&](int v) {
      const int j = v >> 3, bb = (v >> 2) & 1, i = v & 3;
      p[v] = __builtin_fmaf(sc[bb][j][i], scale_log2, mb[j]);
    };
    auto prob_exp = [&](int v) { p[v] = ra_exp2(p[v]); };
    auto prob_pack = [&](int v) {
      if (v & 1) pw[v >> 1] = ra_pack_bf16x2(p[v - 1], p[v]);
    };
    if constexpr (HAS_NEXT) {
#pragma unroll
      for (int ks = 0; ks < KP; ++ks)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) kf[ks][bb] = kpre[ks][bb];
      __builtin_amdgcn_sched_barrier(0);
      constexpr int PPG = (NP + NS - 1) / NS;  // probabilities per S^T MFMA
#pragma unroll
      for (int v = 0; v < PPG && v < NP; ++v) prob_fma(v);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int n = 0; n < NS; ++n) {
        const int ks = n / (2 * kQB), bb = (n / kQB) & 1, j = n % kQB;
        if (ks == 0) s_mfma_first(sn[bb][j], kf[ks][bb], qT[j][ks]);
        else s_mfma_acc(sn[bb][j], kf[ks][bb], qT[j][ks]);
        // group n: fma of the next group's values, exp of this group's,
        // packs of the previous group's
#pragma unroll
        for (int v = (n + 1) * PPG; v < (n + 2) * PPG && v < NP; ++v) prob_fma(v);
#pragma unroll
        for (int v = n * PPG; v < (n + 1) * PPG && v < NP; ++v) prob_exp(v);
#pragma unroll
        for (int v = (n - 1) * PPG; v < n * PPG && v >= 0 && v < NP; ++v) prob_pack(v);
        if (n % (2 * kQB) == 2 * kQB - 1 && ks + 2 < KS) read_k(ks + 2);
        // the first V^T operands, spread over the last S^T MFMAs
        if (n >= NS - VA && n - (NS - VA) < DB) read_v(n - (NS - VA));
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int v = (NS - 1) * PPG; v < NS * PPG && v < NP; ++v) prob_pack(v);
#pragma unroll
      for (int v = NS * PPG; v < NP; ++v) prob(v);
    } else {
#pragma unroll
      for (int db = 0; db < VA && db < DB; ++db) read_v(db);
#pragma unroll
      for (int v = 0; v < NP; ++v) prob(v);
    }
    bf16x8_t pT[kQB];
#pragma unroll
    for (int j = 0; j < kQB; ++j)
      pT[j] = __builtin_bit_cast(bf16x8_t, make_uint4(pw[4 * j], pw[4 * j + 1], pw[4 * j + 2], pw[4 * j + 3]));
    // two wait states between the VALU writes of P^T and the MFMAs reading it
    asm volatile("s_nop 1" : "+v"(pT[0]), "+v"(pT[1]), "+v"(ones));
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      if (db + VA < DB) read_v(db + VA);
      const bf16x8_t a = __builtin_shufflevector(vf[db][0], vf[db][1], 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
      for (int j = 0; j < kQB; ++j) pv_mfma(o[db][j], a, pT[j]);
      // the next half's maxima, one column per PV step once its S^T has retired
      if constexpr (HAS_NEXT) {
        if (db >= 2 && db - 2 < kQB) mt[db - 2] = half_max(sn, db - 2);
      }
      if constexpr (COPIES) {
        if (db % CSTEP == CSTEP - 1 && db / CSTEP < 2 * LOADS) issue_copy(cp, db / CSTEP);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < kQB; ++j) pv_mfma(o[DB][j], ones, pT[j]);
    if constexpr (COPIES) {
#pragma unroll
      for (int i = DB / CSTEP; i < 2 * LOADS; ++i) issue_copy(cp, i);
    }
    if (pf) {
      const unsigned char* kf_st = kv_lds + static_cast<int>(sk_f) * TILE_B + 32 * k2_f * RB;
#pragma unroll
      for (int ks = 0; ks < KP; ++ks)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
          kpre[ks][bb] =
              __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(kf_st + koff[ks] + 4 * bb * RB));
    }
    if constexpr (HAS_NEXT) {
      if constexpr (DB - 2 < kQB) {
#pragma unroll
        for (int j = (DB - 2 > 0 ? DB - 2 : 0); j < kQB; ++j) mt[j] = half_max(sn, j);
      }
    }
  };

  // ---- main loop: half h's exponentials and PV run beside half h+1's S^T ---
  // Every wave takes the tile barrier at the top of its iteration.  The K
  // operands of each step's first two k-steps were read at the end of the
  // step before (for the first half of tile t + 1 that read comes after the
  // barrier of the top of t + 1, so the tile is resident).
  using yes = std::integral_constant<bool, true>;
  using no = std::integral_constant<bool, false>;
  f32x4_t sa[2][kQB], sb[2][kQB];
  float mt[kQB];
  bf16x8_t kpre[KP][2];
  // A wave whose 32 query rows are all past the request's last new token
  // (short extends leave part of the tile empty) still takes every tile
  // barrier and issues its share of each tile's copies, but computes
  // nothing, leaving its SIMD to the other wave.
  if (tok0 + (32 * wave) / grp >= tok_end) {
    for (int u = 0; u < n_tiles; ++u) {
      tile_top(u);
#pragma unroll
      for (int i = 0; i < 2 * LOADS; ++i) issue_copy(cp, i);
    }
    ra_wait_vmcnt<0>();
    return;
  }
  tile_top(0);
#pragma unroll
  for (int i = 0; i < 2 * LOADS; ++i) issue_copy(cp, i);
  compute_s(sa, 0, 0);
#pragma unroll
  for (int j = 0; j < kQB; ++j) mt[j] = half_max(sa, j);
  // K operands of the first two k-steps of a half, read ahead of its step
  auto load_kpre = [&](auto stage, int k2) {
    const unsigned char* kf_st = kv_lds + static_cast<int>(stage) * TILE_B + 32 * k2 * RB;
#pragma unroll
    for (int ks = 0; ks < KP; ++ks)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
        kpre[ks][bb] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(kf_st + koff[ks] + 4 * bb * RB));
  };
  if constexpr (BN == 64) load_kpre(ic<0>{}, 1);
  pre(sa, 0, 0, mt);
  // The last tile is peeled off the loop so that no branch inside it has two
  // sides computing the same probabilities (the compiler would hoist them out
  // of the fused step).
  if constexpr (BN == 64) {
    // one tile per call; the tile's ring stage J = t % kStages is a constant
    int t = 0;
    auto tile_body = [&](auto J) -> bool {
      constexpr int j = decltype(J)::value, j1 = (j + 1) % kStages;
      if (t + 1 >= n_tiles) return false;
      tile_top(t + 1);
      fused(yes{}, yes{}, sb, ic<j>{}, 1, sa, ic<j>{}, 0, mt, kpre, true, ic<j1>{}, 0);
      pre(sb, t, 1, mt);
      fused(yes{}, no{}, sa, ic<j1>{}, 0, sb, ic<j>{}, 1, mt, kpre, true, ic<j1>{}, 1);
      pre(sa, t + 1, 0, mt);
      ++t;
      return true;
    };
    while (tile_body(ic<0>{}) && tile_body(ic<1>{}) && tile_body(ic<2>{}) && tile_body(ic<3>{})) {
    }
    const int ts = t % kStages;
    fused(yes{}, no{}, sb, ts, 1, sa, ts, 0, mt, kpre, false, 0, 0);
    pre(sb, t, 1, mt);
    fused(no{}, no{}, sa, 0, 0, sb, ts, 1, mt, kpre, false, 0, 0);
  } else {
    // One half per tile: the step of tile t + 1 follows that tile's barrier
    // (its K operands are read there); two tiles per iteration so the S^T
    // buffers alternate without copies.  (The ring stages stay runtime
    // values here: unrolled over them, this shape's register allocation
    // moves accumulators next to the inline-assembly MFMAs.)
    int t = 0;
    for (; t + 2 < n_tiles; t += 2) {
      const int s0 = t % kStages, s1 = (t + 1) % kStages, s2 = (t + 2) % kStages;
      tile_top(t + 1);
      load_kpre(s1, 0);
      fused(yes{}, yes{}, sb, s1, 0, sa, s0, 0, mt, kpre, false, 0, 0);
      pre(sb, t + 1, 0, mt);
      tile_top(t + 2);
      load_kpre(s2, 0);
      fused(yes{}, yes{}, sa, s2, 0, sb, s1, 0, mt, kpre, false, 0, 0);
      pre(sa, t + 2, 0, mt);
    }
    const int ts = t % kStages, ts1 = (t + 1) % kStages;
    if (t + 1 < n_tiles) {
      tile_top(t + 1);
      load_kpre(ts1, 0);
      fused(yes{}, yes{}, sb, ts1, 0, sa, ts, 0, mt, kpre, false, 0, 0);
      pre(sb, t + 1, 0, mt);
      fused(no{}, no{}, sa, 0, 0, sb, ts1, 0, mt, kpre, false, 0, 0);
    } else {
      fused(no{}, no{}, sb, 0, 0, sa, ts, 0, mt, kpre, false, 0, 0);
    }
  }

  // No copy may still be landing in LDS once the work-group ends (the last
  // index copies were issued past the final tile).
  ra_wait_vmcnt<0>();
  // Epilogue: let the last MFMAs retire, then normalise by the row sums.
#pragma unroll
  for (int j = 0; j < kQB; ++j) {
    if constexpr (DB == 8) {
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3"
                   : "+a"(o[0][j]), "+a"(o[1][j]), "+a"(o[2][j]), "+a"(o[3][j]), "+a"(o[4][j]), "+a"(o[5][j]),
                     "+a"(o[6][j]), "+a"(o[7][j]), "+a"(o[8][j]));
    } else {
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3"
                   : "+a"(o[0][j]), "+a"(o[1][j]), "+a"(o[2][j]), "+a"(o[3][j]), "+a"(o[4][j]));
    }
  }
  if (nsplit > 1) {
    // Partial output over this split's keys.  A row whose keys all lie past
    // its causal limit has a zero sum: zero output, log2-sum-exp -inf.
#pragma unroll
    for (int j = 0; j < kQB; ++j) {
      if (!qok[j]) continue;
      const float l = o[DB][j][0];
      const float inv = l > 0.f ? 1.f / l : 0.f;
      float* wp = ws_o + (ws_row0 + qrow[j]) * D + 4 * g4;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<float4*>(wp + 16 * db) =
            make_float4(o[db][j][0] * inv, o[db][j][1] * inv, o[db][j][2] * inv, o[db][j][3] * inv);
      if (g4 == 0) ws_lse[ws_row0 + qrow[j]] = l > 0.f ? m_run[j] * scale_log2 + __log2f(l) : -INFINITY;
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < kQB; ++j) {
    if (!qok[j]) continue;
    const float inv = 1.f / o[DB][j][0];
    __bf16* op = out + qrow[j] * D + 4 * g4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      uint2 w;
      w.x = ra_pack_bf16x2(o[db][j][0] * inv, o[db][j][1] * inv);
      w.y = ra_pack_bf16x2(o[db][j][2] * inv, o[db][j][3] * inv);
      *reinterpret_cast<uint2*>(op + 16 * db) = w;
    }
  }
}

// Merges the key splits of every new token's rows: each request's output
// rows [start, start + E) x Hq x D are one contiguous run, read four values
// per thread; weights 2^(lse_i - max lse) (0 for a split that saw no key of
// the row: lse -inf, output zero).  The loads of two splits go out before any
// is used, so a thread waits for memory once per pair of splits.  max_tok
// bounds E as the extend kernel's query tiles do.
template <int D>
__global__ __launch_bounds__(256) void extend_combine_kernel(const float* __restrict__ ws_o,
                                                             const float* __restrict__ ws_lse,
                                                             const int32_t* __restrict__ extend_lens,
                                                             const int32_t* __restrict__ extend_start,
                                                             int64_t total_tokens, int32_t max_tok, int32_t hq,
                                                             int32_t nsplit, __bf16* __restrict__ out) {
  const int b = blockIdx.x;  // request (the grid's y extent is limited to 65535)
  const int64_t start = extend_start[b];
  if (start < 0 || start > total_tokens) return;
  const int64_t E = min(min<int64_t>(extend_lens[b], total_tokens - start), static_cast<int64_t>(max_tok));
  const int64_t n4 = E * hq * (D / 4);                 // four-value groups of the request
  const int64_t rows_total = total_tokens * hq;        // rows per split
  const int64_t base = start * hq * (D / 4);
  for (int64_t i = static_cast<int64_t>(blockIdx.y) * 256 + threadIdx.x; i < n4;
       i += static_cast<int64_t>(gridDim.y) * 256) {
    const int64_t e = base + i;
    const int64_t row = e / (D / 4);
    float m = -INFINITY, wsum = 0.f;  // running maximum of the lse seen, weight sum
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < nsplit; s0 += 2) {
      float l[2];
      float4 v[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int64_t s = min(s0 + k, nsplit - 1);  // an odd count repeats the last split, weighted 0
        l[k] = ws_lse[s * rows_total + row];
        v[k] = *reinterpret_cast<const float4*>(ws_o + (s * rows_total) * D + 4 * e);
      }
      if (s0 + 1 >= nsplit) l[1] = -INFINITY;
      const float mn = fmaxf(m, fmaxf(l[0], l[1]));
      if (mn == -INFINITY) continue;
      const float a = ra_exp2(m - mn);  // 0 while m = -inf
      wsum *= a;
      acc.x *= a, acc.y *= a, acc.z *= a, acc.w *= a;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const float w = ra_exp2(l[k] - mn);
        wsum += w;
        acc.x += w * v[k].x, acc.y += w * v[k].y, acc.z += w * v[k].z, acc.w += w * v[k].w;
      }
      m = mn;
    }
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    uint2 w;
    w.x = ra_pack_bf16x2(acc.x * inv, acc.y * inv);
    w.y = ra_pack_bf16x2(acc.z * inv, acc.w * inv);
    *reinterpret_cast<uint2*>(out + 4 * e) = w;
  }
}

template <int D, int WAVES, int BN>
void launch_wide(int64_t items, hipStream_t stream, const __bf16* qp, const __bf16* knp, const __bf16* vnp,
                 int64_t total_tokens, const __bf16* kp, const __bf16* vp, int64_t pool_slots, const int32_t* rtt,
                 int64_t rtt_rows, int64_t rtt_stride, const int32_t* rpi, const int32_t* pl, const int32_t* el,
                 const int32_t* es, int32_t batch, int32_t hkv, int32_t grp, int32_t n_qtiles, int32_t lpt, float scale_log2,
                 int32_t nsplit, float* ws_o, float* ws_lse, __bf16* op) {
  hipLaunchKernelGGL((extend_kernel<D, WAVES, BN>), dim3(static_cast<uint32_t>(items)), dim3(WAVES * 64), 0,
                     stream, qp, knp, vnp, total_tokens, kp, vp, pool_slots, rtt, rtt_rows, rtt_stride, rpi, pl, el,
                     es, batch, hkv, grp, n_qtiles, lpt, scale_log2, nsplit, ws_o, ws_lse, op);
}

// Shape and key splits of a call: 256 or 128 query rows per work-group and
// the number of key splits per item.
struct ExtendPlan {
  int32_t rows;
  int32_t nsplit;
};

// num_splits < 0: the entry point without a workspace (no splits).  At least
// 256 query rows per kv head (new tokens x query heads per kv head) take the
// 256-row configuration; fewer would leave most of its tile empty, so they
// take the 128-row one.  Without splits the 128-row one also serves a batch
// whose 256-row work-groups would not reach one per CU (few requests and few
// kv heads, e.g. a head shard): twice the work-groups, so more CUs share the
// work.  With num_splits = 0 such a batch keeps its shape and its items' keys
// are split until the work-groups fill every work-group slot of the chip
// once; num_splits > 0 asks for that many splits (at most kMaxSplits).
ExtendPlan extend_plan(int32_t batch, int32_t max_extend_len, int32_t grp, int32_t hkv, int32_t num_splits) {
  ExtendPlan pl{static_cast<int64_t>(max_extend_len) * grp >= 256 ? 256 : 128, 1};
  const int32_t tpb = pl.rows / grp;
  const int64_t items = static_cast<int64_t>(batch) * hkv * ((static_cast<int64_t>(max_extend_len) + tpb - 1) / tpb);
  const int64_t slots = static_cast<int64_t>(ra_device_cus()) * (pl.rows == 256 ? 1 : 2);
  if (num_splits < 0) {
    if (pl.rows == 256 && items < ra_device_cus()) pl.rows = 128;
  } else if (num_splits > 0) {
    pl.nsplit = std::min(num_splits, kMaxSplits);
  } else if (items > 0 && items < slots) {
    pl.nsplit = static_cast<int32_t>(std::min<int64_t>(kMaxSplits, (slots + items - 1) / items));
  }
  return pl;
}

}  // namespace

// Compute units of the current device (cached per device; 256 if the query
// fails).
int ra_device_cus() {
  static std::atomic<int> cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Launches the fused-step kernel with 256 (rows = 256) or 128 query rows per
// work-group for arguments ra_extend_validate accepted.
static int extend_launch(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                          const void* k_pool, const void* v_pool, int64_t pool_slots, const int32_t* req_to_token,
                          int64_t rtt_rows, int64_t rtt_stride, const int32_t* req_pool_idx,
                          const int32_t* prefix_lens, const int32_t* extend_lens, const int32_t* extend_start,
                          int32_t batch, int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                          void* out, ExtendPlan plan, void* workspace, hipStream_t stream) {
  const int32_t grp = hq / hkv;
  const int32_t rows = plan.rows;
  const int32_t tpb = (rows == 256 ? 256 : 128) / grp;
  const int64_t n_qtiles = (static_cast<int64_t>(max_extend_len) + tpb - 1) / tpb;
  const int64_t items = (static_cast<int64_t>(batch) * hkv * n_qtiles * plan.nsplit + 7) / 8 * 8;  // whole XCD rounds
  if (items > INT32_MAX) return ra_fail(RA_EINVAL, "ra_extend_attention: too many work items");
  const float scale_log2 = scale * RA_LOG2E;
  auto* qp = static_cast<const __bf16*>(q);
  auto* knp = static_cast<const __bf16*>(k_new);
  auto* vnp = static_cast<const __bf16*>(v_new);
  auto* kp = static_cast<const __bf16*>(k_pool);
  auto* vp = static_cast<const __bf16*>(v_pool);
  auto* op = static_cast<__bf16*>(out);
  const int32_t nq = static_cast<int32_t>(n_qtiles);
  float* ws_o = plan.nsplit > 1 ? static_cast<float*>(workspace) : nullptr;
  float* ws_lse = plan.nsplit > 1 ? ws_o + static_cast<int64_t>(plan.nsplit) * total_tokens * hq * d : nullptr;
  // Longest first only matters when the work-groups take more than one round
  // of the chip's work-group slots (two per CU with 128 rows, one with 256).
  const int64_t slots = static_cast<int64_t>(ra_device_cus()) * (rows == 256 ? 1 : 2);
  const int32_t lpt = batch <= kLptMaxBatch && items > slots ? 1 : 0;
#define RA_WIDE_LAUNCH(DD, W, B)                                                                                   \
  launch_wide<DD, W, B>(items, stream, qp, knp, vnp, total_tokens, kp, vp, pool_slots, req_to_token, rtt_rows,     \
                        rtt_stride, req_pool_idx, prefix_lens, extend_lens, extend_start, batch, hkv, grp, nq, lpt, \
                        scale_log2, plan.nsplit, ws_o, ws_lse, op)
  if (rows == 256) {
    if (d == 128) RA_WIDE_LAUNCH(128, 8, 64);
    else RA_WIDE_LAUNCH(64, 8, 64);
  } else {
    if (d == 128) RA_WIDE_LAUNCH(128, 4, 32);
    else RA_WIDE_LAUNCH(64, 4, 32);
  }
#undef RA_WIDE_LAUNCH
  int st = ra_check_launch("ra_extend_attention(fused)");
  if (st != RA_OK || plan.nsplit <= 1) return st;
  const int64_t max_tok = n_qtiles * tpb;
  const int64_t groups = max_tok * hq * d / 4;
  const dim3 cgrid(static_cast<uint32_t>(batch), static_cast<uint32_t>(std::min<int64_t>((groups + 255) / 256, 1024)));
  if (d == 128)
    hipLaunchKernelGGL(extend_combine_kernel<128>, cgrid, dim3(256), 0, stream, ws_o, ws_lse, extend_lens,
                       extend_start, total_tokens, static_cast<int32_t>(max_tok), hq, plan.nsplit, op);
  else
    hipLaunchKernelGGL(extend_combine_kernel<64>, cgrid, dim3(256), 0, stream, ws_o, ws_lse, extend_lens,
                       extend_start, total_tokens, static_cast<int32_t>(max_tok), hq, plan.nsplit, op);
  return ra_check_launch("ra_extend_attention(combine)");
}

// Argument checks shared with ra_mixed_attention: RA_OK when the call may
// launch (or has nothing to do), an error status otherwise.
int ra_extend_validate(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                       const void* k_pool, const void* v_pool, int64_t pool_slots, const int32_t* req_to_token,
                       int64_t rtt_rows, int64_t rtt_stride, const int32_t* req_pool_idx,
                       const int32_t* prefix_lens, const int32_t* extend_lens, const int32_t* extend_start,
                       int32_t batch, int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                       void* out) {
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0 || (d != 64 && d != 128) || pool_slots <= 0 ||
      rtt_rows <= 0 || rtt_stride <= 0 || max_extend_len < 0 || total_tokens < 0 || !(scale > 0.f))
    return ra_fail(RA_EINVAL, "ra_extend_attention: bad sizes or scale");
  const int32_t grp = hq / hkv;
  if (grp != 1 && grp != 2 && grp != 4 && grp != 8 && grp != 16)
    return ra_fail(RA_EINVAL, "ra_extend_attention: Hq / Hkv must be 1, 2, 4, 8 or 16");
  if (batch == 0 || max_extend_len == 0 || total_tokens == 0) return ra_ok();
  if (!q || !k_new || !v_new || !k_pool || !v_pool || !req_to_token || !req_pool_idx || !prefix_lens ||
      !extend_lens || !extend_start || !out)
    return ra_fail(RA_EINVAL, "ra_extend_attention: NULL pointer");
  if (!ra_aligned16(q) || !ra_aligned16(k_new) || !ra_aligned16(v_new) || !ra_aligned16(k_pool) ||
      !ra_aligned16(v_pool) || !ra_aligned16(out))
    return ra_fail(RA_EINVAL, "ra_extend_attention: pointers must be 16-byte aligned");
  return ra_ok();
}

extern "C" int ra_extend_attention(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                                   const void* k_pool, const void* v_pool, int64_t pool_slots,
                                   const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                   const int32_t* req_pool_idx, const int32_t* prefix_lens,
                                   const int32_t* extend_lens, const int32_t* extend_start, int32_t batch,
                                   int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                                   void* out, hipStream_t stream) {
  const int st = ra_extend_validate(q, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows,
                                    rtt_stride, req_pool_idx, prefix_lens, extend_lens, extend_start, batch,
                                    max_extend_len, hq, hkv, d, scale, out);
  if (st != RA_OK || batch == 0 || max_extend_len == 0 || total_tokens == 0) return st;
  if (ra_debug_checks_enabled()) {
    const int cst = ra_check_batch(req_to_token, rtt_rows, rtt_stride, pool_slots, req_pool_idx, batch, prefix_lens,
                                   extend_lens, extend_start, total_tokens, max_extend_len, nullptr, 0, stream);
    if (cst != RA_OK) return cst;
  }
  const ExtendPlan plan = extend_plan(batch, max_extend_len, hq / hkv, hkv, -1);
  return extend_launch(q, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride,
                       req_pool_idx, prefix_lens, extend_lens, extend_start, batch, max_extend_len, hq, hkv, d,
                       scale, out, plan, nullptr, stream);
}

extern "C" int32_t ra_extend_num_splits(int32_t batch, int32_t max_extend_len, int32_t hq, int32_t hkv,
                                        int32_t num_splits) {
  if (batch <= 0 || max_extend_len <= 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0 || num_splits < 0) return 1;
  return extend_plan(batch, max_extend_len, hq / hkv, hkv, num_splits).nsplit;
}

extern "C" size_t ra_extend_workspace_bytes(int64_t total_tokens, int32_t batch, int32_t max_extend_len, int32_t hq,
                                            int32_t hkv, int32_t d, int32_t num_splits) {
  if (total_tokens <= 0 || d <= 0) return 0;
  const int32_t ns = ra_extend_num_splits(batch, max_extend_len, hq, hkv, num_splits);
  if (ns <= 1) return 0;
  return static_cast<size_t>(ns) * static_cast<size_t>(total_tokens) * hq * (d + 1) * sizeof(float);
}

extern "C" int ra_extend_attention_split(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                                         const void* k_pool, const void* v_pool, int64_t pool_slots,
                                         const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                         const int32_t* req_pool_idx, const int32_t* prefix_lens,
                                         const int32_t* extend_lens, const int32_t* extend_start, int32_t batch,
                                         int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                                         int32_t num_splits, void* workspace, size_t workspace_bytes, void* out,
                                         hipStream_t stream) {
  if (num_splits < 0) return ra_fail(RA_EINVAL, "ra_extend_attention_split: negative num_splits");
  const int st = ra_extend_validate(q, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows,
                                    rtt_stride, req_pool_idx, prefix_lens, extend_lens, extend_start, batch,
                                    max_extend_len, hq, hkv, d, scale, out);
  if (st != RA_OK || batch == 0 || max_extend_len == 0 || total_tokens == 0) return st;
  const ExtendPlan plan = extend_plan(batch, max_extend_len, hq / hkv, hkv, num_splits);
  if (plan.nsplit > 1) {
    const size_t need = ra_extend_workspace_bytes(total_tokens, batch, max_extend_len, hq, hkv, d, num_splits);
    if (workspace_bytes < need || !workspace)
      return ra_fail(RA_EINVAL, "ra_extend_attention_split: workspace too small");
    if (!ra_aligned16(workspace)) return ra_fail(RA_EINVAL, "ra_extend_attention_split: workspace alignment");
  }
  if (ra_debug_checks_enabled()) {
    const int cst = ra_check_batch(req_to_token, rtt_rows, rtt_stride, pool_slots, req_pool_idx, batch, prefix_lens,
                                   extend_lens, extend_start, total_tokens, max_extend_len, nullptr, 0, stream);
    if (cst != RA_OK) return cst;
  }
  return extend_launch(q, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride,
                       req_pool_idx, prefix_lens, extend_lens, extend_start, batch, max_extend_len, hq, hkv, d,
                       scale, out, plan, workspace, stream);
}
