// Extend attention: prefill of a request's new tokens over its cached prefix
// (the work that remains once RadixAttention has reused the prefix's KV
// cache; section 3, Appendix A.1), plus causal attention among the new
// tokens.  This is a dense contraction, so QK^T and PV run on bf16 MFMA
// (v_mfma_f32_16x16x32_bf16) with fp32 accumulation.
//
// Work item = (request, kv head, query tile).  A tile holds 128 query rows
// packed as (new token, query head of the kv head's group): the G heads that
// share a kv head share every K/V tile the work-group stages.  Four waves of
// 32 rows.  Per 64-key tile:
//   * K and V rows are copied HBM -> LDS by direct-to-LDS loads
//     (global_load_lds_dwordx4), no VGPR staging.  Prefix keys are gathered
//     through the request's slot-table row, new keys come from the contiguous
//     k_new / v_new rows.  The slot indices themselves travel by DMA into a
//     small LDS ring two tiles ahead, so a tile's gather never waits on its
//     index load.  The K/V ring has two stages.
//   * A DMA writes lane i's 16 bytes at base + 16 i, so rows sit unpadded at
//     2*D bytes; the 16-byte pieces of row r are XOR-swizzled by ra_kv_swz(r) (the
//     source address picks the piece) to spread LDS banks.
//   * S^T[key, query] = K Q^T with the queries as the MFMA columns: each lane
//     owns one query column, so the row max / row sum are in-lane plus two
//     cross-row shuffles.  K rows are fed to the A operand in the order that
//     makes the accumulator's four 16-lane row groups hold keys 8g..8g+7 of
//     each 32-key step, which is exactly P^T's B-operand layout.
//   * O^T += V^T P^T: V stays row-major in LDS; ds_read_b64_tr_b16 reads it
//     transposed (lane i of a 16-lane group gets column i of four rows), two
//     reads per A operand.
// The DMAs are issued from inline assembly: the compiler would otherwise
// wait for every outstanding DMA before each LDS read, serialising the
// pipeline.  Waits are explicit s_waitcnt vmcnt at the top of each tile.
#include <type_traits>

#include "device_common.h"
#include "lds_dma.h"

namespace {

constexpr int kBM = 128;  // query rows per work-group
constexpr int kBN = 64;   // keys per tile
constexpr int64_t kWideMinRows = 256;  // query rows per kv head from which the 256-row kernel is used

template <int D>
__global__ __launch_bounds__(256, 2) void extend_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k_new, const __bf16* __restrict__ v_new,
    int64_t total_tokens, const __bf16* __restrict__ k_pool, const __bf16* __restrict__ v_pool,
    int64_t pool_slots, const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride,
    const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ prefix_lens,
    const int32_t* __restrict__ extend_lens, const int32_t* __restrict__ extend_start, int32_t batch,
    int32_t hkv, int32_t grp, int32_t n_qtiles, float scale_log2, __bf16* __restrict__ out) {
  constexpr int KS = D / 32;                  // MFMA k-steps over the head dimension = piece groups
  constexpr int DB = D / 16;                  // 16-row blocks of O^T
  constexpr int GROUP_B = kBN * 64;           // bytes of one piece group of a tile
  constexpr int TILE_B = KS * GROUP_B;        // bytes per K (or V) tile
  constexpr int LOADS = TILE_B / (256 * 16);  // DMA instructions per wave per tile per tensor
  constexpr int RING = 4;                     // slot-index ring depth
  // A wave's DMA lane covers tile rows u0 + it * ROW_STEP (it < LOADS); the
  // index ring stores row u at word LOADS * (u % ROW_STEP) + u / ROW_STEP so
  // that a lane's LOADS slot indices are one vector LDS read.
  constexpr int ROW_STEP = kBN / LOADS;
  static_assert(LOADS == 2 || LOADS == 4, "index vector width");
  __shared__ __align__(16) unsigned char kv_lds[2][2][TILE_B];
  __shared__ __align__(16) int32_t idx_lds[RING][kBN];

  // Work-groups go to the 8 XCDs round-robin (block i -> XCD i % 8).  Items
  // are ordered (kv head, request, query tile, longest tile first) and each
  // XCD takes a contiguous eighth of that order, so the work-groups in flight
  // on one XCD share a kv head and mostly one request: they stream the same
  // K/V rows and hit that XCD's L2.
  const int64_t n_items = static_cast<int64_t>(hkv) * batch * n_qtiles;
  const int64_t per_xcd = (n_items + 7) / 8;
  const int64_t item = static_cast<int64_t>(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (item >= n_items) return;
  const int g = static_cast<int>(item / (static_cast<int64_t>(batch) * n_qtiles));
  const int rem = static_cast<int>(item % (static_cast<int64_t>(batch) * n_qtiles));
  const int b = rem / n_qtiles;
  const int qt = n_qtiles - 1 - rem % n_qtiles;
  const int tpb = kBM / grp;  // new tokens per tile

  const int64_t start = extend_start[b];
  int64_t E = extend_lens[b];
  if (start < 0 || start > total_tokens) return;
  E = min(E, total_tokens - start);
  const int tok0 = qt * tpb;
  if (E <= 0 || tok0 >= E) return;
  const int tok_end = static_cast<int>(min<int64_t>(E, tok0 + tpb));
  const int P = static_cast<int>(min<int64_t>(max(prefix_lens[b], 0), rtt_stride));
  int64_t rrow = req_pool_idx[b];
  rrow = (rrow >= 0 && rrow < rtt_rows) ? rrow : 0;
  const int32_t* trow = rtt + rrow * rtt_stride;
  const int kend = P + tok_end;
  const int hq = hkv * grp;
  const int n_tiles = (kend + kBN - 1) / kBN;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int c = lane & 15;
  const int g4 = lane >> 4;

  // ---- DMA lane mapping (fixed for the kernel) ----------------------------
  // instruction ch = it*4 + wave covers row block rb = ch / KS, group pg = ch % KS
  int dma_row[LOADS];
  uint32_t dma_lds[LOADS];   // byte offset inside a tile (uniform per wave)
  uint32_t dma_gofs[LOADS];  // byte offset inside the gathered global row
#pragma unroll
  for (int it = 0; it < LOADS; ++it) {
    const int ch = it * 4 + wave;
    const int rb = ch / KS, pg = ch % KS;
    const int u = 16 * rb + (lane >> 2);
    const int qlog = (lane & 3) ^ ra_kv_swz(u);
    dma_row[it] = u;
    dma_lds[it] = pg * GROUP_B + rb * 1024;
    dma_gofs[it] = static_cast<uint32_t>(g * D * 2 + 16 * (4 * pg + qlog));
  }
  const uint32_t row_bytes = static_cast<uint32_t>(hkv) * D * 2;
  const unsigned char* kpool_b = reinterpret_cast<const unsigned char*>(k_pool);
  const unsigned char* knew_b = reinterpret_cast<const unsigned char*>(k_new);
  // V rows sit at the same offsets from their own bases
  const int64_t vpool_delta = reinterpret_cast<const unsigned char*>(v_pool) - kpool_b;
  const int64_t vnew_delta = reinterpret_cast<const unsigned char*>(v_new) - knew_b;
  const uint32_t smax = static_cast<uint32_t>(pool_slots - 1);
  // per-lane K source addresses of row 0 and per-wave LDS offsets, fixed for
  // the kernel (integer addresses: the new-token base is rebased by -P rows)
  uint64_t kpool_lane[LOADS], knew_lane[LOADS];
  uint32_t lds_k[2][LOADS], lds_v[2][LOADS];
#pragma unroll
  for (int it = 0; it < LOADS; ++it) {
    kpool_lane[it] = reinterpret_cast<uint64_t>(kpool_b) + dma_gofs[it];
    knew_lane[it] = reinterpret_cast<uint64_t>(knew_b) + static_cast<uint64_t>(start - P) * row_bytes + dma_gofs[it];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      lds_k[st][it] = __builtin_amdgcn_readfirstlane(ra_lds_addr(kv_lds[st][0]) + dma_lds[it]);
      lds_v[st][it] = __builtin_amdgcn_readfirstlane(ra_lds_addr(kv_lds[st][1]) + dma_lds[it]);
    }
  }

  const int u0 = dma_row[0];  // = dma_row[it] - it * ROW_STEP
  const int idx_pos = (lane % LOADS) * ROW_STEP + lane / LOADS;  // row whose slot lane's word holds
  auto issue_idx = [&](int tile) {  // wave 0 only: slot indices of one tile
    const int kb = tile * kBN;
    if (wave != 0 || tile >= n_tiles || kb >= P) return;
    const int pos = kb + idx_pos;
    ra_dma4(trow + (pos < P ? pos : 0), ra_lds_addr(&idx_lds[tile % RING][0]));
  };
  auto read_slots = [&](int tile, int32_t (&sl)[LOADS]) {
    const int32_t* w = &idx_lds[tile % RING][LOADS * u0];
    if constexpr (LOADS == 4) {
      const int4 v = *reinterpret_cast<const int4*>(w);
      sl[0] = v.x, sl[1] = v.y, sl[2] = v.z, sl[3] = v.w;
    } else {
      const int2 v = *reinterpret_cast<const int2*>(w);
      sl[0] = v.x, sl[1] = v.y;
    }
  };
  auto issue_kv = [&](int tile, int stage) {
    if (tile >= n_tiles) return;
    const int kb = tile * kBN;
    int32_t sl[LOADS];
    if (kb < P) read_slots(tile, sl);
    if (kb + kBN <= P) {
      // every row of the tile is a cached prefix row: gather through the slots
#pragma unroll
      for (int it = 0; it < LOADS; ++it) {
        const uint32_t slot = min(static_cast<uint32_t>(sl[it]), smax);  // negative -> clamped
        const uint64_t src = kpool_lane[it] + static_cast<uint64_t>(slot) * row_bytes;
        ra_dma16(reinterpret_cast<const void*>(src), lds_k[stage][it]);
        ra_dma16(reinterpret_cast<const void*>(src + vpool_delta), lds_v[stage][it]);
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
        ra_dma16(reinterpret_cast<const void*>(src), lds_k[stage][it]);
        ra_dma16(reinterpret_cast<const void*>(src + vdelta), lds_v[stage][it]);
      }
    }
  };

  // Q^T operands for the wave's two 16-query column blocks (loaded before
  // the first DMA so that the compiler's wait for these loads does not also
  // wait for the prologue's DMAs).
  bf16x8_t qT[2][KS];
  int qlim[2];  // last key position each of this lane's query columns may see
  bool qok[2];
  int64_t qrow[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int m = 32 * wave + 16 * j + c;
    const int it = tok0 + m / grp;
    qok[j] = it < tok_end;
    qlim[j] = P + min(it, tok_end - 1);
    qrow[j] = (start + min(it, tok_end - 1)) * hq + g * grp + m % grp;
    const __bf16* qp = q + qrow[j] * D + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qT[j][ks] = __builtin_bit_cast(bf16x8_t, qok[j] ? ra_ld16(qp + 32 * ks) : make_uint4(0, 0, 0, 0));
  }

  // ---- prologue: indices for tiles 0 and 1, K/V for tile 0 ----------------
  issue_idx(0);
  issue_idx(1);
  ra_wait_vmcnt<0>();
  __syncthreads();
  issue_kv(0, 0);

  // O^T accumulators; block DB holds the row sums (A operand = ones), so the
  // softmax denominator comes from the same bf16 P as the numerator.
  f32x4_t o[DB + 1][2];
#pragma unroll
  for (int i = 0; i <= DB; ++i) o[i][0] = o[i][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-INFINITY, -INFINITY};  // raw score units
  const uint4 ones_w = make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u);
  const bf16x8_t ones = __builtin_bit_cast(bf16x8_t, ones_w);

  // Per-lane LDS offsets.  S^T block bb of 32-key step k2 feeds A-operand row
  // c with key r = 32 k2 + 4 bb + r0, r0 = 8 (c >> 2) + (c & 3), so that the
  // accumulator's row group g4 holds keys 8 g4 .. 8 g4 + 7 of the step:
  // P^T's B-operand k slots in natural order.
  const int r0 = 8 * (c >> 2) + (c & 3);
  const uint32_t koff = r0 * 64 + 16 * (g4 ^ ra_kv_swz(r0));
  // V^T via transposed reads: lane supplies row 32 k2 + 4 h + (8 g4 + (c >> 2))
  // and logical piece 2 db + ((c & 3) >> 1), half (c & 1).
  const int vr = 8 * g4 + (c >> 2);
  uint32_t voff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) voff[e] = vr * 64 + 16 * ((2 * e + ((c & 3) >> 1)) ^ ra_kv_swz(vr)) + 8 * (c & 1);

  auto tile = [&](auto stage_tag, int t) {
    constexpr int ST = decltype(stage_tag)::value;
    const int kbase = t * kBN;
    ra_wait_vmcnt<0>();
    __syncthreads();
    issue_idx(t + 2);
    issue_kv(t + 1, ST ^ 1);

    const unsigned char* kst = kv_lds[ST][0];
    const unsigned char* vst = kv_lds[ST][1];

    f32x4_t sacc[2][2][2];  // [k2][bb][query block]
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb) {
        sacc[k2][bb][0] = sacc[k2][bb][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8_t a = __builtin_bit_cast(
              bf16x8_t, *reinterpret_cast<const uint4*>(kst + koff + ks * GROUP_B + (32 * k2 + 4 * bb) * 64));
          sacc[k2][bb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qT[0][ks], sacc[k2][bb][0], 0, 0, 0);
          sacc[k2][bb][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qT[1][ks], sacc[k2][bb][1], 0, 0, 0);
        }
      }
    // Element (k2, bb, i) is key kbase + 32 k2 + 8 g4 + 4 bb + i.  Online
    // softmax in the base-2 domain with a lazily moved maximum: it only moves
    // when some column's tile maximum exceeds it by more than 2^8 after
    // scaling, so most tiles skip the rescale; exponentials stay <= 2^8.
    const bool need_mask = kbase + kBN - 1 > P + tok0;
    bf16x8_t pT[2][2];  // [k2][query block]
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (need_mask) {
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
          for (int bb = 0; bb < 2; ++bb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (kbase + 32 * k2 + 8 * g4 + 4 * bb + i > qlim[j]) sacc[k2][bb][j][i] = -INFINITY;
      }
      float mt = -INFINITY;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
          mt = fmaxf(mt, fmaxf(fmaxf(sacc[k2][bb][j][0], sacc[k2][bb][j][1]),
                               fmaxf(sacc[k2][bb][j][2], sacc[k2][bb][j][3])));
      mt = ra_max_across_rows(mt);
      if (__builtin_amdgcn_ballot_w64((mt - m_run[j]) * scale_log2 > 8.f) != 0) {
        const float m_new = fmaxf(m_run[j], mt);
        const float alpha = ra_exp2((m_run[j] - m_new) * scale_log2);
#pragma unroll
        for (int db = 0; db <= DB; ++db) o[db][j] *= alpha;
        m_run[j] = m_new;
      }
      const float mb = -m_run[j] * scale_log2;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        float p[8];
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
          for (int i = 0; i < 4; ++i) p[4 * bb + i] = ra_exp2(__builtin_fmaf(sacc[k2][bb][j][i], scale_log2, mb));
        uint4 w;
        w.x = ra_pack_bf16x2(p[0], p[1]);
        w.y = ra_pack_bf16x2(p[2], p[3]);
        w.z = ra_pack_bf16x2(p[4], p[5]);
        w.w = ra_pack_bf16x2(p[6], p[7]);
        pT[k2][j] = __builtin_bit_cast(bf16x8_t, w);
      }
    }
    // O^T += V^T P^T and the row sums += 1 P^T.
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const unsigned char* vb = vst + voff[db & 1] + (db >> 1) * GROUP_B + 32 * k2 * 64;
        const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (__attribute__((address_space(3))) bf16x4_t*)(vb));
        const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (__attribute__((address_space(3))) bf16x4_t*)(vb + 4 * 64));
        const bf16x8_t a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        o[db][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pT[k2][0], o[db][0], 0, 0, 0);
        o[db][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pT[k2][1], o[db][1], 0, 0, 0);
      }
      o[DB][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pT[k2][0], o[DB][0], 0, 0, 0);
      o[DB][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pT[k2][1], o[DB][1], 0, 0, 0);
    }
  };

  for (int t = 0; t < n_tiles; t += 2) {
    tile(std::integral_constant<int, 0>{}, t);
    if (t + 1 < n_tiles) tile(std::integral_constant<int, 1>{}, t + 1);
  }

#pragma unroll
  for (int j = 0; j < 2; ++j) {
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

template <int D>
void launch(int64_t items, hipStream_t stream, const __bf16* qp, const __bf16* knp, const __bf16* vnp,
            int64_t total_tokens, const __bf16* kp, const __bf16* vp, int64_t pool_slots, const int32_t* rtt,
            int64_t rtt_rows, int64_t rtt_stride, const int32_t* rpi, const int32_t* pl, const int32_t* el,
            const int32_t* es, int32_t batch, int32_t hkv, int32_t grp, int32_t n_qtiles, float scale_log2,
            __bf16* op) {
  hipLaunchKernelGGL((extend_kernel<D>), dim3(static_cast<uint32_t>(items)), dim3(256), 0, stream, qp, knp, vnp,
                     total_tokens, kp, vp, pool_slots, rtt, rtt_rows, rtt_stride, rpi, pl, el, es, batch, hkv, grp,
                     n_qtiles, scale_log2, op);
}

}  // namespace

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
  const int32_t grp = hq / hkv;
  // Requests with at least 256 query rows per kv head (new tokens x query
  // heads per kv head) run on the 256-row kernel; shorter ones would leave
  // most of its tile empty.
  if (static_cast<int64_t>(max_extend_len) * grp >= kWideMinRows)
    return ra_extend_wide_launch(q, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows,
                                 rtt_stride, req_pool_idx, prefix_lens, extend_lens, extend_start, batch,
                                 max_extend_len, hq, hkv, d, scale, out, stream);
  const int32_t tpb = kBM / grp;
  const int64_t n_qtiles = (static_cast<int64_t>(max_extend_len) + tpb - 1) / tpb;
  const int64_t items = (static_cast<int64_t>(batch) * hkv * n_qtiles + 7) / 8 * 8;  // whole XCD rounds
  if (items > INT32_MAX) return ra_fail(RA_EINVAL, "ra_extend_attention: too many work items");
  const float scale_log2 = scale * RA_LOG2E;
  auto* qp = static_cast<const __bf16*>(q);
  auto* knp = static_cast<const __bf16*>(k_new);
  auto* vnp = static_cast<const __bf16*>(v_new);
  auto* kp = static_cast<const __bf16*>(k_pool);
  auto* vp = static_cast<const __bf16*>(v_pool);
  auto* op = static_cast<__bf16*>(out);
  const int32_t nq = static_cast<int32_t>(n_qtiles);
  if (d == 128) {
    launch<128>(items, stream, qp, knp, vnp, total_tokens, kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride,
                req_pool_idx, prefix_lens, extend_lens, extend_start, batch, hkv, grp, nq, scale_log2, op);
  } else {
    launch<64>(items, stream, qp, knp, vnp, total_tokens, kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride,
               req_pool_idx, prefix_lens, extend_lens, extend_start, batch, hkv, grp, nq, scale_log2, op);
  }
  return ra_check_launch("ra_extend_attention");
}
