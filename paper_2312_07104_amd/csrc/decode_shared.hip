// Decode attention that reads every shared run of the batch's radix tree once
// (ra_decode_attention_shared).  RadixAttention stores one copy of a prefix
// that several requests share (section 3), so their decode steps ask for the
// same K/V rows; the host plan (ra_decode_share_plan) cuts the batch into
// items, each a run of positions of one slot-table row and the requests
// (members) that hold exactly those slots there.  The result is the same
// attention as ra_decode_attention (each query over positions 0 .. L-1),
// accumulated in a different order.
//
// Work item = (plan item, kv head); one wave per item.  The item's members'
// query heads of the kv head are the columns of CB 16-column MFMA blocks
// (column 16 cb + c = member (16 cb + c) / G, head (16 cb + c) % G), so one
// pass over the run's K/V rows serves G x members queries.  Per 32-token
// tile the rows are read with ordinary vector loads into registers (tiles in
// flight as in decode_partial_vr_kernel): K straight into the MFMA
// A-operand layout, V into one LDS tile for the transposing V^T reads.  Each
// column keeps its own online softmax (base 2, lazily moved maximum).  A
// member whose whole context is this item writes its output; otherwise the
// item writes the member's normalised partial output and log2-sum-exp, and
// decode_shared_combine_kernel merges a request's partials.
#include "device_common.h"
#include "lds_dma.h"

namespace {

constexpr int kShTile = 32;
constexpr int kPlanHeader = 16;
constexpr int kItemWords = 8;

template <int D, int CB>
__global__ __launch_bounds__(64) void decode_shared_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k_pool, const __bf16* __restrict__ v_pool,
    int64_t pool_slots, const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride,
    const int32_t* __restrict__ plan, int32_t n_items, int32_t n_mem, int32_t n_parts, int32_t batch, int32_t hkv,
    int32_t grp, float scale_log2, float* __restrict__ ws_o, float* __restrict__ ws_lse, __bf16* __restrict__ out) {
  constexpr int TILE = kShTile;
  constexpr int KS = D / 32;             // MFMA k-steps over the head dimension (64-byte piece groups)
  constexpr int DB = D / 16;             // 16-row blocks of O^T
  constexpr int NB = TILE / 16;          // S^T blocks per tile
  constexpr int GROUP_B = TILE * 64;     // bytes of one piece group of the V tile
  constexpr int TILE_B = KS * GROUP_B;   // bytes of the V tile
  // tiles in flight: two, or one with four column blocks (whose registers
  // would not hold a second tile; its MFMA work per tile is four times as
  // long, which covers more of the loads' latency)
  constexpr int NP = CB == 4 ? 1 : 2;
  __shared__ __align__(16) unsigned char v_lds[TILE_B];

  const int64_t blk = blockIdx.x;
  const int64_t item = blk / hkv;
  if (item >= n_items) return;
  const int g = static_cast<int>(blk % hkv);
  const int32_t* it = plan + kPlanHeader + kItemWords * item;
  int64_t rrow = it[0];
  rrow = (rrow >= 0 && rrow < rtt_rows) ? rrow : 0;
  const int t_begin = static_cast<int>(min<int64_t>(max(it[1], 0), rtt_stride));
  const int t_end = static_cast<int>(min<int64_t>(max(it[2], t_begin), rtt_stride));
  const int mem_off = min(max(it[3], 0), n_mem);
  const int n_m = min(min(it[4], n_mem - mem_off), (16 * CB) / grp);
  if (t_end <= t_begin || n_m <= 0) return;
  const int32_t* mem = plan + kPlanHeader + static_cast<int64_t>(kItemWords) * n_items + 2 * mem_off;
  const int32_t* trow = rtt + rrow * rtt_stride;
  const int hq = hkv * grp;
  const int n_tiles = (t_end - t_begin + TILE - 1) / TILE;

  const int lane = threadIdx.x;
  const int c = lane & 15;
  const int g4 = lane >> 4;

  // This lane's column in each block: member, head, destination.
  int mb[CB], mpart[CB];
  bool mok[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int col = 16 * cb + c;
    const int m = col / grp;
    mok[cb] = m < n_m;
    mb[cb] = mok[cb] ? min(max(mem[2 * m], 0), batch - 1) : 0;
    mpart[cb] = mok[cb] ? mem[2 * m + 1] : -1;
  }
  bf16x8_t qt[CB][KS];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int col = 16 * cb + c;
    const __bf16* qp = q + (static_cast<int64_t>(mb[cb]) * hq + g * grp + col % grp) * D + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qt[cb][ks] = __builtin_bit_cast(bf16x8_t, mok[cb] ? ra_ld16(qp + 32 * ks) : make_uint4(0, 0, 0, 0));
  }

  // Rows this lane loads (the layout of decode_partial_vr_kernel): K row
  // 8 (c >> 2) + 4 bb + (c & 3) of the tile, its 16 bytes of each k-step;
  // V copy row 16 rb + (lane >> 2), piece (lane & 3) ^ swizzle of each
  // 64-byte piece group, stored at pg * GROUP_B + rb * 1024 + 16 lane.
  int kr[NB];
#pragma unroll
  for (int bb = 0; bb < NB; ++bb) kr[bb] = 8 * (c >> 2) + 4 * bb + (c & 3);
  int vu[2];
  uint32_t vpc[2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    vu[rb] = 16 * rb + (lane >> 2);
    vpc[rb] = 16u * static_cast<uint32_t>((lane & 3) ^ ra_kv_swz(vu[rb]));
  }
  const uint32_t row_bytes = static_cast<uint32_t>(hkv) * D * 2;
  const unsigned char* kbase = reinterpret_cast<const unsigned char*>(k_pool) + g * D * 2 + 16 * g4;
  const unsigned char* vbase = reinterpret_cast<const unsigned char*>(v_pool) + g * D * 2;
  const uint32_t smax = static_cast<uint32_t>(pool_slots - 1);

  auto load_idx = [&](int tile) -> int32_t {
    const int pos = min(t_begin + tile * TILE + (lane & (TILE - 1)), t_end - 1);  // padding repeats a real token
    return trow[pos];
  };
  uint4 kbuf[NP][NB][KS];
  uint4 vbuf[NP][2][KS];
  int32_t ibuf[NP];
  auto load_tile = [&](int j, int32_t idx) {
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
      const uint32_t slot = min(static_cast<uint32_t>(__shfl(idx, kr[bb])), smax);  // negative -> clamped
      const unsigned char* p = kbase + static_cast<uint64_t>(slot) * row_bytes;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kbuf[j][bb][ks] = ra_ld16(p + 64 * ks);
    }
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const uint32_t slot = min(static_cast<uint32_t>(__shfl(idx, vu[rb])), smax);
      const unsigned char* p = vbase + static_cast<uint64_t>(slot) * row_bytes + vpc[rb];
#pragma unroll
      for (int pg = 0; pg < KS; ++pg) vbuf[j][rb][pg] = ra_ld16(p + 64 * pg);
    }
  };

#pragma unroll
  for (int j = 0; j < NP; ++j) ibuf[j] = load_idx(j);
#pragma unroll
  for (int j = 0; j < NP; ++j)
    if (j < n_tiles) load_tile(j, ibuf[j]);
#pragma unroll
  for (int j = 0; j < NP; ++j) ibuf[j] = load_idx(j + NP);

  f32x4_t o[DB][CB];
  float m_run[CB], l_run[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
    for (int i = 0; i < DB; ++i) o[i][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m_run[cb] = -INFINITY;
    l_run[cb] = 0.f;
  }
  const int vr0 = 8 * g4 + (c >> 2);
  uint32_t voff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) voff[e] = vr0 * 64 + 16 * ((2 * e + ((c & 3) >> 1)) ^ ra_kv_swz(vr0)) + 8 * (c & 1);

  for (int tb = 0; tb < n_tiles; tb += NP) {
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int t = tb + j;
      if (t < n_tiles) {
        // V(t) into the LDS tile (the previous tile's transposed reads were
        // consumed by its PV MFMAs, so the tile is free).
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int pg = 0; pg < KS; ++pg)
            *reinterpret_cast<uint4*>(v_lds + pg * GROUP_B + rb * 1024 + 16 * lane) = vbuf[j][rb][pg];
        const int t0 = t_begin + t * TILE;
        f32x4_t sacc[CB][NB];
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) {
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) sacc[cb][bb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const bf16x8_t a = __builtin_bit_cast(bf16x8_t, kbuf[j][bb][ks]);
#pragma unroll
            for (int cb = 0; cb < CB; ++cb)
              sacc[cb][bb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qt[cb][ks], sacc[cb][bb], 0, 0, 0);
          }
        }
        // Slot j is consumed: refill it with tile t + NP, and its index
        // register with the indices of tile t + 2 NP.
        if (t + NP < n_tiles) load_tile(j, ibuf[j]);
        ibuf[j] = load_idx(t + 2 * NP);

        // element (bb, i) of a block is token t0 + 8 g4 + 4 bb + i
        if (t0 + TILE > t_end) {
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
#pragma unroll
            for (int bb = 0; bb < NB; ++bb)
#pragma unroll
              for (int i = 0; i < 4; ++i)
                if (t0 + 8 * g4 + 4 * bb + i >= t_end) sacc[cb][bb][i] = -INFINITY;
        }
        bf16x8_t pt[CB];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          float mt = fmaxf(fmaxf(fmaxf(sacc[cb][0][0], sacc[cb][0][1]), fmaxf(sacc[cb][0][2], sacc[cb][0][3])),
                           fmaxf(fmaxf(sacc[cb][1][0], sacc[cb][1][1]), fmaxf(sacc[cb][1][2], sacc[cb][1][3])));
          mt = ra_max_across_rows(mt);
          if (__builtin_amdgcn_ballot_w64((mt - m_run[cb]) * scale_log2 > 8.f) != 0) {
            const float m_new = fmaxf(m_run[cb], mt);
            const float alpha = ra_exp2((m_run[cb] - m_new) * scale_log2);
            l_run[cb] *= alpha;
#pragma unroll
            for (int i = 0; i < DB; ++i) o[i][cb] *= alpha;
            m_run[cb] = m_new;
          }
          const float mbias = -m_run[cb] * scale_log2;
          float p[8];
#pragma unroll
          for (int bb = 0; bb < NB; ++bb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              p[4 * bb + i] = ra_exp2(__builtin_fmaf(sacc[cb][bb][i], scale_log2, mbias));
              l_run[cb] += p[4 * bb + i];
            }
          uint4 pw;
          pw.x = ra_pack_bf16x2(p[0], p[1]);
          pw.y = ra_pack_bf16x2(p[2], p[3]);
          pw.z = ra_pack_bf16x2(p[4], p[5]);
          pw.w = ra_pack_bf16x2(p[6], p[7]);
          pt[cb] = __builtin_bit_cast(bf16x8_t, pw);
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const unsigned char* vb = v_lds + voff[db & 1] + (db >> 1) * GROUP_B;
          const bf16x4_t lo =
              __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4_t*)(vb));
          const bf16x4_t hi =
              __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4_t*)(vb + 4 * 64));
          const bf16x8_t a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) o[db][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pt[cb], o[db][cb], 0, 0, 0);
        }
      }
    }
  }

#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const float l_tot = ra_sum_across_rows(l_run[cb]);
    if (!mok[cb]) continue;
    const int head = g * grp + (16 * cb + c) % grp;
    const float inv = 1.f / l_tot;
    if (mpart[cb] < 0) {
      __bf16* op = out + (static_cast<int64_t>(mb[cb]) * hq + head) * D + 4 * g4;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        uint2 w;
        w.x = ra_pack_bf16x2(o[db][cb][0] * inv, o[db][cb][1] * inv);
        w.y = ra_pack_bf16x2(o[db][cb][2] * inv, o[db][cb][3] * inv);
        *reinterpret_cast<uint2*>(op + 16 * db) = w;
      }
    } else if (mpart[cb] < n_parts) {
      const int64_t pidx = static_cast<int64_t>(mpart[cb]) * hq + head;
      float* wp = ws_o + pidx * D + 4 * g4;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<float4*>(wp + 16 * db) =
            make_float4(o[db][cb][0] * inv, o[db][cb][1] * inv, o[db][cb][2] * inv, o[db][cb][3] * inv);
      if (g4 == 0) ws_lse[pidx] = m_run[cb] * scale_log2 + __log2f(l_tot);
    }
  }
}

// Merges request b's partials part_off[b] .. part_off[b+1]-1 for one head:
// weights 2^(lse_i - max lse).  Requests with one part wrote their output.
template <int D>
__global__ __launch_bounds__(64) void decode_shared_combine_kernel(const float* __restrict__ ws_o,
                                                                   const float* __restrict__ ws_lse,
                                                                   const int32_t* __restrict__ part_off,
                                                                   int32_t n_parts, int32_t hq,
                                                                   __bf16* __restrict__ out) {
  const int64_t bh = blockIdx.x;
  const int64_t b = bh / hq;
  const int head = static_cast<int>(bh % hq);
  const int p0 = min(max(part_off[b], 0), n_parts);
  const int p1 = min(max(part_off[b + 1], p0), n_parts);
  if (p1 - p0 < 1) return;
  float mx = -INFINITY;
  for (int p = p0; p < p1; ++p) mx = fmaxf(mx, ws_lse[static_cast<int64_t>(p) * hq + head]);
  constexpr int PER = D / 64;
  float acc[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) acc[j] = 0.f;
  float wsum = 0.f;
  for (int p = p0; p < p1; ++p) {
    const int64_t pidx = static_cast<int64_t>(p) * hq + head;
    const float w = ra_exp2(ws_lse[pidx] - mx);
    wsum += w;
    const float* op = ws_o + pidx * D + threadIdx.x * PER;
#pragma unroll
    for (int j = 0; j < PER; ++j) acc[j] += w * op[j];
  }
  const float inv = 1.f / wsum;
  __bf16* dst = out + bh * D + threadIdx.x * PER;
  if constexpr (PER == 2) {
    *reinterpret_cast<uint32_t*>(dst) = ra_pack_bf16x2(acc[0] * inv, acc[1] * inv);
  } else {
    const uint32_t w = ra_pack_bf16x2(acc[0] * inv, 0.f);
    *reinterpret_cast<unsigned short*>(dst) = static_cast<unsigned short>(w & 0xFFFFu);
  }
}

template <int D, int CB>
void launch_shared(int64_t grid, hipStream_t stream, const __bf16* q, const __bf16* kp, const __bf16* vp,
                   int64_t pool_slots, const int32_t* rtt, int64_t rtt_rows, int64_t rtt_stride, const int32_t* plan,
                   int32_t n_items, int32_t n_mem, int32_t n_parts, int32_t batch, int32_t hkv, int32_t grp,
                   float scale_log2, float* ws_o, float* ws_lse, __bf16* out) {
  hipLaunchKernelGGL((decode_shared_kernel<D, CB>), dim3(static_cast<uint32_t>(grid)), dim3(64), 0, stream, q, kp,
                     vp, pool_slots, rtt, rtt_rows, rtt_stride, plan, n_items, n_mem, n_parts, batch, hkv, grp,
                     scale_log2, ws_o, ws_lse, out);
}

}  // namespace

extern "C" size_t ra_decode_shared_workspace_bytes(int32_t n_parts, int32_t hq, int32_t d) {
  if (n_parts <= 0 || hq <= 0 || d <= 0) return 0;
  return static_cast<size_t>(n_parts) * hq * (d + 1) * sizeof(float);
}

// Argument checks shared with ra_mixed_attention_shared: RA_OK when the call
// may launch (or has nothing to do), an error status otherwise.
int ra_decode_shared_validate(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                              const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int32_t batch,
                              int32_t hq, int32_t hkv, int32_t d, float scale, const int32_t* plan, int64_t plan_len,
                              int32_t n_items, int32_t n_member_entries, int32_t n_parts, int32_t members_per_item,
                              const void* workspace, size_t workspace_bytes, const void* out) {
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0 || (d != 64 && d != 128) || pool_slots <= 0 ||
      rtt_stride <= 0 || rtt_rows <= 0 || !(scale > 0.f) || n_items < 0 || n_member_entries < 0 || n_parts < 0)
    return ra_fail(RA_EINVAL, "ra_decode_attention_shared: bad sizes or scale");
  const int32_t grp = hq / hkv;
  if (grp > 16) return ra_fail(RA_EINVAL, "ra_decode_attention_shared: more than 16 query heads per kv head");
  if (members_per_item < 1 || members_per_item * grp > 64)
    return ra_fail(RA_EINVAL, "ra_decode_attention_shared: members_per_item x (Hq / Hkv) must be 1 .. 64");
  if (plan_len != kPlanHeader + static_cast<int64_t>(kItemWords) * n_items + 2 * static_cast<int64_t>(n_member_entries) +
                      batch + 1)
    return ra_fail(RA_EINVAL, "ra_decode_attention_shared: plan length does not match its counts");
  if (batch == 0 || n_items == 0) return ra_ok();
  if (!q || !k_pool || !v_pool || !req_to_token || !plan || !out)
    return ra_fail(RA_EINVAL, "ra_decode_attention_shared: NULL pointer");
  if (!ra_aligned16(q) || !ra_aligned16(k_pool) || !ra_aligned16(v_pool) || !ra_aligned16(out))
    return ra_fail(RA_EINVAL, "ra_decode_attention_shared: pointers must be 16-byte aligned");
  const size_t need = ra_decode_shared_workspace_bytes(n_parts, hq, d);
  if (workspace_bytes < need || (need && !workspace))
    return ra_fail(RA_EINVAL, "ra_decode_attention_shared: workspace too small");
  if (need && !ra_aligned16(workspace)) return ra_fail(RA_EINVAL, "ra_decode_attention_shared: workspace alignment");
  if (static_cast<int64_t>(n_items) * hkv > INT32_MAX || static_cast<int64_t>(batch) * hq > INT32_MAX)
    return ra_fail(RA_EINVAL, "ra_decode_attention_shared: too many work items");
  return ra_ok();
}

extern "C" int ra_decode_attention_shared(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                                          const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                          int32_t batch, int32_t hq, int32_t hkv, int32_t d, float scale,
                                          const int32_t* plan, int64_t plan_len, int32_t n_items,
                                          int32_t n_member_entries, int32_t n_parts, int32_t members_per_item,
                                          void* workspace, size_t workspace_bytes, void* out, hipStream_t stream) {
  const int st0 = ra_decode_shared_validate(q, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride, batch,
                                            hq, hkv, d, scale, plan, plan_len, n_items, n_member_entries, n_parts,
                                            members_per_item, workspace, workspace_bytes, out);
  if (st0 != RA_OK || batch == 0 || n_items == 0) return st0;
  const int32_t grp = hq / hkv;
  const size_t need = ra_decode_shared_workspace_bytes(n_parts, hq, d);
  const int64_t grid = static_cast<int64_t>(n_items) * hkv;
  float* ws_o = static_cast<float*>(workspace);
  float* ws_lse = need ? ws_o + static_cast<int64_t>(n_parts) * hq * d : nullptr;
  const float scale_log2 = scale * RA_LOG2E;
  auto* qp = static_cast<const __bf16*>(q);
  auto* kp = static_cast<const __bf16*>(k_pool);
  auto* vp = static_cast<const __bf16*>(v_pool);
  auto* op = static_cast<__bf16*>(out);
  // 16-column MFMA blocks the members' heads need
  const int32_t cols = members_per_item * grp;
  const int32_t cb = cols <= 16 ? 1 : cols <= 32 ? 2 : 4;
#define RA_SHARED(DD, CC)                                                                                        \
  launch_shared<DD, CC>(grid, stream, qp, kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride, plan, n_items, \
                        n_member_entries, n_parts, batch, hkv, grp, scale_log2, ws_o, ws_lse, op)
  if (d == 128) {
    if (cb == 1) RA_SHARED(128, 1);
    else if (cb == 2) RA_SHARED(128, 2);
    else RA_SHARED(128, 4);
  } else {
    if (cb == 1) RA_SHARED(64, 1);
    else if (cb == 2) RA_SHARED(64, 2);
    else RA_SHARED(64, 4);
  }
#undef RA_SHARED
  int st = ra_check_launch("ra_decode_attention_shared(partial)");
  if (st != RA_OK || n_parts == 0) return st;
  const int32_t* part_off = plan + kPlanHeader + static_cast<int64_t>(kItemWords) * n_items + 2 * static_cast<int64_t>(n_member_entries);
  const int64_t bh = static_cast<int64_t>(batch) * hq;
  if (d == 128)
    hipLaunchKernelGGL(decode_shared_combine_kernel<128>, dim3(static_cast<uint32_t>(bh)), dim3(64), 0, stream, ws_o,
                       ws_lse, part_off, n_parts, hq, op);
  else
    hipLaunchKernelGGL(decode_shared_combine_kernel<64>, dim3(static_cast<uint32_t>(bh)), dim3(64), 0, stream, ws_o,
                       ws_lse, part_off, n_parts, hq, op);
  return ra_check_launch("ra_decode_attention_shared(combine)");
}
