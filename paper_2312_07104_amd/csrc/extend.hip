// Extend attention: prefill of a request's new tokens over its cached prefix
// (the work that remains once RadixAttention has reused the prefix's KV
// cache; section 3, Appendix A.1), plus causal attention among the new
// tokens.  This is a dense contraction, so QK^T and PV run on bf16 MFMA with
// fp32 accumulation.
//
// Work item = (request, kv head, query tile).  A tile holds 128 query rows,
// packed as (new token, query head of the kv head's group): the G heads that
// share a kv head share every K/V tile the work-group stages.  Four waves,
// 32 rows each; per 64-key tile:
//   * all 256 threads gather the next tile's K and V rows into registers
//     (prefix keys through the request's slot-table row, new keys from the
//     contiguous k_new / v_new rows) while the current tile is computed;
//   * K goes to LDS row-major, V transposed (so PV's k dimension is
//     contiguous per lane);
//   * S^T[key, query] = K Q^T with the queries as MFMA columns, so each
//     lane ends up owning one query column and the row max / row sum are
//     in-lane plus two cross-row shuffles;
//   * P^T stays in registers as the B operand of O^T += V^T P^T.
// Masking only runs on tiles that reach past the first query's last key.
#include "device_common.h"

namespace {

constexpr int kBM = 128;  // query rows per work-group
constexpr int kBN = 64;   // keys per tile

__device__ __forceinline__ uint4 ld16(const __bf16* p) { return *reinterpret_cast<const uint4*>(p); }

// Column of key u (0..63) in the transposed V tile.  Inside each 32-key MFMA
// step, the P^T operand of lane group g4 holds keys 4g4..4g4+3 then
// 16+4g4..16+4g4+3 (the S^T accumulator layout), so V^T stores them in
// that order.
__device__ __forceinline__ int vt_col(int u) {
  const int w = u & 31;
  return (u & 32) + 8 * ((w & 15) >> 2) + (w & 3) + ((w & 16) ? 4 : 0);
}

template <int D>
__global__ __launch_bounds__(256, 2) void extend_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k_new, const __bf16* __restrict__ v_new,
    int64_t total_tokens, const __bf16* __restrict__ k_pool, const __bf16* __restrict__ v_pool,
    int64_t pool_slots, const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride,
    const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ prefix_lens,
    const int32_t* __restrict__ extend_lens, const int32_t* __restrict__ extend_start, int32_t batch,
    int32_t hkv, int32_t grp, int32_t n_qtiles, float scale_log2, __bf16* __restrict__ out) {
  constexpr int KS = D / 32;              // MFMA k-steps over the head dimension
  constexpr int DB = D / 16;              // 16-row blocks of O^T
  constexpr int KP = D + 8;               // K tile pitch (bf16)
  constexpr int VP = kBN + 8;             // V^T tile pitch (bf16)
  constexpr int PIECES = D / 8;           // 16-byte pieces per row
  constexpr int LOADS = kBN * PIECES / 256;
  __shared__ __align__(16) unsigned short k_lds[kBN * KP];
  __shared__ __align__(16) unsigned short vt_lds[D * VP];

  const int item = blockIdx.x;
  const int b = item % batch;
  const int rest = item / batch;
  const int g = rest % hkv;
  const int qt = n_qtiles - 1 - rest / hkv;  // longest tiles first
  const int tpb = kBM / grp;                 // new tokens per tile

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

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int c = lane & 15;
  const int g4 = lane >> 4;

  // Q^T operands for the wave's two 16-query column blocks.
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
      qT[j][ks] = __builtin_bit_cast(bf16x8_t, qok[j] ? ld16(qp + 32 * ks) : make_uint4(0, 0, 0, 0));
  }

  f32x4_t o[DB][2];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i][0] = o[i][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};

  // Tile gather into registers.
  uint4 kreg[LOADS], vreg[LOADS];
  auto load_tile = [&](int kbase) {
#pragma unroll
    for (int it = 0; it < LOADS; ++it) {
      const int p = tid + 256 * it;
      const int u = p / PIECES, pc = p % PIECES;
      const int pos = kbase + u;
      if (pos < kend) {
        int64_t roff;
        if (pos < P) {
          int64_t s = trow[pos];
          s = (s >= 0 && s < pool_slots) ? s : 0;
          roff = (s * hkv + g) * D + 8 * pc;
          kreg[it] = ld16(k_pool + roff);
          vreg[it] = ld16(v_pool + roff);
        } else {
          roff = ((start + pos - P) * hkv + g) * D + 8 * pc;
          kreg[it] = ld16(k_new + roff);
          vreg[it] = ld16(v_new + roff);
        }
      } else {
        kreg[it] = make_uint4(0, 0, 0, 0);
        vreg[it] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int it = 0; it < LOADS; ++it) {
      const int p = tid + 256 * it;
      const int u = p / PIECES, pc = p % PIECES;
      *reinterpret_cast<uint4*>(&k_lds[u * KP + 8 * pc]) = kreg[it];
      const int col = vt_col(u);
      const uint32_t w[4] = {vreg[it].x, vreg[it].y, vreg[it].z, vreg[it].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vt_lds[(8 * pc + 2 * e) * VP + col] = static_cast<unsigned short>(w[e] & 0xFFFFu);
        vt_lds[(8 * pc + 2 * e + 1) * VP + col] = static_cast<unsigned short>(w[e] >> 16);
      }
    }
  };

  const int n_tiles = (kend + kBN - 1) / kBN;
  load_tile(0);
  for (int t = 0; t < n_tiles; ++t) {
    const int kbase = t * kBN;
    __syncthreads();
    store_tile();
    __syncthreads();
    if (t + 1 < n_tiles) load_tile(kbase + kBN);

    // S^T blocks: 4 key blocks x 2 query blocks.
    f32x4_t sacc[4][2];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      sacc[tb][0] = sacc[tb][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8_t a =
            __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(&k_lds[(16 * tb + c) * KP + 32 * ks + 8 * g4]));
        sacc[tb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qT[0][ks], sacc[tb][0], 0, 0, 0);
        sacc[tb][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qT[1][ks], sacc[tb][1], 0, 0, 0);
      }
    }
    const bool need_mask = kbase + kBN - 1 > P + tok0;
    bf16x8_t pT[2][2];  // [k-step][query block]
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float s[16];
      float mt = -INFINITY;
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = sacc[tb][j][i] * scale_log2;
          if (need_mask && kbase + 16 * tb + 4 * g4 + i > qlim[j]) v = -INFINITY;
          s[4 * tb + i] = v;
          mt = fmaxf(mt, v);
        }
      }
      mt = ra_max_across_rows(mt);
      const float m_new = fmaxf(m_run[j], mt);
      const float alpha = ra_exp2(m_run[j] - m_new);
      float psum = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        s[i] = ra_exp2(s[i] - m_new);
        psum += s[i];
      }
      l_run[j] = l_run[j] * alpha + psum;
      m_run[j] = m_new;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][j] *= alpha;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        uint4 w;
        w.x = ra_pack_bf16x2(s[8 * k2 + 0], s[8 * k2 + 1]);
        w.y = ra_pack_bf16x2(s[8 * k2 + 2], s[8 * k2 + 3]);
        w.z = ra_pack_bf16x2(s[8 * k2 + 4], s[8 * k2 + 5]);
        w.w = ra_pack_bf16x2(s[8 * k2 + 6], s[8 * k2 + 7]);
        pT[k2][j] = __builtin_bit_cast(bf16x8_t, w);
      }
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const bf16x8_t a = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const uint4*>(&vt_lds[(16 * db + c) * VP + 32 * k2 + 8 * g4]));
        o[db][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pT[k2][0], o[db][0], 0, 0, 0);
        o[db][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pT[k2][1], o[db][1], 0, 0, 0);
      }
    }
  }

#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float l_tot = ra_sum_across_rows(l_run[j]);
    if (!qok[j]) continue;
    const float inv = 1.f / l_tot;
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

}  // namespace

extern "C" int ra_extend_attention(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                                   const void* k_pool, const void* v_pool, int64_t pool_slots,
                                   const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                   const int32_t* req_pool_idx, const int32_t* prefix_lens,
                                   const int32_t* extend_lens, const int32_t* extend_start, int32_t batch,
                                   int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                                   void* out, hipStream_t stream) {
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0 || (d != 64 && d != 128) || pool_slots <= 0 ||
      rtt_rows <= 0 || rtt_stride <= 0 || max_extend_len < 0 || total_tokens < 0)
    return ra_fail(RA_EINVAL, "ra_extend_attention: bad sizes");
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
  const int32_t tpb = kBM / grp;
  const int64_t n_qtiles = (static_cast<int64_t>(max_extend_len) + tpb - 1) / tpb;
  const int64_t items = static_cast<int64_t>(batch) * hkv * n_qtiles;
  if (items > INT32_MAX) return ra_fail(RA_EINVAL, "ra_extend_attention: too many work items");
  const float scale_log2 = scale * RA_LOG2E;
  auto* qp = static_cast<const __bf16*>(q);
  auto* knp = static_cast<const __bf16*>(k_new);
  auto* vnp = static_cast<const __bf16*>(v_new);
  auto* kp = static_cast<const __bf16*>(k_pool);
  auto* vp = static_cast<const __bf16*>(v_pool);
  auto* op = static_cast<__bf16*>(out);
  if (d == 128) {
    hipLaunchKernelGGL(extend_kernel<128>, dim3(static_cast<uint32_t>(items)), dim3(256), 0, stream, qp, knp, vnp,
                       total_tokens, kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx,
                       prefix_lens, extend_lens, extend_start, batch, hkv, grp, static_cast<int32_t>(n_qtiles),
                       scale_log2, op);
  } else {
    hipLaunchKernelGGL(extend_kernel<64>, dim3(static_cast<uint32_t>(items)), dim3(256), 0, stream, qp, knp, vnp,
                       total_tokens, kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx,
                       prefix_lens, extend_lens, extend_start, batch, hkv, grp, static_cast<int32_t>(n_qtiles),
                       scale_log2, op);
  }
  return ra_check_launch("ra_extend_attention");
}
