// Decode attention over the token-granular KV pool: one query token per
// request over its whole context (prefix plus private suffix), read through
// the request's row of the slot table.  Decode dominates when outputs are
// long (evaluation, section 6.2); it is bound by HBM bandwidth.
//
// Work item = (request, kv head, KV chunk); one wave per item.  The G query
// heads that share a kv head are the N = 16 columns of bf16 MFMAs, so every
// K/V row fetched from HBM serves all G heads and the VALU is left for the
// softmax:
//   S^T[token, head] = K[token, :] . Q[head, :]   (A = gathered K rows, loaded
//                                                  straight into registers)
//   O^T[d, head]    += V^T[d, token] P^T[token, head]
// V^T is staged through LDS (each lane writes its gathered 16-byte V piece
// transposed).  Online softmax in the base-2 domain: the running maximum is
// reduced across the four 16-lane rows with lane shuffles; the running sum
// stays per lane and is reduced once at the end.  A chunk writes a normalised
// partial output and its log-sum-exp; a second kernel merges the chunks.
#include "device_common.h"

namespace {

constexpr int kTile = 32;          // tokens per MFMA step (two 16-row blocks)
constexpr int kVtPitch = 40;       // LDS row pitch of V^T in bf16 (32 + 8 pad)

__device__ __forceinline__ uint4 ld16(const __bf16* p) { return *reinterpret_cast<const uint4*>(p); }

template <int D>
__global__ __launch_bounds__(64) void decode_partial_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k_pool, const __bf16* __restrict__ v_pool,
    int64_t pool_slots, const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride,
    const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ seq_lens, int32_t batch,
    int32_t hkv, int32_t grp, int32_t chunk_len, int32_t max_splits, int32_t max_len, float scale_log2,
    float* __restrict__ ws_o, float* __restrict__ ws_lse, __bf16* __restrict__ out) {
  constexpr int KS = D / 32;  // MFMA k-steps over the head dimension
  constexpr int DB = D / 16;  // 16-row blocks of O^T
  __shared__ unsigned short vt[D * kVtPitch];

  const int item = blockIdx.x;
  const int b = item % batch;
  const int rest = item / batch;
  const int g = rest % hkv;
  const int split = rest / hkv;
  const int L = min(seq_lens[b], max_len);  // host bound (<= rtt_stride, <= chunk_len * max_splits)
  if (L <= 0) return;
  const int n_splits = (L + chunk_len - 1) / chunk_len;
  if (split >= n_splits) return;
  const int t_begin = split * chunk_len;
  const int t_end = min(L, t_begin + chunk_len);
  int64_t rrow = req_pool_idx[b];
  rrow = (rrow >= 0 && rrow < rtt_rows) ? rrow : 0;
  const int64_t row = rrow * rtt_stride;
  const int hq = hkv * grp;

  const int lane = threadIdx.x;
  const int c = lane & 15;   // query head column / token row of the A operand
  const int g4 = lane >> 4;  // which 8-wide k slice this lane holds

  // Q^T as the B operand: column c = head g*grp + c, k = 8*g4 .. of each step.
  bf16x8_t qt[KS];
  {
    const bool has = c < grp;
    const __bf16* qp = q + (static_cast<int64_t>(b) * hq + g * grp + (has ? c : 0)) * D + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 w = has ? ld16(qp + 32 * ks) : make_uint4(0, 0, 0, 0);
      qt[ks] = __builtin_bit_cast(bf16x8_t, w);
    }
  }

  f32x4_t o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;
  float l_run = 0.f;

  const int64_t head_off = static_cast<int64_t>(g) * D + 8 * g4;
  const int64_t row_elems = static_cast<int64_t>(hkv) * D;
  // transposed-write column of this lane's two tokens (see P^T k-slot order)
  const int col_a = 8 * (c >> 2) + (c & 3);
  const int col_b = col_a + 4;

  for (int t0 = t_begin; t0 < t_end; t0 += kTile) {
    const int ta = t0 + c, tb = t0 + 16 + c;
    const bool va = ta < t_end, vb = tb < t_end;
    int64_t sa = va ? rtt[row + ta] : 0;
    int64_t sb = vb ? rtt[row + tb] : 0;
    sa = (sa >= 0 && sa < pool_slots) ? sa : 0;
    sb = (sb >= 0 && sb < pool_slots) ? sb : 0;
    const __bf16* kpa = k_pool + sa * row_elems + head_off;
    const __bf16* kpb = k_pool + sb * row_elems + head_off;
    const __bf16* vpa = v_pool + sa * row_elems + head_off;
    const __bf16* vpb = v_pool + sb * row_elems + head_off;
    uint4 ka[KS], kb[KS], wa[KS], wb[KS];
    const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      ka[ks] = va ? ld16(kpa + 32 * ks) : z;
      kb[ks] = vb ? ld16(kpb + 32 * ks) : z;
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      wa[ks] = va ? ld16(vpa + 32 * ks) : z;
      wb[ks] = vb ? ld16(vpb + 32 * ks) : z;
    }

    // S^T for tokens t0 + 4*g4 + i (sA) and t0 + 16 + 4*g4 + i (sB), head c.
    f32x4_t sA = {0.f, 0.f, 0.f, 0.f}, sB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sA = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka[ks]), qt[ks], sA, 0, 0, 0);
      sB = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kb[ks]), qt[ks], sB, 0, 0, 0);
    }
    float s[8];
    float mt = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tA = t0 + 4 * g4 + i, tB = t0 + 16 + 4 * g4 + i;
      s[i] = tA < t_end ? sA[i] * scale_log2 : -INFINITY;
      s[4 + i] = tB < t_end ? sB[i] * scale_log2 : -INFINITY;
      mt = fmaxf(mt, fmaxf(s[i], s[4 + i]));
    }
    mt = ra_max_across_rows(mt);
    const float m_new = fmaxf(m_run, mt);
    const float alpha = ra_exp2(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s[i] = ra_exp2(s[i] - m_new);
      psum += s[i];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < DB; ++i) o[i] *= alpha;
    uint4 pw;
    pw.x = ra_pack_bf16x2(s[0], s[1]);
    pw.y = ra_pack_bf16x2(s[2], s[3]);
    pw.z = ra_pack_bf16x2(s[4], s[5]);
    pw.w = ra_pack_bf16x2(s[6], s[7]);
    const bf16x8_t pt = __builtin_bit_cast(bf16x8_t, pw);

    // V^T into LDS: element (d, k-slot); this lane holds d = 32ks + 8g4 + e.
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint32_t a4[4] = {wa[ks].x, wa[ks].y, wa[ks].z, wa[ks].w};
      const uint32_t b4[4] = {wb[ks].x, wb[ks].y, wb[ks].z, wb[ks].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int d0 = 32 * ks + 8 * g4 + 2 * e;
        vt[d0 * kVtPitch + col_a] = static_cast<unsigned short>(a4[e] & 0xFFFFu);
        vt[(d0 + 1) * kVtPitch + col_a] = static_cast<unsigned short>(a4[e] >> 16);
        vt[d0 * kVtPitch + col_b] = static_cast<unsigned short>(b4[e] & 0xFFFFu);
        vt[(d0 + 1) * kVtPitch + col_b] = static_cast<unsigned short>(b4[e] >> 16);
      }
    }
    __syncthreads();
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint4 a = *reinterpret_cast<const uint4*>(&vt[(16 * db + c) * kVtPitch + 8 * g4]);
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), pt, o[db], 0, 0, 0);
    }
    __syncthreads();
  }

  const float l_tot = ra_sum_across_rows(l_run);
  if (c >= grp) return;
  const int head = g * grp + c;
  const float inv = 1.f / l_tot;
  if (n_splits == 1) {
    __bf16* op = out + (static_cast<int64_t>(b) * hq + head) * D + 4 * g4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      uint2 w;
      w.x = ra_pack_bf16x2(o[db][0] * inv, o[db][1] * inv);
      w.y = ra_pack_bf16x2(o[db][2] * inv, o[db][3] * inv);
      *reinterpret_cast<uint2*>(op + 16 * db) = w;
    }
  } else {
    const int64_t pidx = (static_cast<int64_t>(b) * hq + head) * max_splits + split;
    float* wp = ws_o + pidx * D + 4 * g4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      *reinterpret_cast<float4*>(wp + 16 * db) =
          make_float4(o[db][0] * inv, o[db][1] * inv, o[db][2] * inv, o[db][3] * inv);
    }
    if (g4 == 0) ws_lse[pidx] = m_run + __log2f(l_tot);
  }
}

// Merges the chunks of one (request, head): weights 2^(lse_i - max lse).
template <int D>
__global__ __launch_bounds__(64) void decode_combine_kernel(const float* __restrict__ ws_o,
                                                            const float* __restrict__ ws_lse,
                                                            const int32_t* __restrict__ seq_lens,
                                                            int32_t hq, int32_t chunk_len, int32_t max_splits,
                                                            int32_t max_len, __bf16* __restrict__ out) {
  const int bh = blockIdx.x;
  const int b = bh / hq;
  const int L = min(seq_lens[b], max_len);
  const int n = (L + chunk_len - 1) / chunk_len;
  if (n <= 1) return;
  const float* lse = ws_lse + static_cast<int64_t>(bh) * max_splits;
  float mx = -INFINITY;
  for (int i = 0; i < n; ++i) mx = fmaxf(mx, lse[i]);
  constexpr int PER = D / 64;
  float acc[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) acc[j] = 0.f;
  float wsum = 0.f;
  const float* op = ws_o + static_cast<int64_t>(bh) * max_splits * D + threadIdx.x * PER;
  for (int i = 0; i < n; ++i) {
    const float w = ra_exp2(lse[i] - mx);
    wsum += w;
#pragma unroll
    for (int j = 0; j < PER; ++j) acc[j] += w * op[static_cast<int64_t>(i) * D + j];
  }
  const float inv = 1.f / wsum;
  __bf16* dst = out + static_cast<int64_t>(bh) * D + threadIdx.x * PER;
  if constexpr (PER == 2) {
    *reinterpret_cast<uint32_t*>(dst) = ra_pack_bf16x2(acc[0] * inv, acc[1] * inv);
  } else {
    const uint32_t w = ra_pack_bf16x2(acc[0] * inv, 0.f);
    *reinterpret_cast<unsigned short*>(dst) = static_cast<unsigned short>(w & 0xFFFFu);
  }
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

extern "C" int32_t ra_decode_chunk_len(int32_t batch, int32_t hkv, int32_t max_seq_len, int32_t num_splits) {
  if (max_seq_len <= 0) return kTile;
  if (num_splits > 0) {
    int64_t c = ceil_div(max_seq_len, num_splits);
    return static_cast<int32_t>(ceil_div(c, kTile) * kTile);
  }
  // Largest chunk that still gives enough work items to fill the chip
  // (256 CUs x 4 SIMDs, several waves each).
  const int64_t target = 4096;
  for (int32_t c : {2048, 1024, 512}) {
    if (static_cast<int64_t>(batch) * hkv * ceil_div(max_seq_len, c) >= target) return c;
  }
  return 256;
}

extern "C" size_t ra_decode_workspace_bytes(int32_t batch, int32_t hq, int32_t hkv, int32_t d,
                                            int32_t max_seq_len, int32_t num_splits) {
  if (batch <= 0 || hq <= 0 || hkv <= 0 || d <= 0 || max_seq_len <= 0) return 0;
  const int32_t chunk = ra_decode_chunk_len(batch, hkv, max_seq_len, num_splits);
  const int64_t splits = ceil_div(max_seq_len, chunk);
  if (splits <= 1) return 0;
  return static_cast<size_t>(batch) * hq * splits * (d + 1) * sizeof(float);
}

extern "C" int ra_decode_attention(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                                   const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                   const int32_t* req_pool_idx, const int32_t* seq_lens, int32_t batch, int32_t max_seq_len, int32_t hq,
                                   int32_t hkv, int32_t d, float scale, int32_t num_splits, void* workspace,
                                   size_t workspace_bytes, void* out, hipStream_t stream) {
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0 || (d != 64 && d != 128) || pool_slots <= 0 ||
      rtt_stride <= 0 || rtt_rows <= 0 || num_splits < 0)
    return ra_fail(RA_EINVAL, "ra_decode_attention: bad sizes");
  const int32_t grp = hq / hkv;
  if (grp > 16) return ra_fail(RA_EINVAL, "ra_decode_attention: more than 16 query heads per kv head");
  if (batch == 0) return ra_ok();
  if (max_seq_len <= 0) max_seq_len = static_cast<int32_t>(std::min<int64_t>(rtt_stride, INT32_MAX));
  if (max_seq_len > rtt_stride) return ra_fail(RA_EINVAL, "ra_decode_attention: max_seq_len > rtt_stride");
  if (!q || !k_pool || !v_pool || !req_to_token || !req_pool_idx || !seq_lens || !out)
    return ra_fail(RA_EINVAL, "ra_decode_attention: NULL pointer");
  if (!ra_aligned16(q) || !ra_aligned16(k_pool) || !ra_aligned16(v_pool) || !ra_aligned16(out))
    return ra_fail(RA_EINVAL, "ra_decode_attention: pointers must be 16-byte aligned");
  const int32_t chunk = ra_decode_chunk_len(batch, hkv, max_seq_len, num_splits);
  const int64_t splits = ceil_div(max_seq_len, chunk);
  const size_t need = ra_decode_workspace_bytes(batch, hq, hkv, d, max_seq_len, num_splits);
  if (workspace_bytes < need || (need && !workspace))
    return ra_fail(RA_EINVAL, "ra_decode_attention: workspace too small");
  if (need && !ra_aligned16(workspace)) return ra_fail(RA_EINVAL, "ra_decode_attention: workspace alignment");
  const int64_t items = static_cast<int64_t>(batch) * hkv * splits;
  if (items > INT32_MAX) return ra_fail(RA_EINVAL, "ra_decode_attention: too many work items");
  float* ws_o = static_cast<float*>(workspace);
  float* ws_lse = need ? ws_o + static_cast<int64_t>(batch) * hq * splits * d : nullptr;
  const float scale_log2 = scale * RA_LOG2E;
  const int32_t max_splits = static_cast<int32_t>(splits);
  auto* qp = static_cast<const __bf16*>(q);
  auto* kp = static_cast<const __bf16*>(k_pool);
  auto* vp = static_cast<const __bf16*>(v_pool);
  auto* op = static_cast<__bf16*>(out);
  if (d == 128) {
    hipLaunchKernelGGL(decode_partial_kernel<128>, dim3(static_cast<uint32_t>(items)), dim3(64), 0, stream, qp,
                       kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx, seq_lens, batch, hkv, grp,
                       chunk, max_splits, max_seq_len, scale_log2, ws_o, ws_lse, op);
  } else {
    hipLaunchKernelGGL(decode_partial_kernel<64>, dim3(static_cast<uint32_t>(items)), dim3(64), 0, stream, qp,
                       kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx, seq_lens, batch, hkv, grp,
                       chunk, max_splits, max_seq_len, scale_log2, ws_o, ws_lse, op);
  }
  int st = ra_check_launch("ra_decode_attention(partial)");
  if (st != RA_OK || splits <= 1) return st;
  const int64_t bh = static_cast<int64_t>(batch) * hq;
  if (d == 128) {
    hipLaunchKernelGGL(decode_combine_kernel<128>, dim3(static_cast<uint32_t>(bh)), dim3(64), 0, stream, ws_o,
                       ws_lse, seq_lens, hq, chunk, max_splits, max_seq_len, op);
  } else {
    hipLaunchKernelGGL(decode_combine_kernel<64>, dim3(static_cast<uint32_t>(bh)), dim3(64), 0, stream, ws_o,
                       ws_lse, seq_lens, hq, chunk, max_splits, max_seq_len, op);
  }
  return ra_check_launch("ra_decode_attention(combine)");
}
