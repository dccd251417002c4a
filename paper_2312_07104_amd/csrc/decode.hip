// Decode attention over the token-granular KV pool: one query token per
// request over its whole context (prefix plus private suffix), read through
// the request's row of the slot table.  Decode dominates when outputs are
// long (evaluation, section 6.2); it is bound by HBM bandwidth, so the design
// goal is a steady stream of gathered 256-byte K/V rows.
//
// Work item = (request, kv head, KV chunk); one wave per item.  Items go out
// in (split, request) order with the kv head fastest (ra_decode_item), or,
// for chunks of 2048 tokens and up, longest first (ra_decode_lpt_item).  Two
// partial-pass kernels share the item layout, the per-tile arithmetic and the
// outputs: decode_partial_vr_kernel (D = 128) stages the gathered rows in
// registers, decode_partial_kernel (D = 64) copies them straight into LDS:
//   * Gather: every 32-token tile's K and V rows are copied HBM -> LDS with
//     direct-to-LDS loads (global_load_lds_dwordx4), kNS tiles deep, no VGPR
//     staging; the slot indices travel the same way one tile further ahead,
//     so no load waits on an index.  Rows are unpadded (2*D bytes) with their
//     16-byte pieces XOR-swizzled by ra_kv_swz(row) (conflict-free reads).
//   * The G query heads that share the kv head are the N = 16 columns of
//     bf16 MFMAs, so each K/V row fetched serves all G heads and the VALU is
//     left for the softmax:  S^T[token, head] = K Q^T, O^T += V^T P^T, V^T
//     read from the row-major LDS tile with ds_read_b64_tr_b16.
//   * Online softmax in the base-2 domain with a lazily moved maximum; the
//     maximum is reduced across the four 16-lane rows with permlane swaps,
//     the sum stays per lane and is reduced once at the end.
// A chunk writes a normalised partial output and its log2-sum-exp; a second
// kernel merges the chunks.  DMAs are issued from inline assembly (the
// compiler would wait for them before every LDS read); waits are explicit.

#include <mutex>

#include "device_common.h"
#include "lds_dma.h"

namespace {

constexpr int kTile = 32;  // tokens per tile (two 16-row MFMA blocks)

// Work item of block k: unit k / hkv of kv head k % hkv, units ordered
// (split, request).  The dispatcher deals blocks to the 8 XCDs round-robin,
// so with 8 kv heads each XCD serves one kv head (its requests in flight
// share prefix chunks through its L2), and with fewer kv heads the XCDs that
// share a kv head take its units in turn: every XCD gets the same mix of
// requests, not a contiguous run of them.  Returns false past the last item.
__device__ __forceinline__ bool ra_decode_item(int64_t k, int32_t hkv, int32_t max_splits, int32_t batch, int& g,
                                               int& split, int& b) {
  const int64_t unit = k / hkv;
  if (unit >= static_cast<int64_t>(max_splits) * batch) return false;
  g = static_cast<int>(k % hkv);
  split = static_cast<int>(unit / batch);
  b = static_cast<int>(unit % batch);
  return true;
}

// Longest-first variant for batches up to kDecLptMaxBatch requests whose
// contexts span at most kDecLptMaxSplits chunks.  Units are the (request,
// chunk) pairs.  Full chunks come first, in (split, request) order as above
// (requests that share a prefix read the same rows side by side); then each
// request's partial last chunk, longest first (lengths in 64 buckets of
// chunk_len / 64 tokens, ties by request index).  Without it the partial
// chunks sit among the full ones and a few full chunks start last.  One wave
// per work-group: it reads the batch's lengths once into `lds` (batch + 129
// words, the work-group's staging LDS before its first use), counts requests
// by full chunks and partial chunks by bucket, and finds unit k / hkv with
// wave scans and ballots.  Returns false past the last unit.
constexpr int kDecLptMaxBatch = 1536;
constexpr int kDecLptMaxSplits = 64;
// Words of LDS the ranking uses: the lengths, the full-chunk histogram
// (kDecLptMaxSplits + 1 bins) and the partial-chunk histogram (64 bins).
constexpr int kDecLptWords = kDecLptMaxBatch + kDecLptMaxSplits + 1 + 64;

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int up = __shfl_up(v, d, 64);
    if (lane >= d) v += up;
  }
  return v;
}

// Index (in request order) of the i-th request among those with pred set,
// or -1; pred(t) for t < batch.  Wave-uniform.
template <typename Pred>
__device__ __forceinline__ int wave_select(int batch, int i, Pred pred) {
  const int lane = threadIdx.x & 63;
  const uint64_t below = (uint64_t{1} << lane) - 1;
  for (int base = 0; base < batch; base += 64) {
    const int t = base + lane;
    const bool p = t < batch && pred(t);
    const uint64_t m = __ballot(p);
    const int cnt = __popcll(m);
    if (i < cnt) {
      const uint64_t hit = __ballot(p && __popcll(m & below) == i);
      return base + __ffsll(static_cast<unsigned long long>(hit)) - 1;
    }
    i -= cnt;
  }
  return -1;
}

__device__ bool ra_decode_lpt_item(int32_t* lds, int64_t k, int32_t hkv, int32_t batch, int32_t chunk_len,
                                   int32_t max_len, const int32_t* __restrict__ seq_lens, int& g, int& split,
                                   int& b) {
  int32_t* len = lds;                          // [batch] context lengths as the kernel clamps them
  int32_t* hf = lds + batch;                   // [65] requests by number of full chunks
  int32_t* hr = hf + kDecLptMaxSplits + 1;     // [64] partial chunks by length bucket
  const int lane = threadIdx.x;
  hf[lane] = 0;
  hr[lane] = 0;
  if (lane == 0) hf[kDecLptMaxSplits] = 0;
  __syncthreads();
  auto bucket = [&](int rm) { return static_cast<int>(static_cast<int64_t>(rm) * 64 / chunk_len); };
  for (int t = lane; t < batch; t += 64) {
    const int L = max(min(seq_lens[t], max_len), 0);
    len[t] = L;
    const int nf = L / chunk_len, rm = L - nf * chunk_len;
    atomicAdd(&hf[min(nf, kDecLptMaxSplits)], 1);
    if (rm > 0) atomicAdd(&hr[bucket(rm)], 1);
  }
  __syncthreads();
  const int64_t u = k / hkv;
  // lane s: c = full chunks at split s (requests with more than s full chunks)
  const int c = batch - wave_incl_scan(hf[lane]);
  const int cin = wave_incl_scan(c);
  const int64_t n_full = __shfl(cin, 63, 64);
  int req = -1, sp = 0;
  if (u < n_full) {
    const int ui = static_cast<int>(u);
    const uint64_t at = __ballot(ui >= cin - c && ui < cin);
    sp = __ffsll(static_cast<unsigned long long>(at)) - 1;
    const int i = ui - (__shfl(cin, sp, 64) - __shfl(c, sp, 64));
    req = wave_select(batch, i, [&](int t) { return len[t] / chunk_len > sp; });
  } else {
    // lane q: bucket 63 - q, longest first
    const int h = hr[63 - lane];
    const int hin = wave_incl_scan(h);
    const int64_t i64 = u - n_full;
    if (i64 < __shfl(hin, 63, 64)) {
      const int i = static_cast<int>(i64);
      const uint64_t at = __ballot(i >= hin - h && i < hin);
      const int q = __ffsll(static_cast<unsigned long long>(at)) - 1;
      const int bk = 63 - q;
      const int j = i - (__shfl(hin, q, 64) - __shfl(h, q, 64));
      req = wave_select(batch, j, [&](int t) {
        const int rm = len[t] % chunk_len;
        return rm > 0 && bucket(rm) == bk;
      });
      if (req >= 0) sp = len[req] / chunk_len;
    }
  }
  // the scratch is the work-group's staging LDS, which the loads use next
  __syncthreads();
  if (req < 0) return false;
  g = static_cast<int>(k % hkv);
  split = sp;
  b = req;
  return true;
}

// LDS tile layout (K and V alike): [piece group pg = D/32][token row][4
// pieces of 16 B], pieces swizzled by ra_kv_swz (conflict-free operand reads,
// every read one per-lane offset plus an immediate).

// Waits until the K/V tile t (and the slot indices issued with it) are in
// LDS, given that `later` further K/V tiles (2*LOADS DMAs each) were issued
// after it; vmcnt counts outstanding loads in issue order.
template <int LOADS, int K>
__device__ __forceinline__ void wait_for_tile_k(int later) {
  if constexpr (K > 0) {
    if (later >= K) {
      ra_wait_vmcnt<K * 2 * LOADS>();
      return;
    }
    wait_for_tile_k<LOADS, K - 1>(later);
  } else {
    ra_wait_vmcnt<0>();
  }
}
template <int LOADS, int NS>
__device__ __forceinline__ void wait_for_tile(int later) {
  wait_for_tile_k<LOADS, NS - 2>(later);
}

template <int D, int NS>
__global__ __launch_bounds__(64) void decode_partial_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k_pool, const __bf16* __restrict__ v_pool,
    int64_t pool_slots, const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride,
    const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ seq_lens, int32_t batch,
    int32_t hkv, int32_t grp, int32_t chunk_len, int32_t max_splits, int32_t max_len, int32_t lpt,
    float scale_log2, float* __restrict__ ws_o, float* __restrict__ ws_lse, __bf16* __restrict__ out) {
  constexpr int TILE = kTile;
  constexpr int KS = D / 32;             // MFMA k-steps over the head dimension = piece groups
  constexpr int DB = D / 16;             // 16-row blocks of O^T
  constexpr int GROUP_B = TILE * 64;     // bytes of one piece group of a tile
  constexpr int TILE_B = KS * GROUP_B;   // bytes per K (or V) tile
  constexpr int LOADS = TILE_B / 1024;   // DMA instructions per tile per tensor
  constexpr int RING = 2 * NS;           // slot-index ring (indices run NS-1 tiles ahead of K/V)
  constexpr int IDX_AHEAD = NS - 1;
  __shared__ __align__(16) unsigned char kv_lds[NS][2][TILE_B];
  __shared__ __align__(16) int32_t idx_lds[RING][64];
  static_assert(kDecLptWords * 4 <= sizeof(kv_lds), "ranking scratch exceeds the staging LDS");

  int g, split, b;
  if (lpt ? !ra_decode_lpt_item(reinterpret_cast<int32_t*>(&kv_lds[0][0][0]), blockIdx.x, hkv, batch, chunk_len, max_len,
                                seq_lens, g, split, b)
          : !ra_decode_item(blockIdx.x, hkv, max_splits, batch, g, split, b))
    return;
  const int L = min(seq_lens[b], max_len);  // host bound (<= rtt_stride, <= chunk_len * max_splits)
  if (L <= 0) return;
  const int n_splits = (L + chunk_len - 1) / chunk_len;
  if (split >= n_splits) return;
  const int t_begin = split * chunk_len;
  const int t_end = min(L, t_begin + chunk_len);
  int64_t rrow = req_pool_idx[b];
  rrow = (rrow >= 0 && rrow < rtt_rows) ? rrow : 0;
  const int32_t* trow = rtt + rrow * rtt_stride;
  const int hq = hkv * grp;
  const int n_tiles = (t_end - t_begin + TILE - 1) / TILE;

  const int lane = threadIdx.x;
  const int c = lane & 15;   // query head column / A-operand row
  const int g4 = lane >> 4;  // which 16-lane row of the wave

  // DMA lane mapping: instruction ch covers rows 16 (ch / KS) .. +15 of piece group ch % KS.
  int dma_row[LOADS];
  uint32_t dma_lds[LOADS], dma_gofs[LOADS];
#pragma unroll
  for (int ch = 0; ch < LOADS; ++ch) {
    const int rb = ch / KS, pg = ch % KS;
    const int u = 16 * rb + (lane >> 2);
    dma_row[ch] = u;
    dma_lds[ch] = pg * GROUP_B + rb * 1024;
    dma_gofs[ch] = static_cast<uint32_t>(g * D * 2 + 16 * (4 * pg + ((lane & 3) ^ ra_kv_swz(u))));
  }
  const uint32_t row_bytes = static_cast<uint32_t>(hkv) * D * 2;
  const unsigned char* kpool_b = reinterpret_cast<const unsigned char*>(k_pool);
  const unsigned char* vpool_b = reinterpret_cast<const unsigned char*>(v_pool);
  const uint32_t smax = static_cast<uint32_t>(pool_slots - 1);

  auto issue_idx = [&](int tile) {
    if (tile >= n_tiles) return;
    const int pos = min(t_begin + tile * TILE + (lane & (TILE - 1)), t_end - 1);  // padding repeats a real token
    ra_dma4(trow + pos, ra_lds_addr(&idx_lds[tile % RING][0]));
  };
  auto issue_kv = [&](int tile) {
    if (tile >= n_tiles) return;
    const int32_t* ring = idx_lds[tile % RING];
    const uint32_t kst = ra_lds_addr(kv_lds[tile % NS][0]);
    const uint32_t vst = ra_lds_addr(kv_lds[tile % NS][1]);
#pragma unroll
    for (int ch = 0; ch < LOADS; ++ch) {
      const uint32_t slot = min(static_cast<uint32_t>(ring[dma_row[ch]]), smax);  // negative -> clamped
      const uint64_t off = static_cast<uint64_t>(slot) * row_bytes + dma_gofs[ch];
      ra_dma16(kpool_b + off, __builtin_amdgcn_readfirstlane(kst + dma_lds[ch]));
      ra_dma16(vpool_b + off, __builtin_amdgcn_readfirstlane(vst + dma_lds[ch]));
    }
  };

  // Q^T (loaded before the first DMA so that the compiler's wait for
  // these loads does not also wait for the prologue's DMAs).
  // Q^T as the B operand: column c = head g*grp + c, k = 8*g4 .. of each step.
  bf16x8_t qt[KS];
  {
    const bool has = c < grp;
    const __bf16* qp = q + (static_cast<int64_t>(b) * hq + g * grp + (has ? c : 0)) * D + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qt[ks] = __builtin_bit_cast(bf16x8_t, has ? ra_ld16(qp + 32 * ks) : make_uint4(0, 0, 0, 0));
  }

  // prologue: indices for the first NS-1+IDX_AHEAD tiles, K/V for the first NS-1
  for (int t = 0; t < NS - 1 + IDX_AHEAD; ++t) issue_idx(t);
  ra_wait_vmcnt<0>();
  __syncthreads();
  for (int t = 0; t < NS - 1; ++t) issue_kv(t);

  f32x4_t o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // raw score units
  float l_run = 0.f;

  // K A-operand rows: row c of block bb gets token 8 (c >> 2) + 4 bb + (c & 3),
  // so accumulator row group g4 holds tokens 8 g4 .. 8 g4 + 7 (P^T's k slots
  // in natural order).
  const int kr0 = 8 * (c >> 2) + (c & 3);
  const uint32_t koff = kr0 * 64 + 16 * (g4 ^ ra_kv_swz(kr0));
  // V^T by transposed reads: lane supplies row vr0 (+ 4 h), logical piece
  // 2 db + ((c & 3) >> 1), half (c & 1).
  const int vr0 = 8 * g4 + (c >> 2);
  uint32_t voff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) voff[e] = vr0 * 64 + 16 * ((2 * e + ((c & 3) >> 1)) ^ ra_kv_swz(vr0)) + 8 * (c & 1);
  constexpr int NB = TILE / 16;  // S^T blocks per tile

  for (int t = 0; t < n_tiles; ++t) {
    wait_for_tile<LOADS, NS>(min(NS - 2, n_tiles - 1 - t));
    __syncthreads();
    issue_idx(t + NS - 1 + IDX_AHEAD);
    issue_kv(t + NS - 1);

    const unsigned char* kst = kv_lds[t % NS][0];
    const unsigned char* vst = kv_lds[t % NS][1];
    const int t0 = t_begin + t * TILE;

    f32x4_t sacc[NB];
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
      sacc[bb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8_t a = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const uint4*>(kst + koff + ks * GROUP_B + 4 * bb * 64));
        sacc[bb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qt[ks], sacc[bb], 0, 0, 0);
      }
    }
    // element (bb, i) is token t0 + 8 g4 + 4 bb + i
    if (t0 + TILE > t_end) {
#pragma unroll
      for (int bb = 0; bb < NB; ++bb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = t0 + 8 * g4 + 4 * bb + i;
          if (tok >= t_end) sacc[bb][i] = -INFINITY;
        }
    }
    float mt = fmaxf(fmaxf(fmaxf(sacc[0][0], sacc[0][1]), fmaxf(sacc[0][2], sacc[0][3])),
                     fmaxf(fmaxf(sacc[1][0], sacc[1][1]), fmaxf(sacc[1][2], sacc[1][3])));
    mt = ra_max_across_rows(mt);
    if (__builtin_amdgcn_ballot_w64((mt - m_run) * scale_log2 > 8.f) != 0) {
      const float m_new = fmaxf(m_run, mt);
      const float alpha = ra_exp2((m_run - m_new) * scale_log2);
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < DB; ++i) o[i] *= alpha;
      m_run = m_new;
    }
    const float mb = -m_run * scale_log2;
    float p[8];
#pragma unroll
    for (int bb = 0; bb < NB; ++bb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[4 * bb + i] = ra_exp2(__builtin_fmaf(sacc[bb][i], scale_log2, mb));
        l_run += p[4 * bb + i];
      }
    uint4 pw;
    pw.x = ra_pack_bf16x2(p[0], p[1]);
    pw.y = ra_pack_bf16x2(p[2], p[3]);
    pw.z = ra_pack_bf16x2(p[4], p[5]);
    pw.w = ra_pack_bf16x2(p[6], p[7]);
    const bf16x8_t pt = __builtin_bit_cast(bf16x8_t, pw);

    // O^T += V^T P^T: lane receives column 16 db + c of rows vr0 - (c >> 2) + 0..3 (+ 4 h).
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const unsigned char* vb = vst + voff[db & 1] + (db >> 1) * GROUP_B;
      const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4_t*)(vb));
      const bf16x4_t hi =
          __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4_t*)(vb + 4 * 64));
      const bf16x8_t a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pt, o[db], 0, 0, 0);
    }
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
    if (g4 == 0) ws_lse[pidx] = m_run * scale_log2 + __log2f(l_tot);
  }
}

// Decode partial pass with register staging (D = 128).  The kernel above
// copies K and V straight into LDS, so its tiles in flight are bounded twice
// (measured with D = 128):
// a wave's vector-memory counter holds 63 loads (three 16 KB tiles of 1 KB
// copies), and LDS holds two such rings per CU, 96 KB in flight per CU in
// all.  Decode is bound by exactly that: with one of the two waves per CU
// removed it runs at 0.54-0.65x.  Here each tile's rows are read with
// ordinary vector loads into registers: K straight into the MFMA A-operand
// layout (16 bytes of one row per lane, the same lanes and rows the LDS
// kernel reads), V in the copy layout, written to a single 8 KB LDS tile just
// before its PV step (V^T needs the transposing LDS read).  Registers hold
// the NP tiles in flight, the compiler tracks every load (no hand-counted
// waits), and LDS no longer limits the waves per CU.  Per tile the arithmetic
// (operands, accumulation order, maximum rule, rounding) is that of
// decode_partial_kernel, so the two write bit-identical partial outputs.
template <int NP>
__global__ __launch_bounds__(64) void decode_partial_vr_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k_pool, const __bf16* __restrict__ v_pool,
    int64_t pool_slots, const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride,
    const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ seq_lens, int32_t batch,
    int32_t hkv, int32_t grp, int32_t chunk_len, int32_t max_splits, int32_t max_len, int32_t lpt,
    float scale_log2, float* __restrict__ ws_o, float* __restrict__ ws_lse, __bf16* __restrict__ out) {
  constexpr int D = 128;
  constexpr int TILE = kTile;
  constexpr int KS = D / 32;
  constexpr int DB = D / 16;
  constexpr int NB = TILE / 16;
  constexpr int GROUP_B = TILE * 64;
  constexpr int TILE_B = KS * GROUP_B;
  __shared__ __align__(16) unsigned char v_lds[TILE_B];
  static_assert(kDecLptWords * 4 <= sizeof(v_lds), "ranking scratch exceeds the staging LDS");

  int g, split, b;
  if (lpt ? !ra_decode_lpt_item(reinterpret_cast<int32_t*>(v_lds), blockIdx.x, hkv, batch, chunk_len, max_len,
                                seq_lens, g, split, b)
          : !ra_decode_item(blockIdx.x, hkv, max_splits, batch, g, split, b))
    return;
  const int L = min(seq_lens[b], max_len);
  if (L <= 0) return;
  const int n_splits = (L + chunk_len - 1) / chunk_len;
  if (split >= n_splits) return;
  const int t_begin = split * chunk_len;
  const int t_end = min(L, t_begin + chunk_len);
  int64_t rrow = req_pool_idx[b];
  rrow = (rrow >= 0 && rrow < rtt_rows) ? rrow : 0;
  const int32_t* trow = rtt + rrow * rtt_stride;
  const int hq = hkv * grp;
  const int n_tiles = (t_end - t_begin + TILE - 1) / TILE;

  const int lane = threadIdx.x;
  const int c = lane & 15;
  const int g4 = lane >> 4;
  // Rows of a tile this lane loads.  K: A-operand row c of block bb is token
  // 8 (c >> 2) + 4 bb + (c & 3) (so accumulator row group g4 holds tokens
  // 8 g4 .. 8 g4 + 7, P^T's k slots in order); the lane's 16 bytes of each
  // k-step are d = 32 ks + 8 g4 .. + 7.  V: copy row u = 16 rb + (lane >> 2),
  // logical piece (lane & 3) ^ swizzle(u) of each 64-byte piece group, stored
  // at LDS byte pg * GROUP_B + rb * 1024 + 16 lane (the LDS kernel's layout).
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

  // Slot index of token (lane & 31) of a tile; padding repeats the last token.
  auto load_idx = [&](int tile) -> int32_t {
    const int pos = min(t_begin + tile * TILE + (lane & (TILE - 1)), t_end - 1);
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

  bf16x8_t qt[KS];
  {
    const bool has = c < grp;
    const __bf16* qp = q + (static_cast<int64_t>(b) * hq + g * grp + (has ? c : 0)) * D + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qt[ks] = __builtin_bit_cast(bf16x8_t, has ? ra_ld16(qp + 32 * ks) : make_uint4(0, 0, 0, 0));
  }

#pragma unroll
  for (int j = 0; j < NP; ++j) ibuf[j] = load_idx(j);
#pragma unroll
  for (int j = 0; j < NP; ++j)
    if (j < n_tiles) load_tile(j, ibuf[j]);
#pragma unroll
  for (int j = 0; j < NP; ++j) ibuf[j] = load_idx(j + NP);

  f32x4_t o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;
  float l_run = 0.f;
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
        f32x4_t sacc[NB];
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) {
          sacc[bb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            sacc[bb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kbuf[j][bb][ks]),
                                                                qt[ks], sacc[bb], 0, 0, 0);
        }
        // Slot j is consumed: refill it with tile t + NP, and its index
        // register with the indices of tile t + 2 NP.
        if (t + NP < n_tiles) load_tile(j, ibuf[j]);
        ibuf[j] = load_idx(t + 2 * NP);

        if (t0 + TILE > t_end) {
#pragma unroll
          for (int bb = 0; bb < NB; ++bb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int tok = t0 + 8 * g4 + 4 * bb + i;
              if (tok >= t_end) sacc[bb][i] = -INFINITY;
            }
        }
        float mt = fmaxf(fmaxf(fmaxf(sacc[0][0], sacc[0][1]), fmaxf(sacc[0][2], sacc[0][3])),
                         fmaxf(fmaxf(sacc[1][0], sacc[1][1]), fmaxf(sacc[1][2], sacc[1][3])));
        mt = ra_max_across_rows(mt);
        if (__builtin_amdgcn_ballot_w64((mt - m_run) * scale_log2 > 8.f) != 0) {
          const float m_new = fmaxf(m_run, mt);
          const float alpha = ra_exp2((m_run - m_new) * scale_log2);
          l_run *= alpha;
#pragma unroll
          for (int i = 0; i < DB; ++i) o[i] *= alpha;
          m_run = m_new;
        }
        const float mb = -m_run * scale_log2;
        float p[8];
#pragma unroll
        for (int bb = 0; bb < NB; ++bb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            p[4 * bb + i] = ra_exp2(__builtin_fmaf(sacc[bb][i], scale_log2, mb));
            l_run += p[4 * bb + i];
          }
        uint4 pw;
        pw.x = ra_pack_bf16x2(p[0], p[1]);
        pw.y = ra_pack_bf16x2(p[2], p[3]);
        pw.z = ra_pack_bf16x2(p[4], p[5]);
        pw.w = ra_pack_bf16x2(p[6], p[7]);
        const bf16x8_t pt = __builtin_bit_cast(bf16x8_t, pw);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const unsigned char* vb = v_lds + voff[db & 1] + (db >> 1) * GROUP_B;
          const bf16x4_t lo =
              __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4_t*)(vb));
          const bf16x4_t hi =
              __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4_t*)(vb + 4 * 64));
          const bf16x8_t a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pt, o[db], 0, 0, 0);
        }
      }
    }
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
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<float4*>(wp + 16 * db) =
          make_float4(o[db][0] * inv, o[db][1] * inv, o[db][2] * inv, o[db][3] * inv);
    if (g4 == 0) ws_lse[pidx] = m_run * scale_log2 + __log2f(l_tot);
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
  // Largest chunk that still gives enough work items to keep every CU
  // streaming (256 CUs, a few waves each, several rounds for balance).
  constexpr int64_t kTargetItems = 4096;
  for (int32_t c : {4096, 2048, 1024, 512}) {
    if (static_cast<int64_t>(batch) * hkv * ceil_div(max_seq_len, c) >= kTargetItems) return c;
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

// Argument checks shared with ra_mixed_attention: RA_OK when the call may
// launch (or has nothing to do), an error status otherwise.
int ra_decode_validate(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                       const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, const int32_t* req_pool_idx,
                       const int32_t* seq_lens, int32_t batch, int32_t max_seq_len, int32_t hq, int32_t hkv, int32_t d,
                       float scale, int32_t num_splits, const void* workspace, size_t workspace_bytes,
                       const void* out) {
  if (batch < 0 || hq <= 0 || hkv <= 0 || hq % hkv != 0 || (d != 64 && d != 128) || pool_slots <= 0 ||
      rtt_stride <= 0 || rtt_rows <= 0 || num_splits < 0 || !(scale > 0.f))
    return ra_fail(RA_EINVAL, "ra_decode_attention: bad sizes or scale");
  if (hq / hkv > 16) return ra_fail(RA_EINVAL, "ra_decode_attention: more than 16 query heads per kv head");
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
  if (static_cast<int64_t>(batch) * hkv * splits + 8 > INT32_MAX)
    return ra_fail(RA_EINVAL, "ra_decode_attention: too many work items");
  return ra_ok();
}

extern "C" int ra_decode_attention(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                                   const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                   const int32_t* req_pool_idx, const int32_t* seq_lens, int32_t batch,
                                   int32_t max_seq_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                                   int32_t num_splits, void* workspace, size_t workspace_bytes, void* out,
                                   hipStream_t stream) {
  const int st0 = ra_decode_validate(q, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx,
                                     seq_lens, batch, max_seq_len, hq, hkv, d, scale, num_splits, workspace,
                                     workspace_bytes, out);
  if (st0 != RA_OK || batch == 0) return st0;
  if (max_seq_len <= 0) max_seq_len = static_cast<int32_t>(std::min<int64_t>(rtt_stride, INT32_MAX));
  if (ra_debug_checks_enabled()) {
    const int cst = ra_check_batch(req_to_token, rtt_rows, rtt_stride, pool_slots, req_pool_idx, batch, nullptr,
                                   nullptr, nullptr, 0, 0, seq_lens, max_seq_len, stream);
    if (cst != RA_OK) return cst;
  }
  const int32_t grp = hq / hkv;
  const int32_t chunk = ra_decode_chunk_len(batch, hkv, max_seq_len, num_splits);
  const int64_t splits = ceil_div(max_seq_len, chunk);
  const size_t need = ra_decode_workspace_bytes(batch, hq, hkv, d, max_seq_len, num_splits);
  const int64_t items = static_cast<int64_t>(batch) * hkv * splits;
  float* ws_o = static_cast<float*>(workspace);
  float* ws_lse = need ? ws_o + static_cast<int64_t>(batch) * hq * splits * d : nullptr;
  const float scale_log2 = scale * RA_LOG2E;
  const int32_t max_splits = static_cast<int32_t>(splits);
  auto* qp = static_cast<const __bf16*>(q);
  auto* kp = static_cast<const __bf16*>(k_pool);
  auto* vp = static_cast<const __bf16*>(v_pool);
  auto* op = static_cast<__bf16*>(out);
  const int64_t grid = (items + 7) / 8 * 8;  // whole XCD rounds
  // Longest first when the batch's items take more than one round of the
  // chip's wave slots (four per CU), its lengths fit the ranking scratch, and
  // its chunks are long (2048 tokens and up).  The ranking costs each item
  // about 2 us; on shorter chunks that outweighs the shorter tail (measured:
  // 4-8% slower on batches of 256- to 1024-token chunks, 1.5-5% faster on
  // 2048- and 4096-token chunks).
  const int32_t lpt = batch <= kDecLptMaxBatch && max_splits <= kDecLptMaxSplits && chunk >= 2048 &&
                      items > static_cast<int64_t>(ra_device_cus()) * 4 ? 1 : 0;
#define RA_LAUNCH_DECODE(DD, NN)                                                                                  \
  hipLaunchKernelGGL((decode_partial_kernel<DD, NN>), dim3(static_cast<uint32_t>(grid)), dim3(64), 0, stream, \
                     qp, kp, vp, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx, seq_lens, batch, hkv, \
                     grp, chunk, max_splits, max_seq_len, lpt, scale_log2, ws_o, ws_lse, op)
  // D = 128: register staging, two tiles in flight per wave, four waves per
  // CU (measured against the LDS-copy kernel with a three- or four-tile
  // ring: 7% faster on 512 requests of 1k-16k tokens, 8% on 256-request chat
  // batches, 11% on the branching decode, 2-7% on head shards; three or four
  // tiles in flight per wave are no faster).  D = 64: the LDS-copy kernel,
  // three-tile ring.
  if (d == 128) {
    hipLaunchKernelGGL((decode_partial_vr_kernel<2>), dim3(static_cast<uint32_t>(grid)), dim3(64), 0, stream, qp, kp,
                       vp, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx, seq_lens, batch, hkv, grp,
                       chunk, max_splits, max_seq_len, lpt, scale_log2, ws_o, ws_lse, op);
  } else {
    RA_LAUNCH_DECODE(64, 3);
  }
#undef RA_LAUNCH_DECODE
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

// ---------------------------------------------------------------------------
// Allocation-free variant: the split-KV partials live in a file-scope device
// array instead of a caller workspace.
// ---------------------------------------------------------------------------

// One copy per device, held until the process ends.  In host code `scratch`
// names a host-side stand-in, never device memory: kernels receive the
// address hipGetSymbolAddress reports for the current device.
constexpr size_t kNoAllocScratchBytes = size_t{128} << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[64] = {};

// Device address of this device's scratch, looked up once per device (with
// that device current, as the caller's calls run).
int scratch_for_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
    return ra_fail(RA_EHIP, "ra_decode_attention_noalloc: no usable current device");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr)
      return ra_fail(RA_EHIP, std::string("ra_decode_attention_noalloc: hipGetSymbolAddress: ") +
                                  hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return RA_OK;
}

}  // namespace

extern "C" size_t ra_decode_noalloc_max_scratch_bytes(void) { return kNoAllocScratchBytes; }

extern "C" int ra_decode_attention_noalloc(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                                           const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                           const int32_t* req_pool_idx, const int32_t* seq_lens, int32_t batch,
                                           int32_t max_seq_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                                           int32_t num_splits, void* out, hipStream_t stream) {
  int32_t msl = max_seq_len;
  if (msl <= 0 && rtt_stride > 0) msl = static_cast<int32_t>(std::min<int64_t>(rtt_stride, INT32_MAX));
  const size_t need = ra_decode_workspace_bytes(batch, hq, hkv, d, msl, num_splits);
  if (need > kNoAllocScratchBytes)
    return ra_fail(RA_EINVAL, "ra_decode_attention_noalloc: the batch needs " + std::to_string(need) +
                                  " bytes of split scratch, more than the " +
                                  std::to_string(kNoAllocScratchBytes) + " this entry point holds");
  void* ws = nullptr;
  if (need) {
    const int st = scratch_for_current_device(&ws);
    if (st != RA_OK) return st;
  }
  return ra_decode_attention(q, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx,
                             seq_lens, batch, max_seq_len, hq, hkv, d, scale, num_splits, ws, need, out, stream);
}
