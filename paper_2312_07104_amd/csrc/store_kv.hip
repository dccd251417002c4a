// Scatter of new tokens' K and V rows into the token-granular pool (one
// token per page, section 3).  One wave per token: the slot index is
// wave-uniform, and each pass of the wave reads 1 KB of the token's K row and
// of its V row contiguously and writes them as 1 KB runs at the slot (no
// per-element index arithmetic).
#include "device_common.h"

namespace {

constexpr int kTokensPerBlock = 4;  // four waves of 64 lanes

__global__ __launch_bounds__(64 * kTokensPerBlock) void store_kv_kernel(const int32_t* __restrict__ slots,
                                                                         const uint4* __restrict__ k_new,
                                                                         const uint4* __restrict__ v_new,
                                                                         uint4* __restrict__ k_pool,
                                                                         uint4* __restrict__ v_pool,
                                                                         int64_t n_tokens, int64_t pool_slots,
                                                                         int32_t row_pieces) {
  const int64_t tok = static_cast<int64_t>(blockIdx.x) * kTokensPerBlock +
                      __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  if (tok >= n_tokens) return;
  const int64_t slot = slots[tok];
  if (slot < 0 || slot >= pool_slots) return;
  const uint4* ks = k_new + tok * row_pieces;
  const uint4* vs = v_new + tok * row_pieces;
  uint4* kd = k_pool + slot * row_pieces;
  uint4* vd = v_pool + slot * row_pieces;
  for (int p = threadIdx.x & 63; p < row_pieces; p += 64) {
    const uint4 k = ks[p];
    const uint4 v = vs[p];
    kd[p] = k;
    vd[p] = v;
  }
}

}  // namespace

extern "C" int ra_store_kv(const int32_t* slots, const void* k_new, const void* v_new, int64_t n_tokens,
                           void* k_pool, void* v_pool, int64_t pool_slots, int32_t hkv, int32_t d,
                           hipStream_t stream) {
  if (n_tokens < 0 || hkv <= 0 || (d != 64 && d != 128) || pool_slots <= 0)
    return ra_fail(RA_EINVAL, "ra_store_kv: bad sizes");
  if (n_tokens == 0) return ra_ok();
  if (!slots || !k_new || !v_new || !k_pool || !v_pool)
    return ra_fail(RA_EINVAL, "ra_store_kv: NULL pointer");
  if (!ra_aligned16(k_new) || !ra_aligned16(v_new) || !ra_aligned16(k_pool) || !ra_aligned16(v_pool))
    return ra_fail(RA_EINVAL, "ra_store_kv: pointers must be 16-byte aligned");
  const int32_t row_pieces = hkv * d / 8;  // 8 bf16 per 16-byte piece
  const int64_t blocks = (n_tokens + kTokensPerBlock - 1) / kTokensPerBlock;
  if (blocks > INT32_MAX) return ra_fail(RA_EINVAL, "ra_store_kv: too many tokens");
  hipLaunchKernelGGL(store_kv_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(64 * kTokensPerBlock), 0, stream,
                     slots, static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new),
                     static_cast<uint4*>(k_pool), static_cast<uint4*>(v_pool), n_tokens, pool_slots,
                     row_pieces);
  return ra_check_launch("ra_store_kv");
}
