// Scatter of new tokens' K and V rows into the token-granular pool (one
// token per page, section 3).  Each thread moves one 16-byte piece of a K row
// and the matching piece of the V row; consecutive threads cover consecutive
// pieces of a row, so both the contiguous reads and the scattered writes are
// full 64-byte-or-wider segments per token.
#include "device_common.h"

namespace {

__global__ __launch_bounds__(256) void store_kv_kernel(const int32_t* __restrict__ slots,
                                                        const uint4* __restrict__ k_new,
                                                        const uint4* __restrict__ v_new,
                                                        uint4* __restrict__ k_pool,
                                                        uint4* __restrict__ v_pool, int64_t n_tokens,
                                                        int64_t pool_slots, int32_t row_pieces) {
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  int64_t total = n_tokens * row_pieces;
  if (i >= total) return;
  int64_t tok = i / row_pieces;
  int32_t piece = static_cast<int32_t>(i - tok * row_pieces);
  int64_t slot = slots[tok];
  if (slot < 0 || slot >= pool_slots) return;
  uint4 k = k_new[i];
  uint4 v = v_new[i];
  k_pool[slot * row_pieces + piece] = k;
  v_pool[slot * row_pieces + piece] = v;
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
  int32_t row_pieces = hkv * d / 8;  // 8 bf16 per 16-byte piece
  int64_t total = n_tokens * row_pieces;
  int64_t blocks = (total + 255) / 256;
  if (blocks > INT32_MAX) return ra_fail(RA_EINVAL, "ra_store_kv: too many tokens");
  hipLaunchKernelGGL(store_kv_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, stream, slots,
                     static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new),
                     static_cast<uint4*>(k_pool), static_cast<uint4*>(v_pool), n_tokens, pool_slots,
                     row_pieces);
  return ra_check_launch("ra_store_kv");
}
