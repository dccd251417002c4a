// Per-thread error text behind ra_last_error().
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>

#include <hip/hip_runtime.h>

#include "radixattn.h"

int ra_fail(int code, const std::string& msg);
int ra_ok();

// Argument checks of the attention entry points (no launch), shared with the
// mixed-batch call so that it can reject a bad batch before queuing anything.
int ra_extend_validate(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                       const void* k_pool, const void* v_pool, int64_t pool_slots, const int32_t* req_to_token,
                       int64_t rtt_rows, int64_t rtt_stride, const int32_t* req_pool_idx,
                       const int32_t* prefix_lens, const int32_t* extend_lens, const int32_t* extend_start,
                       int32_t batch, int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                       void* out);
int ra_decode_validate(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                       const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, const int32_t* req_pool_idx,
                       const int32_t* seq_lens, int32_t batch, int32_t max_seq_len, int32_t hq, int32_t hkv, int32_t d,
                       float scale, int32_t num_splits, const void* workspace, size_t workspace_bytes,
                       const void* out);

