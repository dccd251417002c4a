// Per-thread error text behind ra_last_error().
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <new>
#include <string>

#include <hip/hip_runtime.h>

#include "radixattn.h"

int ra_fail(int code, const std::string& msg);
int ra_ok();

// Runs a host entry point's body so that no C++ exception crosses the C ABI:
// running out of host memory becomes RA_ENOMEM, anything else RA_EINVAL.  A
// tree or router whose operation failed this way may be left part-way through
// the operation; the caller should destroy it.
template <class F>
int ra_guard(const char* who, F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    try {
      return ra_fail(RA_ENOMEM, std::string(who) + ": out of host memory");
    } catch (...) {
      return RA_ENOMEM;
    }
  } catch (...) {
    try {
      return ra_fail(RA_EINVAL, std::string(who) + ": internal error");
    } catch (...) {
      return RA_EINVAL;
    }
  }
}

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

int ra_decode_shared_validate(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                              const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int32_t batch,
                              int32_t hq, int32_t hkv, int32_t d, float scale, const int32_t* plan, int64_t plan_len,
                              int32_t n_items, int32_t n_member_entries, int32_t n_parts, int32_t members_per_item,
                              const void* workspace, size_t workspace_bytes, const void* out);

// True while ra_set_debug_checks(1) is in force: the attention entry points
// then run ra_check_batch on their batch before launching.
bool ra_debug_checks_enabled();
