// Mixed continuous batch: extend on the caller's stream, decode on a
// companion stream, joined with events, so the MFMA-bound and the HBM-bound
// kernel share the chip instead of running back to back.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <unordered_map>

#include "ra_error.h"
#include "radixattn.h"

namespace {

struct Companion {
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr;
  hipEvent_t join = nullptr;
};

std::mutex g_mu;
std::unordered_map<int, Companion> g_companions;

int companion_for(int device, Companion** out) {
  auto it = g_companions.find(device);
  if (it != g_companions.end()) {
    *out = &it->second;
    return RA_OK;
  }
  Companion c;
  if (hipStreamCreateWithFlags(&c.stream, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c.fork, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c.join, hipEventDisableTiming) != hipSuccess)
    return ra_fail(RA_EHIP, "ra_mixed_attention: cannot create the companion stream");
  *out = &g_companions.emplace(device, c).first->second;
  return RA_OK;
}

// Queues decode(companion stream) beside extend(stream): the companion waits
// for the work already on the caller's stream, and the caller's stream waits
// for the companion before anything queued after this call.
template <class Decode, class Extend>
int run_beside(hipStream_t stream, Decode&& decode, Extend&& extend) {
  std::lock_guard<std::mutex> lock(g_mu);
  int device = 0;
  if (hipGetDevice(&device) != hipSuccess) return ra_fail(RA_EHIP, "ra_mixed_attention: hipGetDevice failed");
  Companion* comp = nullptr;
  int st = companion_for(device, &comp);
  if (st != RA_OK) return st;
  if (hipEventRecord(comp->fork, stream) != hipSuccess || hipStreamWaitEvent(comp->stream, comp->fork, 0) != hipSuccess)
    return ra_fail(RA_EHIP, "ra_mixed_attention: cannot fork the companion stream");
  st = decode(comp->stream);
  if (st == RA_OK) st = extend(stream);
  // Join even after a failed launch so the caller's stream never runs ahead
  // of work already queued on the companion.
  if (hipEventRecord(comp->join, comp->stream) != hipSuccess || hipStreamWaitEvent(stream, comp->join, 0) != hipSuccess)
    return ra_fail(RA_EHIP, "ra_mixed_attention: cannot join the companion stream");
  return st;
}

}  // namespace

extern "C" int ra_mixed_attention(const void* q_ext, const void* k_new, const void* v_new, int64_t total_tokens,
                                  const int32_t* req_pool_idx_ext, const int32_t* prefix_lens,
                                  const int32_t* extend_lens, const int32_t* extend_start, int32_t n_ext,
                                  int32_t max_extend_len, void* out_ext, const void* q_dec,
                                  const int32_t* req_pool_idx_dec, const int32_t* seq_lens, int32_t n_dec,
                                  int32_t max_seq_len, int32_t num_splits, void* workspace, size_t workspace_bytes,
                                  void* out_dec, const void* k_pool, const void* v_pool, int64_t pool_slots,
                                  const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int32_t hq,
                                  int32_t hkv, int32_t d, float scale, hipStream_t stream) {
  if (n_ext < 0 || n_dec < 0) return ra_fail(RA_EINVAL, "ra_mixed_attention: negative batch");
  if (n_dec == 0) {
    return ra_extend_attention(q_ext, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows,
                               rtt_stride, req_pool_idx_ext, prefix_lens, extend_lens, extend_start, n_ext,
                               max_extend_len, hq, hkv, d, scale, out_ext, stream);
  }
  if (n_ext == 0 || max_extend_len == 0 || total_tokens == 0) {
    return ra_decode_attention(q_dec, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride,
                               req_pool_idx_dec, seq_lens, n_dec, max_seq_len, hq, hkv, d, scale, num_splits,
                               workspace, workspace_bytes, out_dec, stream);
  }
  // Check both halves before queuing either, so a failing call changes nothing.
  int st = ra_extend_validate(q_ext, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows,
                              rtt_stride, req_pool_idx_ext, prefix_lens, extend_lens, extend_start, n_ext,
                              max_extend_len, hq, hkv, d, scale, out_ext);
  if (st == RA_OK)
    st = ra_decode_validate(q_dec, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride, req_pool_idx_dec,
                            seq_lens, n_dec, max_seq_len, hq, hkv, d, scale, num_splits, workspace, workspace_bytes,
                            out_dec);
  if (st != RA_OK) return st;
  if (ra_debug_checks_enabled()) {
    st = ra_check_batch(req_to_token, rtt_rows, rtt_stride, pool_slots, req_pool_idx_ext, n_ext, prefix_lens,
                        extend_lens, extend_start, total_tokens, max_extend_len, nullptr, 0, stream);
    if (st == RA_OK)
      st = ra_check_batch(req_to_token, rtt_rows, rtt_stride, pool_slots, req_pool_idx_dec, n_dec, nullptr, nullptr,
                          nullptr, 0, 0, seq_lens, max_seq_len > 0 ? max_seq_len : static_cast<int32_t>(
                              std::min<int64_t>(rtt_stride, INT32_MAX)), stream);
    if (st != RA_OK) return st;
  }
  return run_beside(
      stream,
      [&](hipStream_t s) {
        return ra_decode_attention(q_dec, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride,
                                   req_pool_idx_dec, seq_lens, n_dec, max_seq_len, hq, hkv, d, scale, num_splits,
                                   workspace, workspace_bytes, out_dec, s);
      },
      [&](hipStream_t s) {
        return ra_extend_attention(q_ext, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token,
                                   rtt_rows, rtt_stride, req_pool_idx_ext, prefix_lens, extend_lens, extend_start,
                                   n_ext, max_extend_len, hq, hkv, d, scale, out_ext, s);
      });
}

extern "C" int ra_mixed_attention_shared(const void* q_ext, const void* k_new, const void* v_new,
                                         int64_t total_tokens, const int32_t* req_pool_idx_ext,
                                         const int32_t* prefix_lens, const int32_t* extend_lens,
                                         const int32_t* extend_start, int32_t n_ext, int32_t max_extend_len,
                                         void* out_ext, const void* q_dec, int32_t n_dec, const int32_t* plan,
                                         int64_t plan_len, int32_t n_items, int32_t n_member_entries,
                                         int32_t n_parts, int32_t members_per_item, void* workspace,
                                         size_t workspace_bytes, void* out_dec, const void* k_pool,
                                         const void* v_pool, int64_t pool_slots, const int32_t* req_to_token,
                                         int64_t rtt_rows, int64_t rtt_stride, int32_t hq, int32_t hkv, int32_t d,
                                         float scale, hipStream_t stream) {
  if (n_ext < 0 || n_dec < 0) return ra_fail(RA_EINVAL, "ra_mixed_attention_shared: negative batch");
  auto decode = [&](hipStream_t s) {
    return ra_decode_attention_shared(q_dec, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride, n_dec,
                                      hq, hkv, d, scale, plan, plan_len, n_items, n_member_entries, n_parts,
                                      members_per_item, workspace, workspace_bytes, out_dec, s);
  };
  auto extend = [&](hipStream_t s) {
    return ra_extend_attention(q_ext, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows,
                               rtt_stride, req_pool_idx_ext, prefix_lens, extend_lens, extend_start, n_ext,
                               max_extend_len, hq, hkv, d, scale, out_ext, s);
  };
  if (n_dec == 0 || n_items == 0) return extend(stream);
  if (n_ext == 0 || max_extend_len == 0 || total_tokens == 0) return decode(stream);
  // Check both halves before queuing either, so a failing call changes nothing.
  int st = ra_extend_validate(q_ext, k_new, v_new, total_tokens, k_pool, v_pool, pool_slots, req_to_token, rtt_rows,
                              rtt_stride, req_pool_idx_ext, prefix_lens, extend_lens, extend_start, n_ext,
                              max_extend_len, hq, hkv, d, scale, out_ext);
  if (st == RA_OK)
    st = ra_decode_shared_validate(q_dec, k_pool, v_pool, pool_slots, req_to_token, rtt_rows, rtt_stride, n_dec, hq,
                                   hkv, d, scale, plan, plan_len, n_items, n_member_entries, n_parts,
                                   members_per_item, workspace, workspace_bytes, out_dec);
  if (st != RA_OK) return st;
  if (ra_debug_checks_enabled()) {
    st = ra_check_batch(req_to_token, rtt_rows, rtt_stride, pool_slots, req_pool_idx_ext, n_ext, prefix_lens,
                        extend_lens, extend_start, total_tokens, max_extend_len, nullptr, 0, stream);
    if (st != RA_OK) return st;
  }
  return run_beside(stream, decode, extend);
}
