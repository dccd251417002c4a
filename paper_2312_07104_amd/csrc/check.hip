// Batch validation on the device (ra_check_batch, ra_set_debug_checks).
//
// The attention kernels keep every access in bounds by clamping: a table row
// outside [0, rtt_rows) reads row 0, a length above its bound is cut, a slot
// outside the pool reads the last slot.  A caller bug therefore gives
// plausible but wrong output.  This check reads the same device arrays the
// kernels read and reports the first bad entry instead: request order first,
// then the kind of fault, then the position.

#include <atomic>
#include <mutex>

#include "device_common.h"

// The check's result word, one per device.  In host code the name is a
// host-side stand-in: the kernels receive the address hipGetSymbolAddress
// reports for the current device.
static __device__ unsigned long long check_result;

namespace {

enum : uint32_t {
  kBadRow = 1,        // req_pool_idx outside [0, rtt_rows)
  kBadPrefix = 2,     // prefix_lens outside [0, rtt_stride]
  kBadExtend = 3,     // extend_lens outside [0, max_extend_len]
  kBadStart = 4,      // extend_start / extend_lens outside [0, total_tokens]
  kBadSeqLen = 5,     // seq_lens outside [1, max_seq_len]
  kBadSlot = 6,       // a slot the request reads outside [0, pool_slots)
};

constexpr uint64_t kNoFault = ~uint64_t{0};

__device__ __forceinline__ uint64_t fault_key(int64_t req, uint32_t code, int64_t pos) {
  const uint64_t p = static_cast<uint64_t>(pos < 0 ? 0 : (pos > 0x7FFFFFF ? 0x7FFFFFF : pos));
  return (static_cast<uint64_t>(req) << 32) | (static_cast<uint64_t>(code) << 27) | p;
}

__global__ void check_reset_kernel(unsigned long long* result) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *result = kNoFault;
}

// One work-group per request.  Extend (prefix_lens != nullptr): the slots of
// positions 0 .. P - 1 (new positions come from k_new / v_new).  Decode: the
// slots of positions 0 .. L - 1.  Every read is inside the arrays whatever
// the values: the slot scan runs only for a row inside the table and over at
// most rtt_stride positions.
__global__ __launch_bounds__(256) void check_batch_kernel(
    const int32_t* __restrict__ rtt, int64_t rtt_rows, int64_t rtt_stride, int64_t pool_slots,
    const int32_t* __restrict__ req_pool_idx, const int32_t* __restrict__ prefix_lens,
    const int32_t* __restrict__ extend_lens, const int32_t* __restrict__ extend_start, int64_t total_tokens,
    int32_t max_extend_len, const int32_t* __restrict__ seq_lens, int32_t max_seq_len,
    unsigned long long* result) {
  const int64_t b = blockIdx.x;
  const int64_t row = req_pool_idx[b];
  int64_t n;  // positions whose slots the request reads
  if (threadIdx.x == 0) {
    uint64_t key = kNoFault;
    if (row < 0 || row >= rtt_rows) key = fault_key(b, kBadRow, 0);
    if (prefix_lens) {
      const int64_t P = prefix_lens[b], E = extend_lens[b], st = extend_start[b];
      if (P < 0 || P > rtt_stride) key = min(key, fault_key(b, kBadPrefix, 0));
      if (E < 0 || E > max_extend_len) key = min(key, fault_key(b, kBadExtend, 0));
      if (st < 0 || E < 0 || st + E > total_tokens) key = min(key, fault_key(b, kBadStart, 0));
    } else {
      const int64_t L = seq_lens[b];
      if (L < 1 || L > max_seq_len) key = min(key, fault_key(b, kBadSeqLen, 0));
    }
    if (key != kNoFault) atomicMin(result, static_cast<unsigned long long>(key));
  }
  if (row < 0 || row >= rtt_rows) return;
  n = prefix_lens ? static_cast<int64_t>(prefix_lens[b]) : static_cast<int64_t>(seq_lens[b]);
  n = n < 0 ? 0 : (n > rtt_stride ? rtt_stride : n);
  if (!prefix_lens && n > max_seq_len) n = max_seq_len;
  const int32_t* trow = rtt + row * rtt_stride;
  int64_t first = -1;
  for (int64_t j = threadIdx.x; j < n; j += blockDim.x) {
    const int64_t s = trow[j];
    if (s < 0 || s >= pool_slots) {
      first = j;
      break;
    }
  }
  if (first >= 0) atomicMin(result, static_cast<unsigned long long>(fault_key(b, kBadSlot, first)));
}

std::mutex g_check_mu;
void* g_check_ptr[64] = {};
std::atomic<int> g_debug_checks{0};

// Device address of this device's result word, looked up once per device.
int result_for_current_device(unsigned long long** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
    return ra_fail(RA_EHIP, "ra_check_batch: no usable current device");
  if (!g_check_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(check_result));
    if (e != hipSuccess || ptr == nullptr)
      return ra_fail(RA_EHIP, std::string("ra_check_batch: hipGetSymbolAddress: ") + hipGetErrorString(e));
    g_check_ptr[dev] = ptr;
  }
  *out = static_cast<unsigned long long*>(g_check_ptr[dev]);
  return RA_OK;
}

const char* fault_name(uint32_t code) {
  switch (code) {
    case kBadRow: return "req_pool_idx outside [0, rtt_rows)";
    case kBadPrefix: return "prefix_lens outside [0, rtt_stride]";
    case kBadExtend: return "extend_lens outside [0, max_extend_len]";
    case kBadStart: return "extend_start + extend_lens outside [0, total_tokens]";
    case kBadSeqLen: return "seq_lens outside [1, max_seq_len]";
    case kBadSlot: return "slot outside [0, pool_slots)";
    default: return "unknown";
  }
}

}  // namespace

extern "C" int ra_set_debug_checks(int32_t enable) {
  g_debug_checks.store(enable ? 1 : 0, std::memory_order_relaxed);
  return RA_OK;
}

bool ra_debug_checks_enabled() { return g_debug_checks.load(std::memory_order_relaxed) != 0; }

extern "C" int ra_check_batch(const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int64_t pool_slots,
                              const int32_t* req_pool_idx, int32_t batch, const int32_t* prefix_lens,
                              const int32_t* extend_lens, const int32_t* extend_start, int64_t total_tokens,
                              int32_t max_extend_len, const int32_t* seq_lens, int32_t max_seq_len,
                              hipStream_t stream) {
  if (batch < 0 || rtt_rows <= 0 || rtt_stride <= 0 || pool_slots <= 0)
    return ra_fail(RA_EINVAL, "ra_check_batch: bad sizes");
  const bool ext = prefix_lens != nullptr;
  if (ext ? (!extend_lens || !extend_start || seq_lens) : !seq_lens)
    return ra_fail(RA_EINVAL, "ra_check_batch: pass prefix_lens, extend_lens and extend_start (extend) or seq_lens "
                              "(decode)");
  if (batch == 0) return ra_ok();
  if (!req_to_token || !req_pool_idx) return ra_fail(RA_EINVAL, "ra_check_batch: NULL pointer");
  std::lock_guard<std::mutex> lock(g_check_mu);
  unsigned long long* res = nullptr;
  int st = result_for_current_device(&res);
  if (st != RA_OK) return st;
  hipLaunchKernelGGL(check_reset_kernel, dim3(1), dim3(64), 0, stream, res);
  hipLaunchKernelGGL(check_batch_kernel, dim3(static_cast<uint32_t>(batch)), dim3(256), 0, stream, req_to_token,
                     rtt_rows, rtt_stride, pool_slots, req_pool_idx, prefix_lens, extend_lens, extend_start,
                     total_tokens, max_extend_len, seq_lens, max_seq_len, res);
  st = ra_check_launch("ra_check_batch");
  if (st != RA_OK) return st;
  unsigned long long host = kNoFault;
  if (hipMemcpyAsync(&host, res, sizeof(host), hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return ra_fail(RA_EHIP, "ra_check_batch: cannot read the result");
  if (host == kNoFault) return ra_ok();
  const int64_t req = static_cast<int64_t>(host >> 32);
  const uint32_t code = static_cast<uint32_t>((host >> 27) & 0x1F);
  const int64_t pos = static_cast<int64_t>(host & 0x7FFFFFF);
  std::string msg = std::string("ra_check_batch: request ") + std::to_string(req) + ": " + fault_name(code);
  if (code == kBadSlot) msg += " at position " + std::to_string(pos);
  return ra_fail(RA_EINVAL, msg);
}
