// GPU version of the content-addressed value generator (workload/contentgen.py):
// the same SplitMix64 counter stream, Irwin-Hall sum of twelve 16-bit
// uniforms and bf16 round-to-nearest-even, bit for bit.  Input generation
// only; it holds no attention or radix-tree arithmetic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#define WG_GAMMA 0x9E3779B97F4A7C15ULL
#define WG_STREAM_SALT 0xD1B54A32D192ED03ULL

__device__ __forceinline__ uint64_t wg_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

// out[rows[p] * n_elem + e] (or out[p * n_elem + e] when rows is NULL) =
// bf16 bits of value(hash p, stream, element e) * 2^scale_pow2.
__global__ void wg_values_kernel(const uint64_t* __restrict__ hashes, const int64_t* __restrict__ rows,
                                 int64_t n, int32_t stream, int32_t n_elem, float mult,
                                 uint16_t* __restrict__ out) {
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n * n_elem) return;
  int64_t p = i / n_elem;
  int32_t e = static_cast<int32_t>(i - p * n_elem);
  uint64_t key = wg_mix64(hashes[p] ^ (static_cast<uint64_t>(stream) * WG_STREAM_SALT));
  int64_t acc = 0;
#pragma unroll
  for (uint64_t k = 0; k < 3; ++k) {
    uint64_t w = wg_mix64(key + (3ull * static_cast<uint64_t>(e) + k + 1ull) * WG_GAMMA);
    acc += static_cast<int64_t>(w & 0xFFFF) + static_cast<int64_t>((w >> 16) & 0xFFFF) +
           static_cast<int64_t>((w >> 32) & 0xFFFF) + static_cast<int64_t>(w >> 48);
  }
  float z = static_cast<float>(static_cast<int32_t>(acc - 393210)) * (1.0f / 65536.0f) * mult;
  uint32_t b = __builtin_bit_cast(uint32_t, z);
  uint16_t h = static_cast<uint16_t>((static_cast<uint64_t>(b) + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
  int64_t r = rows ? rows[p] : p;
  out[r * n_elem + e] = h;
}

extern "C" int wg_values(const uint64_t* hashes, const int64_t* rows, int64_t n, int32_t stream, int32_t n_elem,
                         int32_t scale_pow2, void* out, hipStream_t s) {
  if (n <= 0) return 0;
  int64_t total = n * n_elem;
  int64_t blocks = (total + 255) / 256;
  float mult = ldexpf(1.0f, scale_pow2);
  hipLaunchKernelGGL(wg_values_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, s, hashes, rows, n,
                     stream, n_elem, mult, static_cast<uint16_t*>(out));
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
