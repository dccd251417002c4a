// Device-side helpers shared by the gfx950 kernels of this library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "ra_error.h"

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// log2(e): scores are kept in the base-2 domain so exponentials are exp2.
#define RA_LOG2E 1.4426950408889634f

__device__ __forceinline__ float ra_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Packs two fp32 into two bf16 (round to nearest even) in one 32-bit word:
// low half from a, high half from b.
__device__ __forceinline__ uint32_t ra_pack_bf16x2(float a, float b) {
  uint32_t ua = __builtin_bit_cast(uint32_t, a);
  uint32_t ub = __builtin_bit_cast(uint32_t, b);
  ua = (ua + 0x7FFFu + ((ua >> 16) & 1u)) >> 16;
  ub = (ub + 0x7FFFu + ((ub >> 16) & 1u)) & 0xFFFF0000u;
  return ua | ub;
}

__device__ __forceinline__ float ra_bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float ra_bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xFFFF0000u); }

// Maximum over the four lanes that share (lane & 15): lanes l, l^16, l^32, l^48.
__device__ __forceinline__ float ra_max_across_rows(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}
__device__ __forceinline__ float ra_sum_across_rows(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

inline int ra_check_launch(const char* who) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return ra_fail(RA_EHIP, std::string(who) + ": " + hipGetErrorString(e));
  return ra_ok();
}

inline bool ra_aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
