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

// Packs two fp32 into two bf16 (round to nearest even, v_cvt_pk_bf16_f32) in
// one 32-bit word: low half from a, high half from b.
__device__ __forceinline__ uint32_t ra_pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {static_cast<__bf16>(a), static_cast<__bf16>(b)};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float ra_bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float ra_bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xFFFF0000u); }

// Reductions over the four lanes that share (lane & 15): lanes l, l^16, l^32,
// l^48.  v_permlane32_swap / v_permlane16_swap exchange 32- / 16-lane halves
// of a register pair, so each step is one swap and one VALU op.
__device__ __forceinline__ float ra_max_across_rows(float v) {
  uint32_t u = __builtin_bit_cast(uint32_t, v);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  v = fmaxf(__builtin_bit_cast(float, static_cast<uint32_t>(r[0])), __builtin_bit_cast(float, static_cast<uint32_t>(r[1])));
  u = __builtin_bit_cast(uint32_t, v);
  r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, static_cast<uint32_t>(r[0])), __builtin_bit_cast(float, static_cast<uint32_t>(r[1])));
}
__device__ __forceinline__ float ra_sum_across_rows(float v) {
  uint32_t u = __builtin_bit_cast(uint32_t, v);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  v = __builtin_bit_cast(float, static_cast<uint32_t>(r[0])) + __builtin_bit_cast(float, static_cast<uint32_t>(r[1]));
  u = __builtin_bit_cast(uint32_t, v);
  r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __builtin_bit_cast(float, static_cast<uint32_t>(r[0])) + __builtin_bit_cast(float, static_cast<uint32_t>(r[1]));
}

inline int ra_check_launch(const char* who) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return ra_fail(RA_EHIP, std::string(who) + ": " + hipGetErrorString(e));
  return ra_ok();
}

inline bool ra_aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Compute units of the current device (cached per device; 256 if the query
// fails).  Defined in extend.hip.
int ra_device_cus();
