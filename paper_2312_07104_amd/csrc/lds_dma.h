// Direct global -> LDS copies and explicit vector-memory waits, shared by the
// attention kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

__device__ __forceinline__ uint4 ra_ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ uint32_t ra_lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}

// global_load_lds_dwordx4 / _dword: lane i's 16 (4) bytes land at
// lds_base + 16 i (4 i); the source address is per lane.  Issued from inline
// assembly because the compiler would otherwise wait for every outstanding
// copy before each later LDS read; callers wait with ra_wait_vmcnt.
__device__ __forceinline__ void ra_dma16(const void* g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g),
               "s"(__builtin_amdgcn_readfirstlane(lds_base))
               : "memory");
}
__device__ __forceinline__ void ra_dma4(const void* g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(g),
               "s"(__builtin_amdgcn_readfirstlane(lds_base))
               : "memory");
}

// s_waitcnt vmcnt(n) with expcnt / lgkmcnt left unconstrained (gfx9 layout).
// vmcnt counts this wave's outstanding vector-memory loads, which complete in
// issue order.
template <int N>
__device__ __forceinline__ void ra_wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

// Layout of a 64-row K or V tile staged by the extend kernels: [piece group
// pg = D/32][row 0..63][4 pieces of 16 B]; the 16-byte piece q of row r sits
// at physical slot q ^ ra_kv_swz(r), ra_kv_swz(r) = (bit 3 of r) << 1.
// Bank model of the gfx950 LDS (64 banks of 4 bytes, measured with the
// SQ_LDS_BANK_CONFLICT counter): ds_read_b128 is served in four cycles of 16
// lanes, the lane groups being the 8-lane blocks {0-7, 24-31}, {8-15, 16-23},
// {32-39, 56-63} and {40-47, 48-55}; ds_read_b64 and ds_read_b64_tr_b16 in
// two cycles of 32 lanes (0-31, 32-63).  K operand reads (rows
// 8 (c >> 2) + (c & 3) + const, piece g4 = lane >> 4) and V^T transposed
// reads (rows 8 g4 + (c >> 2) + const, piece pair per lane) then hit 64
// distinct banks per cycle, and the direct-to-LDS copies write 1 KB runs.
// The swizzle ignores row bits 2 and 5, so every operand read is one
// per-lane offset plus a compile-time immediate.
__device__ __forceinline__ int ra_kv_swz(int r) { return ((r >> 3) & 1) << 1; }
