// Machine-peak microbenchmarks for the roofline report (bench.py --peaks):
// the HBM read bandwidth a streaming kernel reaches, the bandwidth of random
// 256-byte row gathers (the access pattern of attention over a pool of
// one-token pages, also in the decode kernels' own tile pattern), and the
// bf16 rate of a loop of matrix-core instructions.
// They compute no attention; each folds what it reads into one word per
// thread so the compiler keeps every load.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

typedef __bf16 pk_bf16x8 __attribute__((ext_vector_type(8)));
typedef float pk_f32x4 __attribute__((ext_vector_type(4)));
typedef float pk_f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint32_t pk_fold(uint4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

// Streaming read of n16 16-byte words, grid-stride, four loads in flight per
// thread.
__global__ __launch_bounds__(256) void pk_read_kernel(const uint4* __restrict__ src, int64_t n16,
                                                      uint32_t* __restrict__ sink) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= pk_fold(a) ^ pk_fold(b) ^ pk_fold(c) ^ pk_fold(d);
  }
  for (; i < n16; i += stride) acc ^= pk_fold(src[i]);
  sink[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = acc;
}

// Random row gather: row r is the 256-byte head row (r % heads) of slot
// slots[r] in a pool of slot_bytes-byte slots.  Sixteen lanes read one row
// (16 bytes each), so a wave instruction reads four rows; each wave walks its
// own run of rows, sixteen rows (four instructions) in flight.
__global__ __launch_bounds__(256) void pk_gather_kernel(const unsigned char* __restrict__ pool,
                                                        const int32_t* __restrict__ slots, int64_t n_rows,
                                                        int32_t heads, int32_t slot_bytes,
                                                        uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) >> 6;
  const int64_t n_waves = static_cast<int64_t>(gridDim.x) * 4;
  const int64_t per_wave = (n_rows + n_waves - 1) / n_waves;
  const int64_t r0 = wave * per_wave;
  const int64_t r1 = r0 + per_wave < n_rows ? r0 + per_wave : n_rows;
  uint32_t acc = 0;
  for (int64_t r = r0; r < r1; r += 16) {
    uint4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      int64_t row = r + 4 * k + (lane >> 4);
      row = row < r1 ? row : r1 - 1;
      const int64_t off = static_cast<int64_t>(slots[row]) * slot_bytes + (row % heads) * 256 + (lane & 15) * 16;
      v[k] = *reinterpret_cast<const uint4*>(pool + off);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) acc ^= pk_fold(v[k]);
  }
  sink[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = acc;
}

// Gather in the decode kernels' own pattern: 32-row tiles of one head's K row
// and V row (256 bytes each, two pools of slot_bytes-byte slots), each wave
// instruction reading 64 bytes of 16 rows (lane: row lane & 15 of a 16-row
// half, 16-byte piece lane >> 4 of a 64-byte quarter); a tile is 8 K and 8 V
// instructions (16 KB), two tiles in flight per wave, one wave per SIMD.  The
// slot indices of a tile (one per lane of the first 32) are loaded two tiles
// ahead, after the loads of the tile before, and spread with a lane shuffle.
// Wave w walks tiles w * tiles .. w * tiles + tiles - 1 of the row list.
__global__ __launch_bounds__(256) void pk_gather_kv_kernel(const unsigned char* __restrict__ kpool,
                                                           const unsigned char* __restrict__ vpool,
                                                           const int32_t* __restrict__ slots, int32_t tiles,
                                                           int32_t slot_bytes, uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int head = static_cast<int>(wave & 7);
  uint4 kb[2][2][4], vb[2][2][4];
  int32_t ib[2];
  uint32_t acc = 0;
  auto idx_of = [&](int t) { return slots[(wave * tiles + min(t, tiles - 1)) * 32 + (lane & 31)]; };
  auto load = [&](int j, int32_t idx) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t off = static_cast<int64_t>(__shfl(idx, (lane & 15) + 16 * h)) * slot_bytes + head * 256 +
                          16 * (lane >> 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        kb[j][h][q] = *reinterpret_cast<const uint4*>(kpool + off + 64 * q);
        vb[j][h][q] = *reinterpret_cast<const uint4*>(vpool + off + 64 * q);
      }
    }
  };
  ib[0] = idx_of(0);
  ib[1] = idx_of(1);
  load(0, ib[0]);
  load(1, ib[1]);
  ib[0] = idx_of(2);
  ib[1] = idx_of(3);
  for (int t = 0; t < tiles; t += 2) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc ^= pk_fold(kb[j][h][q]) ^ pk_fold(vb[j][h][q]);
      if (t + j + 2 < tiles) load(j, ib[j]);
      ib[j] = idx_of(t + j + 4);
    }
  }
  sink[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = acc;
}

// Matrix-core loop: eight independent accumulator chains per wave of bf16
// MFMAs on register operands, one wave per SIMD (one 256-thread work-group
// per CU), so each wave's cycles are its SIMD's.  SHAPE 16: 16x16x32
// (16384 flops per instruction); SHAPE 32: 32x32x16 (32768).  Lane 0 of
// each wave records the loop's shader-clock cycles and real-time ticks.
template <int SHAPE>
__global__ __launch_bounds__(256) void pk_mfma_kernel(int32_t iters, float* __restrict__ sink,
                                                      uint64_t* __restrict__ clocks) {
  typedef typename std::conditional<SHAPE == 16, pk_f32x4, pk_f32x16>::type acc_t;
  const int lane = threadIdx.x & 63;
  pk_bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<__bf16>(0.001f * (lane + i));
    b[i] = static_cast<__bf16>(0.002f * (lane - i));
  }
  acc_t c[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) c[k] = acc_t{};
  const uint64_t t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
    // inline assembly keeps each accumulator in place (the compiler's own
    // MFMAs here came with register moves between them)
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if constexpr (SHAPE == 16) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c[k]) : "v"(a), "v"(b));
      else asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c[k]) : "v"(a), "v"(b));
    }
  }
  // wait states before the VALU reads the last MFMAs' results
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  float r = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) r += c[k][0];
  sink[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = r;
  const uint64_t t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  if (lane == 0) {
    const int64_t w = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) >> 6;
    clocks[2 * w] = t1 - t0;      // shader clock cycles of this wave's loop
    clocks[2 * w + 1] = r1 - r0;  // 100 MHz real-time ticks
  }
}

extern "C" int pk_read(const void* src, int64_t bytes, void* sink, int32_t blocks, hipStream_t s) {
  hipLaunchKernelGGL(pk_read_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const uint4*>(src), bytes / 16,
                     static_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int pk_gather(const void* pool, const int32_t* slots, int64_t n_rows, int32_t heads, int32_t slot_bytes,
                         void* sink, int32_t blocks, hipStream_t s) {
  hipLaunchKernelGGL(pk_gather_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const unsigned char*>(pool), slots,
                     n_rows, heads, slot_bytes, static_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// tiles must be even; slots holds blocks * 4 * tiles * 32 entries in [0, pool rows).
extern "C" int pk_gather_kv(const void* kpool, const void* vpool, const int32_t* slots, int32_t tiles,
                            int32_t slot_bytes, void* sink, int32_t blocks, hipStream_t s) {
  if (tiles < 2 || tiles % 2 != 0 || slot_bytes < 8 * 256) return -2;
  hipLaunchKernelGGL(pk_gather_kv_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const unsigned char*>(kpool),
                     static_cast<const unsigned char*>(vpool), slots, tiles, slot_bytes, static_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int pk_mfma(int32_t shape, int32_t iters, void* sink, void* clocks, int32_t blocks, hipStream_t s) {
  if (shape == 16)
    hipLaunchKernelGGL(pk_mfma_kernel<16>, dim3(blocks), dim3(256), 0, s, iters, static_cast<float*>(sink),
                       static_cast<uint64_t*>(clocks));
  else
    hipLaunchKernelGGL(pk_mfma_kernel<32>, dim3(blocks), dim3(256), 0, s, iters, static_cast<float*>(sink),
                       static_cast<uint64_t*>(clocks));
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
