// Device helpers shared by the gfx950 kernels: BF16 conversion, wave64 reductions, and the
// LDS layout that GEMV kernels use for their input vector.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tasp {

constexpr int kWave = 64;
constexpr int kBlock = 256;               // 4 waves per workgroup
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// float32 -> BF16, round to nearest even (inputs are finite on every path that calls it).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}

// Block-wide sum over 256 threads; `red` is 4 floats of LDS. Every thread gets the total.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// GEMV input staging. A wave reads a weight row in 1 KiB chunks, lane l taking the 16 bytes at
// chunk offset 16 l. For INT8 rows the lane's 16 columns are k = c*1024 + 16 l + j (j < 16); the
// vector element k is stored at float index ((c*4 + j/4)*64 + l)*4 + j%4, so the lane's four
// float4 reads of a chunk hit consecutive 16-byte slots across the wave.
__device__ __forceinline__ int xs_slot_i8(int k) {
  const int c = k >> 10, l = (k >> 4) & 63, j = k & 15;
  return ((((c << 2) + (j >> 2)) << 6) + l) * 4 + (j & 3);
}
// For BF16 rows a 16-byte lane load holds 8 columns: k = c*512 + 8 l + j (j < 8).
__device__ __forceinline__ int xs_slot_bf16(int k) {
  const int c = k >> 9, l = (k >> 3) & 63, j = k & 7;
  return ((((c << 1) + (j >> 2)) << 6) + l) * 4 + (j & 3);
}

// Loads that must observe other workgroups' stores made visible by a fence + atomic.
__device__ __forceinline__ float ld_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace tasp
