// Device-side helpers shared by the ltd_verify kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ltd_verify.h"

namespace ltd {

constexpr int kWave = 64;

// bf16 <-> f32.  Widening is exact; narrowing rounds to nearest even
// (finite inputs only: the kernels never produce NaN/Inf from finite data).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T>
__device__ __forceinline__ float load_f32(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_f32<float>(const float* p, int64_t i) {
  return p[i];
}
template <>
__device__ __forceinline__ float load_f32<uint16_t>(const uint16_t* p, int64_t i) {
  return bf16_to_f32(p[i]);
}

template <typename T>
__device__ __forceinline__ void store_f32(T* p, int64_t i, float v);
template <>
__device__ __forceinline__ void store_f32<float>(float* p, int64_t i, float v) {
  p[i] = v;
}
template <>
__device__ __forceinline__ void store_f32<uint16_t>(uint16_t* p, int64_t i, float v) {
  p[i] = f32_to_bf16(v);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Element offset of logical cache row `row` of sequence b, kv head g.
// Contiguous: [B][Hkv][kv_rows][d]; paged: [num_blocks][Hkv][kv_rows][d]
// with the block id from block_table[b][row / kv_rows].
__device__ __forceinline__ int64_t cache_row(const int32_t* __restrict__ block_table, int b, int g,
                                             int row, int Hkv, int d, int kv_rows,
                                             int max_blocks) {
  if (block_table == nullptr) return ((static_cast<int64_t>(b) * Hkv + g) * kv_rows + row) * d;
  const int64_t blk = block_table[static_cast<int64_t>(b) * max_blocks + row / kv_rows];
  return ((blk * Hkv + g) * kv_rows + (row % kv_rows)) * static_cast<int64_t>(d);
}

// A kernel launched with validate != 0 does nothing once the validation
// kernel that precedes it on the stream reported malformed data.
__device__ __forceinline__ bool halted(const int32_t* status) {
  return status != nullptr && *reinterpret_cast<const volatile int32_t*>(status) != 0;
}

}  // namespace ltd
