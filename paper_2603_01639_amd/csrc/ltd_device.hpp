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

// The value lane (l ^ kDist) holds, for every lane l of a wave64: gfx950's
// permlane swaps for distances 32 and 16 (swapping (v, v) hands the lower
// half of each pair the upper half's value in the second result and the
// upper half the lower half's in the first), DPP row rotations for 8 and 4
// (rotating a row of 16 by 8 is xor 8; by 4 and 12 give the two halves of
// xor 4), quad permutations for 2 and 1.  All VALU, no LDS.
template <int kCtrl>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return static_cast<uint32_t>(
      __builtin_amdgcn_mov_dpp(static_cast<int>(v), kCtrl, 0xF, 0xF, false));
}
template <int kDist>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v, int lane) {
  static_assert(kDist == 1 || kDist == 2 || kDist == 4 || kDist == 8 || kDist == 16 ||
                    kDist == 32,
                "");
  if constexpr (kDist == 32) {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return (lane & 32) ? r[0] : r[1];
  } else if constexpr (kDist == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return (lane & 16) ? r[0] : r[1];
  } else if constexpr (kDist == 8) {
    return dpp_mov<0x128>(v);  // row_ror:8
  } else if constexpr (kDist == 4) {
    const uint32_t a = dpp_mov<0x124>(v);  // row_ror:4
    const uint32_t b = dpp_mov<0x12C>(v);  // row_ror:12
    return (lane & 4) ? a : b;
  } else if constexpr (kDist == 2) {
    return dpp_mov<0x4E>(v);  // quad_perm [2,3,0,1]
  } else {
    return dpp_mov<0xB1>(v);  // quad_perm [1,0,3,2]
  }
}
template <int kDist>
__device__ __forceinline__ float lane_xor_f(float v, int lane) {
  return __uint_as_float(lane_xor<kDist>(__float_as_uint(v), lane));
}
template <int kDist>
__device__ __forceinline__ uint64_t lane_xor_u64(uint64_t v, int lane) {
  const uint32_t lo = lane_xor<kDist>(static_cast<uint32_t>(v), lane);
  const uint32_t hi = lane_xor<kDist>(static_cast<uint32_t>(v >> 32), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
// Maximum of a 64-bit key over the wave, in every lane.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v, int lane) {
  uint64_t o;
  o = lane_xor_u64<32>(v, lane); v = o > v ? o : v;
  o = lane_xor_u64<16>(v, lane); v = o > v ? o : v;
  o = lane_xor_u64<8>(v, lane);  v = o > v ? o : v;
  o = lane_xor_u64<4>(v, lane);  v = o > v ? o : v;
  o = lane_xor_u64<2>(v, lane);  v = o > v ? o : v;
  o = lane_xor_u64<1>(v, lane);  v = o > v ? o : v;
  return v;
}

// Wave-wide argmax over (key, index) pairs: the largest key, ties to the
// lowest index.  A 32-bit max over the wave, then a ballot of the lanes that
// hold it; only when several do, a 32-bit min over their indices.  Returns the
// winning index (uniform) and stores the winning key in *key_out.
__device__ __forceinline__ uint32_t wave_argmax(uint32_t key, uint32_t index, int lane,
                                                uint32_t* key_out) {
  uint32_t m = key;
  m = max(m, lane_xor<32>(m, lane));
  m = max(m, lane_xor<16>(m, lane));
  m = max(m, lane_xor<8>(m, lane));
  m = max(m, lane_xor<4>(m, lane));
  m = max(m, lane_xor<2>(m, lane));
  m = max(m, lane_xor<1>(m, lane));
  const uint64_t tied = __ballot(key == m);
  uint32_t idx;
  if (__popcll(tied) == 1) {
    idx = static_cast<uint32_t>(
        __builtin_amdgcn_readlane(static_cast<int>(index), __ffsll(static_cast<long long>(tied)) - 1));
  } else {
    uint32_t c = key == m ? index : 0xFFFFFFFFu;
    c = min(c, lane_xor<32>(c, lane));
    c = min(c, lane_xor<16>(c, lane));
    c = min(c, lane_xor<8>(c, lane));
    c = min(c, lane_xor<4>(c, lane));
    c = min(c, lane_xor<2>(c, lane));
    c = min(c, lane_xor<1>(c, lane));
    idx = c;
  }
  *key_out = m;
  return idx;
}

// A kernel launched with validate != 0 does nothing once the validation
// kernel that precedes it on the stream reported malformed data.
__device__ __forceinline__ bool halted(const int32_t* status) {
  return status != nullptr && *reinterpret_cast<const volatile int32_t*>(status) != 0;
}

}  // namespace ltd
