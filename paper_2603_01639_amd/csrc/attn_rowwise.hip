// Tree attention on the vector ALUs, the fp32 path: one workgroup of four
// waves per (sequence, node, kv head) handles the G query heads of that kv
// head, four at a time (one a wave).  Keys are visited in tiles of 64, each
// tile's K and V rows staged in LDS by the whole workgroup with coalesced
// 16-byte loads, so the G heads (and, per pass, the four waves) share one
// read of them.  Scores take one key per lane (a dot product over an LDS row
// padded against bank conflicts); an online (running-max) softmax per head;
// the value accumulation takes one or two head dimensions per lane.
//
// The visible key set of node i is the prefix [0, P_b) plus the tree rows of
// the node's root path (arXiv 2603.01639, section 3.2: the tree attention
// mask shows each candidate its ancestors only).
#include "ltd_device.hpp"
#include "ltd_launch.hpp"
#include "tree_walk.hpp"

namespace ltd {
namespace {

constexpr int kTileKeys = 64;
constexpr int kVecWaves = 4;
constexpr int kVecThreads = kVecWaves * kWave;
constexpr int kMaxD = 128;
constexpr int kPieces = kTileKeys * kMaxD / 4 / kVecThreads;  // 16-byte pieces a thread loads

// Wave-wide reductions without the LDS crossbar: within each 16-lane row by
// DPP (quad swaps, then the half-row and row mirrors: every lane ends with its
// row's total), then across rows with v_permlane16_swap and
// v_permlane32_swap of the value with itself (their two results hold the
// other row, or half, in every lane).
template <int kCtrl>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), kCtrl,
                                                               0xF, 0xF, false));
}
template <class Op>
__device__ __forceinline__ float wave_reduce(float v, Op op) {
  v = op(v, dpp<0xB1>(v));   // quad_perm [1, 0, 3, 2]
  v = op(v, dpp<0x4E>(v));   // quad_perm [2, 3, 0, 1]
  v = op(v, dpp<0x141>(v));  // row_half_mirror
  v = op(v, dpp<0x140>(v));  // row_mirror
  uint32_t u = __builtin_bit_cast(uint32_t, v);
  const auto r16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  // (the halves are copied out first: hipcc folds a bit-cast of element 1 of
  // the result to element 0)
  const uint32_t a = r16[0], b = r16[1];
  v = op(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
  u = __builtin_bit_cast(uint32_t, v);
  const auto r32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const uint32_t c = r32[0], e = r32[1];
  return op(__builtin_bit_cast(float, c), __builtin_bit_cast(float, e));
}
__device__ __forceinline__ float wave_max_dpp(float v) {
  return wave_reduce(v, [](float x, float y) { return fmaxf(x, y); });
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
  return wave_reduce(v, [](float x, float y) { return x + y; });
}

// Four consecutive elements of a cache row as floats (16-byte loads when the
// row data is float and 16-byte aligned).
template <typename T, bool kVec>
__device__ __forceinline__ void load4(const T* p, int64_t i, float (&x)[4]) {
  if constexpr (kVec) {
    const float4 v = *reinterpret_cast<const float4*>(p + i);
    x[0] = v.x;
    x[1] = v.y;
    x[2] = v.z;
    x[3] = v.w;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = load_f32(p, i + e);
  }
}

template <typename T, bool kVec>
__global__ void __launch_bounds__(kVecThreads) attn_vector_kernel(
    const T* __restrict__ q, const T* __restrict__ k_cache, const T* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ prefix_len,
    const int32_t* __restrict__ parents, const int32_t* __restrict__ n_nodes, T* __restrict__ out,
    int Nmax, int Hq, int Hkv, int d, int kv_rows, int max_blocks, float scale,
    const int32_t* status) {
  // K transposed by groups of 4 dims (lane = key reads 16 consecutive bytes,
  // consecutive lanes consecutive 16-byte words); V by rows (lanes = dims)
  __shared__ float4 kt_s[kMaxD / 4][kTileKeys];
  __shared__ __attribute__((aligned(16))) float v_s[kTileKeys * kMaxD];
  __shared__ float4 q_s[kVecWaves][kMaxD / 4];
  __shared__ __attribute__((aligned(16))) float p_s[kVecWaves][kTileKeys];
  __shared__ int path_s[LTD_MAX_NODES];
  __shared__ int path_len_s;

  const int i = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x, lane = t % kWave, w = t / kWave;
  if (halted(status)) return;
  if (i >= n_nodes[b]) return;  // uniform for the workgroup
  const int G = Hq / Hkv;
  const int P = prefix_len[b];
  const int32_t* par = parents + static_cast<int64_t>(b) * Nmax;
  if (t == 0) path_len_s = root_path(par, i, path_s);  // tree rows node i may see
  __syncthreads();
  const int n_keys = P + path_len_s;
  const int n_tiles = (n_keys + kTileKeys - 1) / kTileKeys;
  const int dq = d / 4;  // 16-byte pieces of a row

  for (int h0 = 0; h0 < G; h0 += kVecWaves) {
    const int h = h0 + w;             // this wave's head within the group
    const bool head = h < G;
    const int64_t q_off = ((static_cast<int64_t>(b) * Nmax + i) * Hq + g * G + (head ? h : 0)) * d;
    for (int e = lane; e < d; e += kWave)
      reinterpret_cast<float*>(q_s[w])[e] = head ? load_f32(q, q_off + e) * scale : 0.f;
    float m = -INFINITY, l = 0.f;
    float acc0 = 0.f, acc1 = 0.f;  // head dims lane and lane + 64
    // Tile loads go through registers one tile ahead: thread t holds the
    // 16-byte pieces x = t + 256 j of the tile's rows (piece x: row x / dq,
    // dims 4 (x % dq) .. + 3), so the next tile's loads are in flight while
    // the current one is computed.
    float kr4[kPieces][4], vr4[kPieces][4];
    auto fetch = [&](int tile) {
      const int base = tile * kTileKeys;
      const int cnt = min(kTileKeys, n_keys - base);
#pragma unroll
      for (int j = 0; j < kPieces; ++j) {
        const int x = t + j * kVecThreads;
        const int r = x / dq, c = (x % dq) * 4;
        if (r < cnt) {
          const int kt = base + r;
          const int row = kt < P ? kt : P + path_s[kt - P];
          const int64_t off = cache_row(block_table, b, g, row, Hkv, d, kv_rows, max_blocks) + c;
          load4<T, kVec>(k_cache, off, kr4[j]);
          load4<T, kVec>(v_cache, off, vr4[j]);
        }
      }
    };
    if (n_tiles > 0) fetch(0);
    for (int tile = 0; tile < n_tiles; ++tile) {
      const int base = tile * kTileKeys;
      const int cnt = min(kTileKeys, n_keys - base);
      __syncthreads();  // every wave is done with the previous tile (and q_s is written)
      // (rows past the tile's keys are zero: their weights are zero too, and
      // stale LDS could hold NaN)
#pragma unroll
      for (int j = 0; j < kPieces; ++j) {
        const int x = t + j * kVecThreads;
        const int r = x / dq, c = (x % dq) * 4;
        if (r < kTileKeys) {
          const bool in = r < cnt;
          kt_s[c / 4][r] = in ? make_float4(kr4[j][0], kr4[j][1], kr4[j][2], kr4[j][3])
                              : make_float4(0.f, 0.f, 0.f, 0.f);
          *reinterpret_cast<float4*>(v_s + r * kMaxD + c) =
              in ? make_float4(vr4[j][0], vr4[j][1], vr4[j][2], vr4[j][3])
                 : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      if (tile + 1 < n_tiles) fetch(tile + 1);
      __syncthreads();
      if (!head) continue;
      // score of key `lane`: four independent partial sums over groups of 4 dims
      float s = -INFINITY;
      {
        float d4[4] = {0.f, 0.f, 0.f, 0.f};
        for (int eg = 0; eg < dq; eg += 4) {
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float4 kv = kt_s[eg + u][lane];
            const float4 qv = q_s[w][eg + u];
            d4[u] += qv.x * kv.x + qv.y * kv.y + qv.z * kv.z + qv.w * kv.w;
          }
        }
        if (lane < cnt) s = (d4[0] + d4[1]) + (d4[2] + d4[3]);
      }
      const float m_new = fmaxf(m, wave_max_dpp(s));
      const float p = lane < cnt ? expf(s - m_new) : 0.f;
      const float alpha = expf(m - m_new);
      l = l * alpha + wave_sum_dpp(p);
      acc0 *= alpha;
      acc1 *= alpha;
      m = m_new;
      p_s[w][lane] = p;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // (weights past cnt are 0, and so are those rows of V)
      float a0[4] = {0.f, 0.f, 0.f, 0.f}, a1[4] = {0.f, 0.f, 0.f, 0.f};
      const int cnt4 = (cnt + 3) & ~3;
      for (int u = 0; u < cnt4; u += 4) {
        const float4 p4 = *reinterpret_cast<const float4*>(&p_s[w][u]);
        const float pu[4] = {p4.x, p4.y, p4.z, p4.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          a0[k] += pu[k] * v_s[(u + k) * kMaxD + lane];
          if (d > kWave) a1[k] += pu[k] * v_s[(u + k) * kMaxD + lane + kWave];
        }
      }
      acc0 += (a0[0] + a0[1]) + (a0[2] + a0[3]);
      acc1 += (a1[0] + a1[1]) + (a1[2] + a1[3]);
    }
    if (head) {
      const float inv = 1.f / l;
      if (lane < d) store_f32(out, q_off + lane, acc0 * inv);
      if (lane + kWave < d) store_f32(out, q_off + lane + kWave, acc1 * inv);
    }
    __syncthreads();  // q_s and the tiles are reused by the next head group
  }
}

}  // namespace

hipError_t launch_attn_rowwise(const AttnShape& s, const void* q, const void* k_cache,
                               const void* v_cache, const int32_t* block_table,
                               const int32_t* prefix_len, const int32_t* parents,
                               const int32_t* n_nodes, void* out, float scale,
                               const int32_t* status, hipStream_t stream) {
  const dim3 grid(s.Nmax, s.Hkv, s.B);
  if (s.dtype == LTD_DTYPE_F32) {
    // 16-byte loads when both caches are 16-byte aligned (every row and piece
    // offset is a multiple of 4 elements)
    const bool vec = (reinterpret_cast<uintptr_t>(k_cache) % 16) == 0 &&
                     (reinterpret_cast<uintptr_t>(v_cache) % 16) == 0;
    auto kern = vec ? attn_vector_kernel<float, true> : attn_vector_kernel<float, false>;
    hipLaunchKernelGGL(kern, grid, dim3(kVecThreads), 0, stream,
                       static_cast<const float*>(q), static_cast<const float*>(k_cache),
                       static_cast<const float*>(v_cache), block_table, prefix_len, parents,
                       n_nodes, static_cast<float*>(out), s.Nmax, s.Hq, s.Hkv, s.d, s.kv_rows,
                       s.max_blocks, scale, status);
  } else {
    hipLaunchKernelGGL((attn_vector_kernel<uint16_t, false>), grid, dim3(kVecThreads), 0, stream,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_cache),
                       static_cast<const uint16_t*>(v_cache), block_table, prefix_len, parents,
                       n_nodes, static_cast<uint16_t*>(out), s.Nmax, s.Hq, s.Hkv, s.d,
                       s.kv_rows, s.max_blocks, scale, status);
  }
  return hipGetLastError();
}

}  // namespace ltd
