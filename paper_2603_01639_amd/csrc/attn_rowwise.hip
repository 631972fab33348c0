// Row-wise tree attention on the vector ALUs: one wavefront per (sequence,
// node, query head).  This is the fp32 path (and the path for shapes the
// bf16 MFMA kernel does not cover).  Keys are visited in chunks of 64, one
// key per lane for the scores, one or two head dimensions per lane for the
// value accumulation, with an online (running-max) softmax across chunks.
//
// The visible key set of node i is the prefix [0, P_b) plus the tree rows of
// the node's root path (arXiv 2603.01639, section 3.2: the tree attention
// mask shows each candidate its ancestors only).
#include "ltd_device.hpp"
#include "ltd_launch.hpp"
#include "tree_walk.hpp"

namespace ltd {
namespace {

template <typename T>
__global__ void __launch_bounds__(kWave) attn_rowwise_kernel(
    const T* __restrict__ q, const T* __restrict__ k_cache, const T* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ prefix_len,
    const int32_t* __restrict__ parents, const int32_t* __restrict__ n_nodes, T* __restrict__ out,
    int Nmax, int Hq, int Hkv, int d, int kv_rows, int max_blocks, float scale,
    const int32_t* status) {
  __shared__ float q_s[128];
  __shared__ int path_s[LTD_MAX_NODES];
  __shared__ float p_s[kWave];
  __shared__ int row_s[kWave];
  __shared__ int path_len_s;

  const int b = blockIdx.y;
  const int i = blockIdx.x / Hq;
  const int h = blockIdx.x % Hq;
  const int lane = threadIdx.x;
  if (halted(status)) return;
  if (i >= n_nodes[b]) return;
  const int g = h / (Hq / Hkv);
  const int P = prefix_len[b];
  const int32_t* par = parents + static_cast<int64_t>(b) * Nmax;

  const int64_t q_off = ((static_cast<int64_t>(b) * Nmax + i) * Hq + h) * d;
  for (int e = lane; e < d; e += kWave) q_s[e] = load_f32(q, q_off + e) * scale;
  if (lane == 0) path_len_s = root_path(par, i, path_s);  // tree rows node i may see
  __syncthreads();
  const int n_keys = P + path_len_s;

  float m = -INFINITY, l = 0.f;
  float acc0 = 0.f, acc1 = 0.f;  // head dims lane and lane + 64
  for (int base = 0; base < n_keys; base += kWave) {
    const int t = base + lane;
    float s = -INFINITY;
    int row = 0;
    if (t < n_keys) {
      row = t < P ? t : P + path_s[t - P];
      const int64_t off = cache_row(block_table, b, g, row, Hkv, d, kv_rows, max_blocks);
      float dot = 0.f;
      for (int e = 0; e < d; ++e) dot += q_s[e] * load_f32(k_cache, off + e);
      s = dot;
    }
    const float m_new = fmaxf(m, wave_max(s));
    const float p = (t < n_keys) ? expf(s - m_new) : 0.f;
    const float alpha = expf(m - m_new);
    l = l * alpha + wave_sum(p);
    acc0 *= alpha;
    acc1 *= alpha;
    m = m_new;
    p_s[lane] = p;
    row_s[lane] = row;
    __syncthreads();
    const int cnt = min(kWave, n_keys - base);
    for (int u = 0; u < cnt; ++u) {
      const int64_t off = cache_row(block_table, b, g, row_s[u], Hkv, d, kv_rows, max_blocks);
      const float pu = p_s[u];
      if (lane < d) acc0 += pu * load_f32(v_cache, off + lane);
      if (lane + kWave < d) acc1 += pu * load_f32(v_cache, off + lane + kWave);
    }
    __syncthreads();
  }
  const float inv = 1.f / l;
  if (lane < d) store_f32(out, q_off + lane, acc0 * inv);
  if (lane + kWave < d) store_f32(out, q_off + lane + kWave, acc1 * inv);
}

}  // namespace

hipError_t launch_attn_rowwise(const AttnShape& s, const void* q, const void* k_cache,
                               const void* v_cache, const int32_t* block_table,
                               const int32_t* prefix_len, const int32_t* parents,
                               const int32_t* n_nodes, void* out, float scale,
                               const int32_t* status, hipStream_t stream) {
  const dim3 grid(s.Nmax * s.Hq, s.B);
  if (s.dtype == LTD_DTYPE_F32) {
    hipLaunchKernelGGL(attn_rowwise_kernel<float>, grid, dim3(kWave), 0, stream,
                       static_cast<const float*>(q), static_cast<const float*>(k_cache),
                       static_cast<const float*>(v_cache), block_table, prefix_len, parents,
                       n_nodes, static_cast<float*>(out), s.Nmax, s.Hq, s.Hkv, s.d, s.kv_rows,
                       s.max_blocks, scale, status);
  } else {
    hipLaunchKernelGGL(attn_rowwise_kernel<uint16_t>, grid, dim3(kWave), 0, stream,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_cache),
                       static_cast<const uint16_t*>(v_cache), block_table, prefix_len, parents,
                       n_nodes, static_cast<uint16_t*>(out), s.Nmax, s.Hq, s.Hkv, s.d,
                       s.kv_rows, s.max_blocks, scale, status);
  }
  return hipGetLastError();
}

}  // namespace ltd
