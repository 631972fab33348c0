// Acceptance at temperature T > 0 by recursive rejection sampling over each
// node's children (drafts drawn without replacement from the node's draft
// distribution Q, tried in ascending node order against the target
// P = softmax(logits / T)): child token x is accepted with probability
// min(1, P(x)/Q(x)); on rejection P becomes max(P - Q, 0) renormalised and Q
// drops x; with no child accepted the bonus token is drawn from P.
//
// The residuals never need to be stored.  Children carry distinct tokens, and
// after k rejections at a node every token v has
//     P_k(v) = max(P(v) - g_k Q(v), 0) / s_k,   Q_k(v) = Q(v) / (1 - D_k)
// (a rejected token's residual is already 0), with g_1 = 0, s_1 = 1, D_1 = 0
// and, on the k-th rejection of token x,
//     g_{k+1} = g_k + s_k / (1 - D_k),  D_{k+1} = D_k + Q(x),
//     s_{k+1} = sum_v max(P(v) - g_{k+1} Q(v), 0)   (kept if it is 0).
// So an accept test needs only P(x) and Q(x) and two scalars, each rejection
// one pass over the vocabulary for s_{k+1}, and the bonus one inverse-CDF pass.
// The first rejection at any node sets g_2 = 1 exactly, so the masses at g = 0
// and g = 1 can be taken for every node at once, before the walk.
//
//   sample_stats_kernel  grid (vocab chunks of 4096, Nmax, B): per node, the
//                        chunk's partial of the softmax of logits / T (max and
//                        sum of exp) and, for nodes with children, the sum of
//                        its draft row;
//   sample_mass_kernel   the same grid, nodes with children only: per chunk,
//                        the residual mass at g = 1 with the walk's own
//                        parameters (the mass at g = 0 is the chunk's softmax
//                        partial);
//   sample_walk_kernel   one 1024-thread workgroup per sequence walks the tree:
//                        scalar accept tests; a node's first rejection reads
//                        its mass from the table, each later one takes a
//                        block-wide pass; the bonus takes its chunk from the
//                        table when g is 0 or 1, and otherwise narrows the
//                        range holding the target mass sixteenfold per level
//                        (one coalesced segment sum per wave); a wave scan of
//                        the last 64 tokens or fewer ends the search.
// Element arithmetic is float32, every sum over the vocabulary is finished in
// double.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kStatThreads = 256;
constexpr int kChunk = 4096;
constexpr int kPerThread = kChunk / kStatThreads;
constexpr int kWalkThreads = 1024;
constexpr int kWalkWaves = kWalkThreads / kWave;
constexpr int kMaxChunks = LTD_SAMPLING_MAX_CHUNKS;
static_assert(kMaxChunks <= kWave, "the walk merges one chunk partial a lane");

// Node j's parent as every kernel here reads it: in [0, j - 1] (the links of
// a valid tree; malformed ones are clamped, so all kernels agree on the tree).
__device__ __forceinline__ int link(const int32_t* __restrict__ parents, int64_t nb, int j) {
  return j == 0 ? -1 : min(max(parents[nb + j], 0), j - 1);
}

struct NodeStats {  // per (sequence, node, chunk)
  float m;   // max of logits / T over the chunk
  float z;   // sum of exp(logits / T - m)
  float qs;  // sum of the draft row over the chunk (nodes with children)
  float pad;
};

__global__ void __launch_bounds__(kStatThreads) sample_stats_kernel(
    const float* __restrict__ logits, const float* __restrict__ draft_probs,
    const int32_t* __restrict__ parents, const int32_t* __restrict__ n_nodes, int Nmax, int Voc,
    float inv_t, NodeStats* __restrict__ ws, const int32_t* status) {
  __shared__ float red_s[3][kStatThreads / kWave];
  __shared__ int has_child_s;
  if (halted(status)) return;
  const int chunk = blockIdx.x, i = blockIdx.y, b = blockIdx.z;
  const int chunks = gridDim.x;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int n = min(max(n_nodes[b], 1), Nmax);
  if (i >= n) return;  // uniform for the block
  const int64_t row = (static_cast<int64_t>(b) * Nmax + i) * Voc;
  const int base = chunk * kChunk;
  float l[kPerThread], q[kPerThread];
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int v = base + k * kStatThreads + t;
    const float lv = logits[row + min(v, Voc - 1)];
    l[k] = v < Voc ? lv * inv_t : -INFINITY;
  }
  // the draft row is read only for nodes with children
  if (t == 0) has_child_s = 0;
  __syncthreads();
  for (int j = t; j < n; j += kStatThreads)
    if (j > i && link(parents, static_cast<int64_t>(b) * Nmax, j) == i) has_child_s = 1;
  __syncthreads();
  const bool want_q = has_child_s != 0;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int v = base + k * kStatThreads + t;
    const float qv = want_q ? draft_probs[row + min(v, Voc - 1)] : 0.f;
    q[k] = v < Voc ? qv : 0.f;
  }
  float m = -INFINITY;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) m = fmaxf(m, l[k]);
  float z = 0.f, qs = 0.f;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    z += m == -INFINITY ? 0.f : __expf(l[k] - m);
    qs += q[k];
  }
  // (m, z) and qs over the block
  float mm = m;
  mm = fmaxf(mm, lane_xor_f<32>(mm, lane));
  mm = fmaxf(mm, lane_xor_f<16>(mm, lane));
  mm = fmaxf(mm, lane_xor_f<8>(mm, lane));
  mm = fmaxf(mm, lane_xor_f<4>(mm, lane));
  mm = fmaxf(mm, lane_xor_f<2>(mm, lane));
  mm = fmaxf(mm, lane_xor_f<1>(mm, lane));
  if (lane == 0) red_s[0][w] = mm;
  __syncthreads();
  float M = red_s[0][0];
#pragma unroll
  for (int k = 1; k < kStatThreads / kWave; ++k) M = fmaxf(M, red_s[0][k]);
  float zz = m == -INFINITY ? 0.f : z * __expf(m - M);
  zz = wave_sum(zz);
  const float qq = want_q ? wave_sum(qs) : 0.f;
  if (lane == 0) {
    red_s[1][w] = zz;
    red_s[2][w] = qq;
  }
  __syncthreads();
  if (t == 0) {
    float Z = 0.f, QS = 0.f;
#pragma unroll
    for (int k = 0; k < kStatThreads / kWave; ++k) {
      Z += red_s[1][k];
      QS += red_s[2][k];
    }
    ws[(static_cast<int64_t>(b) * Nmax + i) * chunks + chunk] = NodeStats{M, Z, QS, 0.f};
  }
}

// The residual R(v) = max(P(v) - g Q(v), 0) of one node, with P(v) =
// exp(l_v/T - M) / Z and Q(v) = q_v / QS, as one FMA, one exp2 and one FMA
// per token: P(v) = 2^(l_v a - b) with a = log2(e)/T and b = log2(e) (M +
// ln Z), and g Q(v) = gq q_v with gq = g / QS.
struct Residual {
  float a, b, gq;
};
__device__ __forceinline__ float residual_elem(float l, float q, const Residual& r) {
  const float p = __builtin_amdgcn_exp2f(fmaf(l, r.a, -r.b));
  return fmaxf(fmaf(-r.gq, q, p), 0.f);
}

// One thread's share of sum_v R(v): float4 loads of both rows in batches of
// kBatch, all issued before any use (a strided, coalesced layout; rows of a
// vocabulary that is not a multiple of 4 take the scalar path).
constexpr int kBatch = 4;
__device__ float residual_pass(const float* __restrict__ l, const float* __restrict__ q, int Voc,
                               int t, const Residual& r) {
  float part = 0.f;
  const bool aligned = (Voc & 3) == 0 && (reinterpret_cast<uintptr_t>(l) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(q) & 15) == 0;
  if (aligned) {
    const int n4 = Voc / 4;
    const float4* l4 = reinterpret_cast<const float4*>(l);
    const float4* q4 = reinterpret_cast<const float4*>(q);
    for (int i0 = t; i0 < n4; i0 += kBatch * kWalkThreads) {
      float4 lv[kBatch], qv[kBatch];
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const int i = min(i0 + k * kWalkThreads, n4 - 1);
        lv[k] = l4[i];
        qv[k] = q4[i];
      }
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        if (i0 + k * kWalkThreads < n4) {
          part += residual_elem(lv[k].x, qv[k].x, r);
          part += residual_elem(lv[k].y, qv[k].y, r);
          part += residual_elem(lv[k].z, qv[k].z, r);
          part += residual_elem(lv[k].w, qv[k].w, r);
        }
      }
    }
  } else {
    for (int v0 = t; v0 < Voc; v0 += kBatch * kWalkThreads) {
      float lv[kBatch], qv[kBatch];
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const int v = min(v0 + k * kWalkThreads, Voc - 1);
        lv[k] = l[v];
        qv[k] = q[v];
      }
#pragma unroll
      for (int k = 0; k < kBatch; ++k)
        if (v0 + k * kWalkThreads < Voc)
          part += residual_elem(lv[k], qv[k], r);
    }
  }
  return part;
}

// The node's softmax maximum (float, logits / T units), normaliser Z and
// draft-row sum QS (double) from its chunk partials, by one wave (lane c
// takes chunk c), in the same order wherever it is called, so every kernel
// derives bit-identical residual parameters.
struct NodeTotals {
  float Mf;
  double Z, QS;
};
__device__ NodeTotals merge_node_stats_of(const NodeStats st, int chunks, int lane) {
  const float m_l = lane < chunks ? st.m : -INFINITY;
  float Mf = m_l;
  Mf = fmaxf(Mf, lane_xor_f<32>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<16>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<8>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<4>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<2>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<1>(Mf, lane));
  double zl =
      m_l != -INFINITY ? static_cast<double>(st.z) * exp(static_cast<double>(m_l - Mf)) : 0.0;
  double ql = lane < chunks ? static_cast<double>(st.qs) : 0.0;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    uint64_t oz, oq;
    const uint64_t bz = static_cast<uint64_t>(__double_as_longlong(zl));
    const uint64_t bq = static_cast<uint64_t>(__double_as_longlong(ql));
    switch (d) {
      case 32: oz = lane_xor_u64<32>(bz, lane); oq = lane_xor_u64<32>(bq, lane); break;
      case 16: oz = lane_xor_u64<16>(bz, lane); oq = lane_xor_u64<16>(bq, lane); break;
      case 8: oz = lane_xor_u64<8>(bz, lane); oq = lane_xor_u64<8>(bq, lane); break;
      case 4: oz = lane_xor_u64<4>(bz, lane); oq = lane_xor_u64<4>(bq, lane); break;
      case 2: oz = lane_xor_u64<2>(bz, lane); oq = lane_xor_u64<2>(bq, lane); break;
      default: oz = lane_xor_u64<1>(bz, lane); oq = lane_xor_u64<1>(bq, lane);
    }
    zl += __longlong_as_double(static_cast<long long>(oz));
    ql += __longlong_as_double(static_cast<long long>(oq));
  }
  return NodeTotals{Mf, zl, ql};
}
__device__ NodeTotals merge_node_stats(const NodeStats* __restrict__ st_row, int chunks, int lane) {
  return merge_node_stats_of(st_row[min(lane, chunks - 1)], chunks, lane);
}

constexpr double kLog2e = 1.4426950408889634;
__device__ __forceinline__ Residual residual_params(const NodeTotals& nt, float inv_t, double g) {
  Residual r;
  r.a = static_cast<float>(kLog2e * static_cast<double>(inv_t));
  r.b = static_cast<float>(kLog2e * (static_cast<double>(nt.Mf) + log(nt.Z)));
  r.gq = g > 0.0 && nt.QS > 0.0 ? static_cast<float>(g / nt.QS) : 0.f;
  return r;
}

// Wave-wide double sum (every lane gets it).
__device__ __forceinline__ double wave_sum_d(double v, int lane) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    uint64_t o;
    const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(v));
    switch (d) {
      case 32: o = lane_xor_u64<32>(bits, lane); break;
      case 16: o = lane_xor_u64<16>(bits, lane); break;
      case 8: o = lane_xor_u64<8>(bits, lane); break;
      case 4: o = lane_xor_u64<4>(bits, lane); break;
      case 2: o = lane_xor_u64<2>(bits, lane); break;
      default: o = lane_xor_u64<1>(bits, lane);
    }
    v += __longlong_as_double(static_cast<long long>(o));
  }
  return v;
}

// Block-wide double sum of one value per thread (every thread gets it).
__device__ double block_sum(double v, double* red_s, int lane, int w) {
  v = wave_sum_d(v, lane);
  __syncthreads();  // red_s may still be read from the previous call
  if (lane == 0) red_s[w] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int k = 0; k < kWalkWaves; ++k) s += red_s[k];
  return s;
}

// Sum of R(v) = max(P(v) - g Q(v), 0) over tokens [lo, hi) by one wave, its
// lanes reading consecutive tokens (float4 each when kVec: lo and hi are then
// multiples of 4 and the rows 16-byte aligned), kBatch loads in flight.
template <bool kVec>
__device__ double wave_range_sum(const float* __restrict__ l, const float* __restrict__ q, int lo,
                                 int hi, int lane, bool use_q, const Residual& r) {
  double acc = 0.0;
  if (kVec) {
    constexpr int kStep = 4 * kWave;
    for (int v0 = lo + 4 * lane; v0 < hi; v0 += kBatch * kStep) {
      float4 lv[kBatch], qv[kBatch];
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const int v = min(v0 + k * kStep, hi - 4);
        lv[k] = *reinterpret_cast<const float4*>(l + v);
        qv[k] = use_q ? *reinterpret_cast<const float4*>(q + v) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        if (v0 + k * kStep < hi) {
          float sum4 = residual_elem(lv[k].x, qv[k].x, r);
          sum4 += residual_elem(lv[k].y, qv[k].y, r);
          sum4 += residual_elem(lv[k].z, qv[k].z, r);
          sum4 += residual_elem(lv[k].w, qv[k].w, r);
          acc += static_cast<double>(sum4);
        }
      }
    }
  } else {
    for (int v0 = lo + lane; v0 < hi; v0 += kBatch * kWave) {
      float lv[kBatch], qv[kBatch];
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const int v = min(v0 + k * kWave, hi - 1);
        lv[k] = l[v];
        qv[k] = use_q ? q[v] : 0.f;
      }
#pragma unroll
      for (int k = 0; k < kBatch; ++k)
        if (v0 + k * kWave < hi)
          acc += static_cast<double>(residual_elem(lv[k], qv[k], r));
    }
  }
  return wave_sum_d(acc, lane);
}

// Per (node with children, chunk): the residual mass
// sum_v max(P(v) - Q(v), 0) over the chunk, i.e. at g = 1 (after the node's
// first rejection, g is exactly 1), with the walk's own parameters and element
// arithmetic.
__global__ void __launch_bounds__(kStatThreads) sample_mass_kernel(
    const float* __restrict__ logits, const float* __restrict__ draft_probs,
    const int32_t* __restrict__ parents, const int32_t* __restrict__ n_nodes, int Nmax, int Voc,
    float inv_t, const NodeStats* __restrict__ ws, double* __restrict__ mass1,
    const int32_t* status) {
  __shared__ NodeTotals nt_s;
  __shared__ int has_child_s;
  __shared__ double red_s[kStatThreads / kWave];
  if (halted(status)) return;
  const int chunk = blockIdx.x, i = blockIdx.y, b = blockIdx.z;
  const int chunks = gridDim.x;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int n = min(max(n_nodes[b], 1), Nmax);
  if (i >= n) return;  // uniform for the block
  const int64_t nb = static_cast<int64_t>(b) * Nmax;
  if (t == 0) has_child_s = 0;
  if (w == 0) {
    const NodeTotals nt = merge_node_stats(ws + (nb + i) * chunks, chunks, lane);
    if (lane == 0) nt_s = nt;
  }
  __syncthreads();
  for (int j = t; j < n; j += kStatThreads)
    if (j > i && link(parents, nb, j) == i) has_child_s = 1;
  __syncthreads();
  if (has_child_s == 0) {  // uniform: a leaf never rejects; its entry reads as 0
    if (t == 0) mass1[(nb + i) * chunks + chunk] = 0.0;
    return;
  }
  const int64_t row = (nb + i) * Voc;
  const int base = chunk * kChunk;
  float l[kPerThread], q[kPerThread];
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int64_t v = row + min(base + k * kStatThreads + t, Voc - 1);
    l[k] = logits[v];
    q[k] = draft_probs[v];
  }
  const Residual r1 = residual_params(nt_s, inv_t, 1.0);
  double d1 = 0.0;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k)
    if (base + k * kStatThreads + t < Voc) d1 += static_cast<double>(residual_elem(l[k], q[k], r1));
  d1 = wave_sum_d(d1, lane);
  if (lane == 0) red_s[w] = d1;
  __syncthreads();
  if (t == 0) {
    double a1 = 0.0;
#pragma unroll
    for (int k = 0; k < kStatThreads / kWave; ++k) a1 += red_s[k];
    mass1[(nb + i) * chunks + chunk] = a1;
  }
}

// Whether node u has a child, by one wave over the parent links in LDS.
__device__ __forceinline__ bool child_any(const int32_t* par_s, int n, int u, int lane) {
  bool any = false;
  for (int j = u + 1 + lane; j < n; j += kWave) any = any || par_s[j] == u;
  return __ballot(any) != 0;
}

__global__ void __launch_bounds__(kWalkThreads) sample_walk_kernel(
    const float* __restrict__ logits, const float* __restrict__ draft_probs,
    const int32_t* __restrict__ draft_tokens, const int32_t* __restrict__ parents,
    const int32_t* __restrict__ n_nodes, const float* __restrict__ uniforms, int Nmax, int Voc,
    float inv_t, const NodeStats* __restrict__ ws, const double* __restrict__ mass1, int chunks,
    int32_t* __restrict__ accepted, int32_t* __restrict__ out_tokens,
    int32_t* __restrict__ n_accepted, const int32_t* status) {
  __shared__ int32_t par_s[LTD_MAX_NODES];
  __shared__ int32_t tok_s[LTD_MAX_NODES];
  __shared__ uint64_t child_s[LTD_MAX_NODES / kWave];
  __shared__ int32_t path_s[LTD_MAX_NODES];
  __shared__ int32_t removed_s[LTD_MAX_NODES];
  __shared__ double red_s[kWalkWaves];
  __shared__ double node_s[4];  // M, Z, QS, and the residual mass at g = 1, of the current node
  __shared__ double2 mass_s[LTD_SAMPLING_MAX_CHUNKS];  // the node's chunk masses at g = 0, 1
  __shared__ double target_s;  // the bonus search: mass left to pass in [lo_s, hi_s)
  __shared__ int lo_s, hi_s;
  if (halted(status)) return;
  const int b = blockIdx.x;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int n = min(max(n_nodes[b], 1), Nmax);
  const int64_t nb = static_cast<int64_t>(b) * Nmax;
  if (t < Nmax) {
    par_s[t] = t >= n ? -1 : link(parents, nb, t);
    tok_s[t] = min(max(draft_tokens[nb + t], 0), Voc - 1);
  }
  __syncthreads();

  int u = 0, len = 0;
  if (t == 0) path_s[len] = 0;
  ++len;
  int bonus = 0;
  for (;;) {
    const int64_t row = (nb + u) * Voc;
    // the node's softmax normaliser and draft sum from the chunk partials,
    // and its chunk masses at g = 0 (the chunk's softmax mass, from its
    // partial) and at g = 1 (the mass table; written for nodes with children)
    if (w == 0) {
      // both loads first (a leaf's mass entries are 0)
      const NodeStats st = ws[(nb + u) * chunks + min(lane, chunks - 1)];
      const double m1_any = mass1[(nb + u) * chunks + min(lane, chunks - 1)];
      const NodeTotals nt = merge_node_stats_of(st, chunks, lane);
      const bool kids = child_any(par_s, n, u, lane);
      const double m1c = kids ? m1_any : 0.0;
      const double m0c = st.m != -INFINITY
                             ? static_cast<double>(st.z) *
                                   exp(static_cast<double>(st.m) - static_cast<double>(nt.Mf)) / nt.Z
                             : 0.0;
      if (lane < chunks) mass_s[lane] = make_double2(m0c, m1c);
      const double m1 = wave_sum_d(lane < chunks ? m1c : 0.0, lane);
      if (lane == 0) {
        node_s[0] = nt.Mf;
        node_s[1] = nt.Z;
        node_s[2] = nt.QS;
        node_s[3] = m1;
      }
    }
    // the node's children, in ascending order, as bits of 64-node words
    if (t < LTD_MAX_NODES) {
      const bool is_child = t < n && par_s[t] == u && t > u;
      const uint64_t m = __ballot(is_child);
      if (lane == 0) child_s[w] = m;
    }
    __syncthreads();
    const NodeTotals nt{static_cast<float>(node_s[0]), node_s[1], node_s[2]};
    const float Mf = nt.Mf;
    const double Z = nt.Z;
    const double QS = nt.QS;
    const double mass_g1 = node_s[3];
    Residual res = residual_params(nt, inv_t, 0.0);

    double g = 0.0, s = 1.0, D = 0.0;  // the residual after the rejections so far
    int n_removed = 0;
    int next = -1;
    for (int word = 0; word < LTD_MAX_NODES / kWave && next < 0; ++word) {
      uint64_t bits = child_s[word];
      while (bits != 0 && next < 0) {
        const int c = word * kWave + __ffsll(static_cast<long long>(bits)) - 1;
        bits &= bits - 1;
        const int x = tok_s[c];
        const double Px =
            exp(static_cast<double>(logits[row + x] * inv_t) - static_cast<double>(Mf)) / Z;
        const double Qx = QS > 0.0 ? static_cast<double>(draft_probs[row + x]) / QS : 0.0;
        bool removed = false;
        for (int k = 0; k < n_removed; ++k) removed = removed || removed_s[k] == x;
        const double Pk = fmax(Px - g * Qx, 0.0) / s;
        const double Qk = removed ? 0.0 : Qx / (1.0 - D);
        const double r = static_cast<double>(uniforms[(nb + c) * 2]);
        if (r * Qk < Pk) {
          next = c;
          break;
        }
        // rejected: the next residual's mass.  After the first rejection g is
        // exactly 1 and the mass table holds it; later ones take one pass
        // over the vocabulary.
        const double g2 = g + s / (1.0 - D);
        double s2;
        if (n_removed == 0) {
          s2 = mass_g1;
        } else {
          res = residual_params(nt, inv_t, g2);
          const float part = residual_pass(logits + row, draft_probs + row, Voc, t, res);
          s2 = block_sum(static_cast<double>(part), red_s, lane, w);
        }
        if (t == 0) removed_s[n_removed] = x;
        __syncthreads();
        if (!removed) D += Qx;
        ++n_removed;
        if (s2 > 0.0) {
          g = g2;
          s = s2;
        }
      }
    }
    if (next >= 0) {
      if (t == 0) path_s[len] = next;
      ++len;
      u = next;
      __syncthreads();  // node_s / child_s are rewritten for the new node
      continue;
    }

    // The bonus: inverse CDF of R = max(P - g Q, 0) at uniforms[u][1] times
    // its mass.  The range holding the target is narrowed in levels: the 16
    // waves sum R over 16 equal segments of it, thread 0 scans the sums and
    // keeps the segment where the mass passes the target; at 64 tokens or
    // fewer wave 0 takes an inclusive scan and the first token past the
    // target.  Where rounding leaves the target at or past a level's sum, the
    // last segment (token) with mass is taken, as the plain scan would.
    const bool use_q = g > 0.0;
    res = residual_params(nt, inv_t, g);
    const bool vec = (Voc & 3) == 0 && (reinterpret_cast<uintptr_t>(logits + row) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(draft_probs + row) & 15) == 0;
    int lo = 0, hi = Voc;
    bool first = true;  // no level yet: the final scan sets the target itself
    if (g == 0.0 || g == 1.0) {  // the first level from the mass table's chunks
      if (t == 0) {
        const bool g1 = g == 1.0;
        double total = 0.0;
        for (int c = 0; c < chunks; ++c) total += g1 ? mass_s[c].y : mass_s[c].x;
        const double target = static_cast<double>(uniforms[(nb + u) * 2 + 1]) * total;
        int pick = -1, last = -1;
        double cum = 0.0, before = 0.0, upto_last = 0.0, run = 0.0;
        for (int c = 0; c < chunks && pick < 0; ++c) {
          const double mc = g1 ? mass_s[c].y : mass_s[c].x;
          if (mc > 0.0) {
            last = c;
            upto_last = run;
          }
          before = cum;
          cum += mc;
          run = cum;
          if (cum > target && mc > 0.0) pick = c;
        }
        if (pick < 0) {  // past the end by rounding (or no mass at all)
          pick = last;
          before = upto_last;
        }
        if (pick < 0) {
          lo_s = 0;
          hi_s = 0;  // no mass: token 0
        } else {
          lo_s = pick * kChunk;
          hi_s = min(lo_s + kChunk, Voc);
        }
        target_s = target - before;
      }
      __syncthreads();
      lo = lo_s;
      hi = hi_s;
      first = false;
    }
    for (; hi - lo > kWave; first = false) {
      const int span = hi - lo;
      const int seg = vec ? ((span + 4 * kWalkWaves - 1) / (4 * kWalkWaves)) * 4
                          : (span + kWalkWaves - 1) / kWalkWaves;
      const int s_lo = min(lo + w * seg, hi), s_hi = min(s_lo + seg, hi);
      const double sum =
          vec ? wave_range_sum<true>(logits + row, draft_probs + row, s_lo, s_hi, lane, use_q, res)
              : wave_range_sum<false>(logits + row, draft_probs + row, s_lo, s_hi, lane, use_q, res);
      if (lane == 0) red_s[w] = sum;
      __syncthreads();
      if (t == 0) {
        double target = first ? 0.0 : target_s;
        if (first) {
          double total = 0.0;
          for (int k = 0; k < kWalkWaves; ++k) total += red_s[k];
          target = static_cast<double>(uniforms[(nb + u) * 2 + 1]) * total;
        }
        int pick = -1, last = -1;
        double cum = 0.0, before = 0.0;
        for (int k = 0; k < kWalkWaves && pick < 0; ++k) {
          if (red_s[k] > 0.0) last = k;
          before = cum;
          cum += red_s[k];
          if (cum > target && red_s[k] > 0.0) pick = k;
        }
        if (pick < 0) {  // past the end by rounding (or no mass at all)
          pick = last;
          before = 0.0;
          for (int k = 0; k < last; ++k) before += red_s[k];
        }
        if (pick < 0) {
          lo_s = 0;
          hi_s = 0;  // no mass: token 0
        } else {
          lo_s = min(lo + pick * seg, hi);
          hi_s = min(lo + (pick + 1) * seg, hi);
        }
        target_s = target - before;
      }
      __syncthreads();
      lo = lo_s;
      hi = hi_s;
    }
    if (w == 0) {
      const int v = lo + lane;
      float rv = 0.f;
      if (v < hi) {
        const float qv = use_q ? draft_probs[row + v] : 0.f;
        rv = residual_elem(logits[row + v], qv, res);
      }
      double incl = static_cast<double>(rv);
#pragma unroll
      for (int d = 1; d < kWave; d <<= 1) {
        const double o = __shfl_up(incl, d, kWave);
        if (lane >= d) incl += o;
      }
      const double target =
          first ? static_cast<double>(uniforms[(nb + u) * 2 + 1]) * __shfl(incl, kWave - 1, kWave)
                : target_s;
      const uint64_t past = __ballot(incl > target && rv > 0.f);
      const uint64_t mass = __ballot(rv > 0.f);
      if (lane == 0) {
        int pick = lo;
        if (past != 0)
          pick = lo + __ffsll(static_cast<long long>(past)) - 1;
        else if (mass != 0)
          pick = lo + 63 - __clzll(static_cast<long long>(mass));
        lo_s = pick;
      }
    }
    __syncthreads();
    bonus = lo_s;
    break;
  }

  // outputs
  for (int j = t; j < len; j += kWalkThreads) {
    accepted[nb + j] = path_s[j];
    out_tokens[nb + j] = j + 1 < len ? tok_s[path_s[j + 1]] : bonus;
  }
  if (t == 0) n_accepted[b] = len;
}

}  // namespace

int sampling_chunks(int Voc) { return (Voc + kChunk - 1) / kChunk; }

size_t sampling_workspace_bytes(int B, int Nmax, int Voc) {
  return (sizeof(NodeStats) + sizeof(double)) * static_cast<size_t>(B) * Nmax *
         sampling_chunks(Voc);
}

hipError_t launch_sampling(const float* logits, const float* draft_probs,
                           const int32_t* draft_tokens, const int32_t* parents,
                           const int32_t* n_nodes, const float* uniforms, int B, int Nmax,
                           int Voc, float temperature, int32_t* accepted_nodes,
                           int32_t* out_tokens, int32_t* n_accepted, void* workspace,
                           const int32_t* status, hipStream_t stream) {
  const int chunks = sampling_chunks(Voc);
  auto* ws = static_cast<NodeStats*>(workspace);
  auto* mass1 = reinterpret_cast<double*>(ws + static_cast<size_t>(B) * Nmax * chunks);
  const float inv_t = 1.0f / temperature;
  hipLaunchKernelGGL(sample_stats_kernel, dim3(chunks, Nmax, B), dim3(kStatThreads), 0, stream,
                     logits, draft_probs, parents, n_nodes, Nmax, Voc, inv_t, ws, status);
  hipLaunchKernelGGL(sample_mass_kernel, dim3(chunks, Nmax, B), dim3(kStatThreads), 0, stream,
                     logits, draft_probs, parents, n_nodes, Nmax, Voc, inv_t, ws, mass1, status);
  hipLaunchKernelGGL(sample_walk_kernel, dim3(B), dim3(kWalkThreads), 0, stream, logits,
                     draft_probs, draft_tokens, parents, n_nodes, uniforms, Nmax, Voc, inv_t, ws,
                     mass1, chunks, accepted_nodes, out_tokens, n_accepted, status);
  return hipGetLastError();
}

}  // namespace ltd
