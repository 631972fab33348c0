// Acceptance at temperature T > 0 by recursive rejection sampling over each
// node's children (drafts drawn without replacement from the node's draft
// distribution Q, tried in ascending node order against the target
// P = softmax(logits / T)): child token x is accepted with probability
// min(1, P(x)/Q(x)); on rejection P becomes max(P - Q, 0) renormalised and Q
// drops x; with no child accepted the bonus token is drawn from P.
//
// The residuals never need to be stored.  Children carry distinct tokens, and
// after k rejections at a node every token v has
//     P_k(v) = max(P(v) - g_k Q(v), 0) / s_k,   Q_k(v) = Q(v) / R_k
// for tokens not yet rejected (a rejected token's residual is already 0 and
// its Q_k is 0), with g_1 = 0, s_1 = 1, R_1 = 1 and, on the k-th rejection,
//     g_{k+1} = g_k + s_k / R_k,
//     s_{k+1} = sum_v max(P(v) - g_{k+1} Q(v), 0)   (kept if it is 0),
//     R_{k+1} = sum of Q(v) over the tokens not rejected so far.
// R is summed over the remaining tokens, never taken as 1 minus the rejected
// mass: when the rejected drafts hold nearly all of Q that difference loses
// every digit (a draft row of 0.9998 on one token leaves 2e-4, and a few more
// rejections leave less than double rounding of 1), and g with it.  Once R is
// 0 (every token with draft mass rejected) Q_k is 0: a child is accepted
// where P_k(x) > 0 and a rejection leaves P as it is.
// So an accept test needs only P(x) and Q(x) and three scalars, each rejection
// one pass over the vocabulary for s_{k+1} and R_{k+1}, and the bonus one
// inverse-CDF pass.
// None of g_k, s_k, R_k depends on the uniforms: a node's children are tried in
// a fixed order, so the residual after its k-th rejection is the same whatever
// the draws, and its mass can be taken for every node at once, before the
// walk, one level k per launch (level k needs the total of level k - 1).  The
// first rejection at any node sets g_2 = 1 exactly.
//
//   sample_stats_kernel  grid (vocab chunks of 4096, Nmax, B): per node, the
//                        chunk's partial of the softmax of logits / T (max and
//                        sum of exp) and, for nodes with children, the sum of
//                        its draft row;
//   sample_mass_kernel   the same grid, launched for levels k = 1 .. kLevels,
//                        nodes with at least k children only: per chunk, the
//                        residual mass after the node's k-th rejection, with
//                        the walk's own parameters and arithmetic (the mass at
//                        g = 0 is the chunk's softmax partial), and the
//                        chunk's draft mass outside the rejected tokens;
//   sample_walk_kernel   one 1024-thread workgroup per sequence walks the tree:
//                        scalar accept tests; a node's first kLevels rejections
//                        read their masses from the tables, each later one
//                        takes a block-wide pass (the rejected tokens are bits
//                        of an LDS bitmap of the vocabulary); the bonus takes its chunk from
//                        a table when its residual is one of them, and
//                        otherwise narrows the range holding the target mass
//                        sixteenfold per level (one coalesced segment sum per
//                        wave); a wave scan of the last 64 tokens or fewer ends
//                        the search.
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
constexpr int kLevels = 3;  // rejections per node whose residual masses are tabled

// The residual after a node's rejections so far: P_k = max(P - g Q, 0) / s,
// and R = the draft mass of the tokens not rejected.  The walk and the mass
// tables advance it with the same operations, so both see bit-identical g.
struct RejState {
  double g, s, R;
};
// g of the residual after the next rejection (unchanged once no draft mass
// is left: Q_k is then 0 and a rejection leaves P as it is).
__device__ __forceinline__ double next_g(const RejState& st) {
  return st.R > 0.0 ? st.g + st.s / st.R : st.g;
}
// The rejection after which the residual at g2 has mass s2 and R2 of the
// draft mass is left (a residual without mass leaves P as it was).
__device__ __forceinline__ void reject(RejState& st, double g2, double s2, double R2) {
  st.R = R2;
  if (s2 > 0.0) {
    st.g = g2;
    st.s = s2;
  }
}
// The draft mass left, R = (draft sum outside the rejected tokens) / QS.
__device__ __forceinline__ double left_mass(double keep, double QS) {
  return QS > 0.0 ? keep / QS : 1.0;
}
// One entry of a mass table, per (level, sequence, node, chunk).
struct MassEntry {
  double mass;  // the chunk's residual mass after the level-th rejection
  double keep;  // the chunk's draft sum outside the first `level` children's tokens
};

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

// Whether token v is marked in the rejected-token bitmap.
__device__ __forceinline__ bool marked(const uint32_t* bm, int v) { return (bm[v >> 5] >> (v & 31)) & 1u; }

// One thread's share of sum_v R(v), and in `keep` of the draft sum over the
// tokens not marked in `bm`: float4 loads of both rows in batches of kBatch,
// all issued before any use (a strided, coalesced layout; rows of a
// vocabulary that is not a multiple of 4 take the scalar path).
constexpr int kBatch = 4;
__device__ float residual_pass(const float* __restrict__ l, const float* __restrict__ q, int Voc,
                               int t, const Residual& r, const uint32_t* bm, double& keep) {
  float part = 0.f;
  keep = 0.0;
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
        const int i = i0 + k * kWalkThreads;
        if (i < n4) {
          part += residual_elem(lv[k].x, qv[k].x, r);
          part += residual_elem(lv[k].y, qv[k].y, r);
          part += residual_elem(lv[k].z, qv[k].z, r);
          part += residual_elem(lv[k].w, qv[k].w, r);
          const uint32_t bits = bm[i >> 3] >> (4 * (i & 7));  // tokens 4i .. 4i+3
          keep += (bits & 1u) ? 0.0 : static_cast<double>(qv[k].x);
          keep += (bits & 2u) ? 0.0 : static_cast<double>(qv[k].y);
          keep += (bits & 4u) ? 0.0 : static_cast<double>(qv[k].z);
          keep += (bits & 8u) ? 0.0 : static_cast<double>(qv[k].w);
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
      for (int k = 0; k < kBatch; ++k) {
        const int v = v0 + k * kWalkThreads;
        if (v < Voc) {
          part += residual_elem(lv[k], qv[k], r);
          keep += marked(bm, v) ? 0.0 : static_cast<double>(qv[k]);
        }
      }
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
  // (the chunk's rescale in float: its exponent is a float difference)
  double zl = m_l != -INFINITY ? static_cast<double>(st.z * __expf(m_l - Mf)) : 0.0;
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
  r.b = static_cast<float>(kLog2e * (static_cast<double>(nt.Mf) +
                                      static_cast<double>(__logf(static_cast<float>(nt.Z)))));
  r.gq = g > 0.0 && nt.QS > 0.0 ? static_cast<float>(g / nt.QS) : 0.f;
  return r;
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

// Per (node with at least `level` children, chunk): the residual mass
// sum_v max(P(v) - g Q(v), 0) over the chunk after the node's level-th
// rejection, with the walk's own parameters and element arithmetic.  Level 1
// is at g = 1; level k replays the node's first k - 1 rejections from the
// totals of levels 1 .. k - 1 (tables `mass` + (l - 1) * level_stride), the
// way the walk advances its state.  Other nodes' entries read as 0.
__global__ void __launch_bounds__(kStatThreads) sample_mass_kernel(
    const float* __restrict__ logits, const float* __restrict__ draft_probs,
    const int32_t* __restrict__ draft_tokens, const int32_t* __restrict__ parents,
    const int32_t* __restrict__ n_nodes, int Nmax, int Voc, float inv_t,
    const NodeStats* __restrict__ ws, MassEntry* __restrict__ mass, int level,
    int64_t level_stride, const int32_t* status) {
  static_assert(kStatThreads >= LTD_MAX_NODES, "one thread per node for the child bits");
  __shared__ NodeTotals nt_s;
  __shared__ uint64_t kids_s[kStatThreads / kWave];
  __shared__ int tok_s[kLevels];
  __shared__ int ctok_s[LTD_MAX_NODES];  // tokens of the node's children
  __shared__ double g_s;
  __shared__ double red_s[kStatThreads / kWave];
  __shared__ double keep_s[kStatThreads / kWave];
  if (halted(status)) return;
  const int chunk = blockIdx.x, i = blockIdx.y, b = blockIdx.z;
  const int chunks = gridDim.x;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int n = min(max(n_nodes[b], 1), Nmax);
  if (i >= n) return;  // uniform for the block
  const int64_t nb = static_cast<int64_t>(b) * Nmax;
  const int64_t row = (nb + i) * Voc;
  MassEntry* out = mass + (level - 1) * level_stride + (nb + i) * chunks + chunk;
  {  // the node's children as bits, thread j for node j, and their tokens
    const bool kid = t < n && t > i && link(parents, nb, t) == i;
    const int tok = min(max(draft_tokens[nb + min(t, n - 1)], 0), Voc - 1);
    const uint64_t bits = __ballot(kid);
    if (lane == 0) kids_s[w] = bits;
    if (kid) ctok_s[t] = tok;
  }
  if (w == 0) {
    const NodeTotals nt = merge_node_stats(ws + (nb + i) * chunks, chunks, lane);
    if (lane == 0) nt_s = nt;
  }
  __syncthreads();
  int n_kids = 0;
#pragma unroll
  for (int word = 0; word < kStatThreads / kWave; ++word) n_kids += __popcll(kids_s[word]);
  if (n_kids < level) {  // uniform: the node never rejects `level` times
    if (t == 0) *out = MassEntry{0.0, 0.0};
    return;
  }
  if (t == 0) {  // its first `level` children's tokens, in ascending order
    int nk = 0;
    for (int word = 0; word < kStatThreads / kWave && nk < level; ++word) {
      uint64_t bits = kids_s[word];
      while (bits != 0 && nk < level) {
        const int c = word * kWave + __ffsll(static_cast<long long>(bits)) - 1;
        bits &= bits - 1;
        tok_s[nk++] = ctok_s[c];
      }
    }
  }
  __syncthreads();
  const NodeTotals nt = nt_s;
  // wave 0's loads for the replay first, then every thread's share of the
  // chunk's rows, in flight while the residual's g is worked out
  double prev_mass[kLevels - 1], prev_keep[kLevels - 1];
  if (w == 0) {
#pragma unroll
    for (int k = 0; k < kLevels - 1; ++k) {
      prev_mass[k] = 0.0;
      prev_keep[k] = 0.0;
      if (k < level - 1 && lane < chunks) {
        const MassEntry e = mass[k * level_stride + (nb + i) * chunks + lane];
        prev_mass[k] = e.mass;
        prev_keep[k] = e.keep;
      }
    }
  }
  const int base = chunk * kChunk;
  float l[kPerThread], q[kPerThread];
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int64_t v = row + min(base + k * kStatThreads + t, Voc - 1);
    l[k] = logits[v];
    q[k] = draft_probs[v];
  }
  if (w == 0) {  // g after `level` rejections: the walk's state, replayed
    RejState st{0.0, 1.0, 1.0};
#pragma unroll
    for (int k = 0; k < kLevels - 1; ++k) {
      if (k < level - 1) {
        const double tot = wave_sum_d(prev_mass[k], lane);
        const double keep = wave_sum_d(prev_keep[k], lane);
        const double g2 = next_g(st);
        reject(st, g2, tot, left_mass(keep, nt.QS));
      }
    }
    if (lane == 0) g_s = next_g(st);
  }
  __syncthreads();
  const Residual r = residual_params(nt, inv_t, g_s);
  // The draft sum outside the first `level` children's tokens: a sum of
  // non-negative terms, so float partials keep it to a relative error, however
  // small it is (the difference it replaces would lose every digit).
  int ex[kLevels];
#pragma unroll
  for (int j = 0; j < kLevels; ++j) ex[j] = j < level ? tok_s[j] : -1;
  double d = 0.0;
  float kf = 0.f;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int v = base + k * kStatThreads + t;
    if (v < Voc) {
      d += static_cast<double>(residual_elem(l[k], q[k], r));
      bool gone = false;
#pragma unroll
      for (int j = 0; j < kLevels; ++j) gone = gone || ex[j] == v;
      kf += gone ? 0.f : q[k];
    }
  }
  d = wave_sum_d(d, lane);
  const double kp = static_cast<double>(wave_sum(kf));
  if (lane == 0) {
    red_s[w] = d;
    keep_s[w] = kp;
  }
  __syncthreads();
  if (t == 0) {
    double a = 0.0, kk = 0.0;
#pragma unroll
    for (int k = 0; k < kStatThreads / kWave; ++k) {
      a += red_s[k];
      kk += keep_s[k];
    }
    *out = MassEntry{a, kk};
  }
}

// Whether node u has a child, by one wave over the parent links in LDS.
__device__ __forceinline__ bool child_any(const int32_t* par_s, int n, int u, int lane) {
  bool any = false;
  for (int j = u + 1 + lane; j < n; j += kWave) any = any || par_s[j] == u;
  return __ballot(any) != 0;
}

// What the walk needs of a node, loaded and merged by one wave (lane c takes
// chunk c): its softmax maximum, normaliser and draft sum, the totals of its
// tabled residual masses, and its chunk masses (the softmax's and the
// tables').  0 for rejections the node cannot have.  The loads and the merge
// are separate steps, so a wave can have a node's loads in flight while it
// works on something else.
// node_out: [0] M, [1] Z, [2] QS, [3 + k] the residual mass after the node's
// (k+1)-th rejection, [3 + kLevels + k] the draft sum left after it.
constexpr int kNodeVals = 3 + 2 * kLevels;
struct NodeLoads {
  NodeStats st;
  MassEntry mk[kLevels];
};
__device__ __forceinline__ NodeLoads node_loads(const NodeStats* __restrict__ ws,
                                                const MassEntry* __restrict__ mass,
                                                int64_t level_stride, int64_t nb, int v, int chunks,
                                                int lane) {
  NodeLoads r;
  const int cl = min(lane, chunks - 1);
  r.st = ws[(nb + v) * chunks + cl];
#pragma unroll
  for (int k = 0; k < kLevels; ++k) r.mk[k] = mass[k * level_stride + (nb + v) * chunks + cl];
  return r;
}
__device__ void node_merge(const NodeLoads& ld, const int32_t* par_s, int n, int v, int chunks,
                           int lane, double* node_out, double (*mass_out)[kLevels + 1]) {
  const NodeStats st = ld.st;
  const NodeTotals nt = merge_node_stats_of(st, chunks, lane);
  const bool kids = child_any(par_s, n, v, lane);
  const double m0c =
      st.m != -INFINITY ? static_cast<double>(st.z * __expf(st.m - nt.Mf)) / nt.Z : 0.0;
  if (lane < chunks) mass_out[lane][0] = m0c;
  double tot[kLevels], keep[kLevels];
#pragma unroll
  for (int k = 0; k < kLevels; ++k) {
    const double mc = kids ? ld.mk[k].mass : 0.0;
    const double kc = kids ? ld.mk[k].keep : 0.0;
    if (lane < chunks) mass_out[lane][k + 1] = mc;
    tot[k] = wave_sum_d(lane < chunks ? mc : 0.0, lane);
    keep[k] = wave_sum_d(lane < chunks ? kc : 0.0, lane);
  }
  if (lane == 0) {
    node_out[0] = nt.Mf;
    node_out[1] = nt.Z;
    node_out[2] = nt.QS;
#pragma unroll
    for (int k = 0; k < kLevels; ++k) {
      node_out[3 + k] = tot[k];
      node_out[3 + kLevels + k] = keep[k];
    }
  }
}

__global__ void __launch_bounds__(kWalkThreads) sample_walk_kernel(
    const float* __restrict__ logits, const float* __restrict__ draft_probs,
    const int32_t* __restrict__ draft_tokens, const int32_t* __restrict__ parents,
    const int32_t* __restrict__ n_nodes, const float* __restrict__ uniforms, int Nmax, int Voc,
    float inv_t, const NodeStats* __restrict__ ws, const MassEntry* __restrict__ mass,
    int64_t level_stride, int chunks, int32_t* __restrict__ accepted,
    int32_t* __restrict__ out_tokens, int32_t* __restrict__ n_accepted, const int32_t* status) {
  __shared__ int32_t par_s[LTD_MAX_NODES];
  __shared__ int32_t tok_s[LTD_MAX_NODES];
  __shared__ uint64_t child_s[LTD_MAX_NODES / kWave];
  __shared__ int32_t path_s[LTD_MAX_NODES];
  __shared__ int32_t removed_s[LTD_MAX_NODES];
  __shared__ float cl_s[LTD_MAX_NODES], cq_s[LTD_MAX_NODES], cr_s[LTD_MAX_NODES];  // child inputs
  __shared__ double red_s[kWalkWaves];
  // The current node's M, Z, QS and tabled residual totals, and its chunk
  // masses ([0] the softmax's, [k] after its k-th rejection).
  __shared__ double node_s[1][kNodeVals];
  __shared__ double mass_s[1][LTD_SAMPLING_MAX_CHUNKS][kLevels + 1];
  __shared__ double target_s;  // the bonus search: mass left to pass in [lo_s, hi_s)
  __shared__ double seg_s[kWave];  // the bonus search's segment sums
  __shared__ int lo_s, hi_s;
  // The rejected tokens of the current node, one bit per vocabulary entry.
  __shared__ uint32_t gone_s[LTD_SAMPLING_MAX_CHUNKS * kChunk / 32];
  if (halted(status)) return;
  const int b = blockIdx.x;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  for (int k = t; k < (Voc + 31) / 32; k += kWalkThreads) gone_s[k] = 0u;
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
    // Every load first: each child's accept-test inputs (the target logit and
    // draft probability of its token, its uniform; thread j for node j) and,
    // in wave 0, the node's stats; then the children as bits of 64-node
    // words and the node's merged data.
    const bool is_child = t < n && t < LTD_MAX_NODES && par_s[t] == u && t > u;
    float cl = 0.f, cq = 0.f, cr = 0.f;
    if (is_child) {
      const int x = tok_s[t];
      cl = logits[row + x];
      cq = draft_probs[row + x];
      cr = uniforms[(nb + t) * 2];
    }
    NodeLoads ld{};
    if (w == 0) ld = node_loads(ws, mass, level_stride, nb, u, chunks, lane);
    if (t < LTD_MAX_NODES) {
      const uint64_t m = __ballot(is_child);
      if (lane == 0) child_s[w] = m;
      if (is_child) {
        cl_s[t] = cl;
        cq_s[t] = cq;
        cr_s[t] = cr;
      }
    }
    if (w == 0) node_merge(ld, par_s, n, u, chunks, lane, node_s[0], mass_s[0]);
    __syncthreads();
    const NodeTotals nt{static_cast<float>(node_s[0][0]), node_s[0][1], node_s[0][2]};
    const float Mf = nt.Mf;
    const double Z = nt.Z;
    const double QS = nt.QS;
    const double inv_z = 1.0 / Z;
    Residual res = residual_params(nt, inv_t, 0.0);

    RejState st{0.0, 1.0, 1.0};  // the residual after the rejections so far
    int lvl = 0;                 // the mass table holding that residual (-1: none)
    int n_removed = 0;
    int next = -1;
    for (int word = 0; word < LTD_MAX_NODES / kWave && next < 0; ++word) {
      uint64_t bits = child_s[word];
      while (bits != 0 && next < 0) {
        const int c = word * kWave + __ffsll(static_cast<long long>(bits)) - 1;
        bits &= bits - 1;
        const int x = tok_s[c];
        // P(x) from a float exponential (its argument is float already; the
        // walk's hot chain avoids the double exp and divisions)
        const double Px = static_cast<double>(__expf(cl_s[c] * inv_t - Mf)) * inv_z;
        const double Qx = QS > 0.0 ? static_cast<double>(cq_s[c]) / QS : 0.0;
        bool removed = false;
        for (int k = 0; k < n_removed; ++k) removed = removed || removed_s[k] == x;
        // accept when r Q_k(x) < P_k(x), i.e. r Q(x) s < max(P(x) - g Q(x), 0) R
        // (Q_k(x) = 0 for a token rejected before, and for every token once
        // R = 0)
        const double Pres = fmax(Px - st.g * Qx, 0.0);
        const double r = static_cast<double>(cr_s[c]);
        const bool accept = removed || st.R <= 0.0 ? Pres > 0.0 : r * Qx * st.s < Pres * st.R;
        if (accept) {
          next = c;
          break;
        }
        // rejected: the next residual's mass, from the tables for the
        // node's first kLevels rejections, else one pass over the vocabulary
        const double g2 = next_g(st);
        double s2, R2;
        if (t == 0) gone_s[x >> 5] |= 1u << (x & 31);
        if (n_removed < kLevels) {
          s2 = node_s[0][3 + n_removed];
          R2 = left_mass(node_s[0][3 + kLevels + n_removed], QS);
        } else {
          res = residual_params(nt, inv_t, g2);
          __syncthreads();  // x's bit
          double keep;
          const float part =
              residual_pass(logits + row, draft_probs + row, Voc, t, res, gone_s, keep);
          s2 = block_sum(static_cast<double>(part), red_s, lane, w);
          R2 = left_mass(block_sum(keep, red_s, lane, w), QS);
        }
        // (every thread keeps the list, with the same values: no barrier)
        removed_s[n_removed] = x;
        reject(st, g2, s2, R2);
        if (s2 > 0.0) lvl = n_removed < kLevels ? n_removed + 1 : -1;
        ++n_removed;
      }
    }
    if (next >= 0) {
      if (t == 0) {
        path_s[len] = next;
        for (int k = 0; k < n_removed; ++k) gone_s[removed_s[k] >> 5] = 0u;  // the new node's start
      }
      ++len;
      u = next;
      __syncthreads();  // the node's data, child_s and the bitmap are rewritten for the new node
      continue;
    }

    // The bonus: inverse CDF of R = max(P - g Q, 0) at uniforms[u][1] times
    // its mass.  The range holding the target is narrowed in levels: the 16
    // waves sum R over 16 equal segments of it, thread 0 scans the sums and
    // keeps the segment where the mass passes the target; at 64 tokens or
    // fewer wave 0 takes an inclusive scan and the first token past the
    // target.  Where rounding leaves the target at or past a level's sum, the
    // last segment (token) with mass is taken, as the plain scan would.
    const bool use_q = st.g > 0.0;
    res = residual_params(nt, inv_t, st.g);
    const bool vec = (Voc & 3) == 0 && (reinterpret_cast<uintptr_t>(logits + row) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(draft_probs + row) & 15) == 0;
    int lo = 0, hi = Voc;
    bool first = true;  // no level yet: the final scan sets the target itself
    if (lvl >= 0) {  // the first level from a mass table's chunks
      if (t == 0) {
        double total = 0.0;
        for (int c = 0; c < chunks; ++c) total += mass_s[0][c][lvl];
        const double target = static_cast<double>(uniforms[(nb + u) * 2 + 1]) * total;
        int pick = -1, last = -1;
        double cum = 0.0, before = 0.0, upto_last = 0.0, run = 0.0;
        for (int c = 0; c < chunks && pick < 0; ++c) {
          const double mc = mass_s[0][c][lvl];
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
      if (vec && span <= kWave * kWave) {
        // At most 4096 tokens: 64 segments of at most 64 tokens in one step,
        // 4 per wave, 16 lanes and one float4 per lane and segment; wave 0
        // scans the 64 sums.
        const int seg = ((span + 4 * kWave - 1) / (4 * kWave)) * 4;
        const int k = 4 * w + (lane >> 4);  // this lane's segment
        const int v = lo + k * seg + 4 * (lane & 15);
        float part = 0.f;
        if (v < min(lo + (k + 1) * seg, hi)) {
          const float4 lv = *reinterpret_cast<const float4*>(logits + row + v);
          const float4 qv = use_q ? *reinterpret_cast<const float4*>(draft_probs + row + v)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
          part = residual_elem(lv.x, qv.x, res);
          part += residual_elem(lv.y, qv.y, res);
          part += residual_elem(lv.z, qv.z, res);
          part += residual_elem(lv.w, qv.w, res);
        }
        double sum = static_cast<double>(part);
#pragma unroll
        for (int d = 8; d >= 1; d >>= 1) {  // over the segment's 16 lanes
          uint64_t o;
          const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(sum));
          switch (d) {
            case 8: o = lane_xor_u64<8>(bits, lane); break;
            case 4: o = lane_xor_u64<4>(bits, lane); break;
            case 2: o = lane_xor_u64<2>(bits, lane); break;
            default: o = lane_xor_u64<1>(bits, lane);
          }
          sum += __longlong_as_double(static_cast<long long>(o));
        }
        if (k < kWave && (lane & 15) == 0) seg_s[k] = sum;
        __syncthreads();
        if (w == 0) {
          const double sk = seg_s[lane];
          double incl = sk;
#pragma unroll
          for (int d = 1; d < kWave; d <<= 1) {
            const double o = __shfl_up(incl, d, kWave);
            if (lane >= d) incl += o;
          }
          const double target = first ? static_cast<double>(uniforms[(nb + u) * 2 + 1]) *
                                            __shfl(incl, kWave - 1, kWave)
                                      : target_s;
          const uint64_t past = __ballot(incl > target && sk > 0.0);
          const uint64_t withm = __ballot(sk > 0.0);
          // (past the end by rounding: the last segment with mass; none: token 0)
          const int pick = past != 0 ? __ffsll(static_cast<long long>(past)) - 1
                                     : (withm != 0 ? 63 - __clzll(static_cast<long long>(withm)) : -1);
          const double before = pick >= 0 ? __shfl(incl - sk, pick, kWave) : 0.0;
          if (lane == 0) {
            if (pick < 0) {
              lo_s = 0;
              hi_s = 0;
            } else {
              lo_s = min(lo + pick * seg, hi);
              hi_s = min(lo + (pick + 1) * seg, hi);
            }
            target_s = target - before;
          }
        }
        __syncthreads();
        lo = lo_s;
        hi = hi_s;
        continue;
      }
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
  return (sizeof(NodeStats) + kLevels * sizeof(MassEntry)) * static_cast<size_t>(B) * Nmax *
         sampling_chunks(Voc);
}

hipError_t launch_sampling(const float* logits, const float* draft_probs,
                           const int32_t* draft_tokens, const int32_t* parents,
                           const int32_t* n_nodes, const float* uniforms, int B, int Nmax,
                           int Voc, float temperature, int32_t* accepted_nodes,
                           int32_t* out_tokens, int32_t* n_accepted, void* workspace,
                           const int32_t* status, hipStream_t stream) {
  const int chunks = sampling_chunks(Voc);
  const int64_t level_stride = static_cast<int64_t>(B) * Nmax * chunks;  // entries per table
  auto* ws = static_cast<NodeStats*>(workspace);
  auto* mass = reinterpret_cast<MassEntry*>(ws + level_stride);
  const float inv_t = 1.0f / temperature;
  hipLaunchKernelGGL(sample_stats_kernel, dim3(chunks, Nmax, B), dim3(kStatThreads), 0, stream,
                     logits, draft_probs, parents, n_nodes, Nmax, Voc, inv_t, ws, status);
  // level k needs the totals of level k - 1: one launch per level
  for (int level = 1; level <= kLevels; ++level)
    hipLaunchKernelGGL(sample_mass_kernel, dim3(chunks, Nmax, B), dim3(kStatThreads), 0, stream,
                       logits, draft_probs, draft_tokens, parents, n_nodes, Nmax, Voc, inv_t, ws,
                       mass, level, level_stride, status);
  hipLaunchKernelGGL(sample_walk_kernel, dim3(B), dim3(kWalkThreads), 0, stream, logits,
                     draft_probs, draft_tokens, parents, n_nodes, uniforms, Nmax, Voc, inv_t, ws,
                     mass, level_stride, chunks, accepted_nodes, out_tokens, n_accepted, status);
  return hipGetLastError();
}

}  // namespace ltd
