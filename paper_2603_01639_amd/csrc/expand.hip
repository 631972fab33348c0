// One round of draft tree expansion (section 3.2, "Draft Tree Generation"):
// every frontier node's W most probable tokens become its children, scored by
// cumulative path log-probability, and the W_next best children become the
// next frontier.  The draft model's logits are the input.
//
//   expand_partial_kernel  grid (vocab chunks of 4096, F, B), 256 threads:
//                          each thread holds 16 logits of the chunk as packed
//                          keys (order-preserving value bits above the
//                          complemented token index, so a larger key is a
//                          larger logit or, on ties, a lower index).  It
//                          writes the chunk's online-softmax partial (max,
//                          sum of exp) and its W largest keys: each wave
//                          finds its own W by W rounds of a wave argmax (only
//                          the lane that owned the winner rescans its 16
//                          keys), and one wave merges the four lists;
//   expand_merge_kernel    one wave per (frontier node, sequence): the chunks'
//                          partials give the node's log-sum-exp (double), and
//                          a k-way merge of the chunks' sorted lists gives its
//                          W children (lane c walks chunk c's list in LDS;
//                          W rounds of a wave argmax over the heads), which go
//                          into the pool;
//   expand_beam_kernel     one wave per sequence: the W_next best of the F*W
//                          children (W_next rounds of a wave argmax) become the
//                          next frontier, and the pool size advances.
//
// The chunk pass reads the logits once (HBM bound: 4 bytes per vocabulary
// entry per frontier node); the merge touches a few KB.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kThreads = 256;
constexpr int kChunk = 4096;
constexpr int kPerThread = kChunk / kThreads;  // 16
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxW = LTD_EXPAND_MAX_W;
constexpr int kBeamKeys = LTD_EXPAND_MAX_CHILDREN / kWave;
static_assert(LTD_EXPAND_MAX_CHUNKS <= kWave, "one chunk partial a lane in the merge");
static_assert(kThreads / kWave * kMaxW <= kWave, "the four wave lists fit one wave");

__device__ __forceinline__ uint32_t orderable(float v) {
  const uint32_t u = __float_as_uint(v + 0.0f);  // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_orderable(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
__device__ __forceinline__ uint64_t pack(float v, uint32_t idx) {
  return (static_cast<uint64_t>(orderable(v)) << 32) | (0xFFFFFFFFu - idx);
}
__device__ __forceinline__ uint32_t key_index(uint64_t k) {
  return 0xFFFFFFFFu - static_cast<uint32_t>(k);
}

// (m, z) pairs: z is a sum of exp(x - m).
__device__ __forceinline__ void lse_combine(float& m, float& z, float m2, float z2) {
  const float mx = fmaxf(m, m2);
  if (mx == -INFINITY) return;  // both empty
  z = z * __expf(m - mx) + z2 * __expf(m2 - mx);
  m = mx;
}

template <bool kVec4>
__global__ void __launch_bounds__(kThreads) expand_partial_kernel(const float* __restrict__ logits,
                                                                  int F, int Voc, int W,
                                                                  uint64_t* __restrict__ ws_keys,
                                                                  float2* __restrict__ ws_mz,
                                                                  const int32_t* status) {
  __shared__ uint64_t wave_list_s[kWaves][kMaxW];
  __shared__ float2 wave_mz_s[kWaves];
  if (halted(status)) return;
  const int chunk = blockIdx.x, f = blockIdx.y, b = blockIdx.z;
  const int chunks = gridDim.x;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const float* row = logits + (static_cast<int64_t>(b) * F + f) * Voc;
  const int base = chunk * kChunk;

  // 16 logits a thread: element base + j*1024 + t*4 + e (coalesced float4s)
  float v[kPerThread];
  if constexpr (kVec4) {
#pragma unroll
    for (int j = 0; j < kPerThread / 4; ++j) {
      const int i0 = base + j * kThreads * 4 + t * 4;
      const float4 x = i0 < Voc ? *reinterpret_cast<const float4*>(row + i0)
                                : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      v[4 * j] = x.x;
      v[4 * j + 1] = x.y;
      v[4 * j + 2] = x.z;
      v[4 * j + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kPerThread / 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = base + j * kThreads * 4 + t * 4 + e;
        const float x = row[min(i, Voc - 1)];
        v[4 * j + e] = i < Voc ? x : -INFINITY;
      }
  }
  // keys: order-preserving value bits; a lane's 16 elements have increasing
  // token indices in q order, so scanning with a strict > keeps the lowest
  // index among equal values
  uint32_t key[kPerThread];
  float m = -INFINITY;
#pragma unroll
  for (int q = 0; q < kPerThread; ++q) {
    const int i = base + (q / 4) * kThreads * 4 + t * 4 + (q % 4);
    key[q] = i < Voc ? orderable(v[q]) : 0;
    m = fmaxf(m, v[q]);
  }
  float z = 0.f;
  if (m != -INFINITY) {
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) z += __expf(v[q] - m);
  }
  // softmax partial of the chunk
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    float m2, z2;
    switch (d) {
      case 32: m2 = lane_xor_f<32>(m, lane); z2 = lane_xor_f<32>(z, lane); break;
      case 16: m2 = lane_xor_f<16>(m, lane); z2 = lane_xor_f<16>(z, lane); break;
      case 8: m2 = lane_xor_f<8>(m, lane); z2 = lane_xor_f<8>(z, lane); break;
      case 4: m2 = lane_xor_f<4>(m, lane); z2 = lane_xor_f<4>(z, lane); break;
      case 2: m2 = lane_xor_f<2>(m, lane); z2 = lane_xor_f<2>(z, lane); break;
      default: m2 = lane_xor_f<1>(m, lane); z2 = lane_xor_f<1>(z, lane);
    }
    lse_combine(m, z, m2, z2);
  }
  if (lane == 0) wave_mz_s[w] = make_float2(m, z);

  // each wave's W largest (value, index) pairs by W rounds of a wave argmax;
  // only the lane that owned the winner rescans (a 4-level tree over its 16)
  // (taken is a bit per element; the array itself is never written, which
  // keeps it in plain registers)
  uint32_t taken = 0;
  auto lane_best = [&](uint32_t& bk, int& bq) {
    uint32_t k8[8];
    int q8[8];
#pragma unroll
    for (int a = 0; a < 8; ++a) {
      const uint32_t k0 = (taken >> (2 * a)) & 1 ? 0u : key[2 * a];
      const uint32_t k1 = (taken >> (2 * a + 1)) & 1 ? 0u : key[2 * a + 1];
      const bool hi = k1 > k0;
      k8[a] = hi ? k1 : k0;
      q8[a] = hi ? 2 * a + 1 : 2 * a;
    }
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const bool hi = k8[2 * a + 1] > k8[2 * a];
      k8[a] = hi ? k8[2 * a + 1] : k8[2 * a];
      q8[a] = hi ? q8[2 * a + 1] : q8[2 * a];
    }
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const bool hi = k8[2 * a + 1] > k8[2 * a];
      k8[a] = hi ? k8[2 * a + 1] : k8[2 * a];
      q8[a] = hi ? q8[2 * a + 1] : q8[2 * a];
    }
    const bool hi = k8[1] > k8[0];
    bk = hi ? k8[1] : k8[0];
    bq = hi ? q8[1] : q8[0];
  };
  uint32_t ck;
  int cq;
  lane_best(ck, cq);
  const int q_base = base + t * 4;  // index of element q: q_base + (q/4)*1024 + q%4
  for (int r = 0; r < W; ++r) {
    const uint32_t ci = static_cast<uint32_t>(q_base + (cq / 4) * kThreads * 4 + (cq % 4));
    uint32_t wk;
    const uint32_t wi = wave_argmax(ck, ci, lane, &wk);
    if (lane == 0) wave_list_s[w][r] = (static_cast<uint64_t>(wk) << 32) | (0xFFFFFFFFu - wi);
    if (wk != 0 && ck == wk && ci == wi) {  // the owner takes it and rescans
      taken |= 1u << cq;
      lane_best(ck, cq);
    }
  }
  __syncthreads();
  if (w == 0) {
    // kWaves * W <= 64 candidates, one a lane
    const int n_cand = kWaves * W;
    const uint64_t c = lane < n_cand ? wave_list_s[lane / W][lane % W] : 0;
    uint32_t ck2 = static_cast<uint32_t>(c >> 32);
    const uint32_t ci2 = key_index(c);
    uint64_t* out = ws_keys + ((static_cast<int64_t>(b) * F + f) * chunks + chunk) * W;
    for (int r = 0; r < W; ++r) {
      uint32_t wk;
      const uint32_t wi = wave_argmax(ck2, ci2, lane, &wk);
      if (lane == 0) out[r] = wk == 0 ? 0 : (static_cast<uint64_t>(wk) << 32) | (0xFFFFFFFFu - wi);
      if (wk != 0 && ck2 == wk && ci2 == wi) ck2 = 0;
    }
    if (lane == 0) {
      float mb = wave_mz_s[0].x, zb = wave_mz_s[0].y;
#pragma unroll
      for (int k = 1; k < kWaves; ++k) lse_combine(mb, zb, wave_mz_s[k].x, wave_mz_s[k].y);
      ws_mz[(static_cast<int64_t>(b) * F + f) * chunks + chunk] = make_float2(mb, zb);
    }
  }
}

// One wave per (frontier node, sequence): the node's log-sum-exp and its W
// children by a k-way merge of the chunks' sorted lists (lane c walks chunk
// c's list in LDS with a pointer; W rounds of a wave argmax over the heads).
__global__ void __launch_bounds__(kWave) expand_merge_kernel(
    const uint64_t* __restrict__ ws_keys, const float2* __restrict__ ws_mz, int chunks,
    const int32_t* __restrict__ frontier, int F, int W, float* __restrict__ scores,
    int32_t* __restrict__ pool_parents, int32_t* __restrict__ pool_tokens,
    const int32_t* __restrict__ pool_size, int Vpool, const int32_t* status) {
  __shared__ uint64_t list_s[LTD_EXPAND_MAX_CHUNKS * kMaxW];
  if (halted(status)) return;
  const int f = blockIdx.x, b = blockIdx.y;
  const int lane = threadIdx.x;
  const int64_t node = static_cast<int64_t>(b) * F + f;
  const int64_t pb = static_cast<int64_t>(b) * Vpool;
  const int n_keys = chunks * W;

  // every load is issued up front: the chunk partials (one a lane), the
  // chunks' lists (staged to LDS), the pool size and the parent
  const float2 pm = ws_mz[node * chunks + min(lane, chunks - 1)];
  uint64_t stage[kMaxW];
#pragma unroll
  for (int q = 0; q < kMaxW; ++q) {
    const int i = lane + q * kWave;
    stage[q] = ws_keys[node * n_keys + min(i, n_keys - 1)];
  }
  const int first = pool_size[b];
  const int32_t fnode = frontier[node];
  const int parent = min(max(fnode, 0), Vpool - 1);
  const double pscore = static_cast<double>(scores[pb + parent]);
#pragma unroll
  for (int q = 0; q < kMaxW; ++q) {
    const int i = lane + q * kWave;
    if (i < n_keys) list_s[i] = stage[q];
  }

  // log-sum-exp of the node's logits from the chunk partials (double)
  const float m_l = lane < chunks ? pm.x : -INFINITY;
  float Mf = m_l;
  Mf = fmaxf(Mf, lane_xor_f<32>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<16>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<8>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<4>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<2>(Mf, lane));
  Mf = fmaxf(Mf, lane_xor_f<1>(Mf, lane));
  const double M = static_cast<double>(Mf);
  double Z = m_l != -INFINITY ? static_cast<double>(pm.y) * exp(static_cast<double>(m_l) - M) : 0.0;
  auto add_xor = [&](uint64_t o) { Z += __longlong_as_double(static_cast<long long>(o)); };
  add_xor(lane_xor_u64<32>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
  add_xor(lane_xor_u64<16>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
  add_xor(lane_xor_u64<8>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
  add_xor(lane_xor_u64<4>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
  add_xor(lane_xor_u64<2>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
  add_xor(lane_xor_u64<1>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
  const double lse = M + log(Z);
  __syncthreads();  // the lists are in LDS

  // k-way merge: lane c's head is its chunk's best key not taken yet
  int ptr = 0;
  for (int r = 0; r < W; ++r) {
    const uint64_t head = lane < chunks && ptr < W ? list_s[lane * W + ptr] : 0;
    const uint32_t hk = static_cast<uint32_t>(head >> 32);
    const uint32_t hi = key_index(head);
    uint32_t wk;
    const uint32_t wi = wave_argmax(hk, hi, lane, &wk);
    if (head != 0 && hk == wk && hi == wi) ++ptr;  // the owner moves on
    const float sc = static_cast<float>(pscore + (static_cast<double>(from_orderable(wk)) - lse));
    if (lane == 0) {
      const int64_t o = static_cast<int64_t>(first) + f * W + r;
      if (o >= 0 && o < Vpool) {  // unvalidated pool sizes stay in bounds
        scores[pb + o] = sc;
        pool_parents[pb + o] = fnode;
        pool_tokens[pb + o] = static_cast<int32_t>(wi);
      }
    }
  }
}

// One wave per sequence: the next frontier is the W_next children of
// highest score (lower pool index on ties), by W_next rounds of a wave argmax;
// then the pool size advances.
__global__ void __launch_bounds__(kWave) expand_beam_kernel(const float* __restrict__ scores,
                                                            int F, int W, int W_next,
                                                            int32_t* __restrict__ pool_size,
                                                            int Vpool,
                                                            int32_t* __restrict__ new_frontier,
                                                            const int32_t* status) {
  if (halted(status)) return;
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int n_children = F * W;
  const int first = pool_size[b];
  const int64_t pb = static_cast<int64_t>(b) * Vpool;
  // up to kBeamKeys children a lane; taken is a bit per child
  uint32_t k[kBeamKeys];
#pragma unroll
  for (int q = 0; q < kBeamKeys; ++q) {
    const int c = lane + q * kWave;
    const int64_t o = static_cast<int64_t>(first) + min(c, n_children - 1);
    const float sc = scores[pb + min(max(o, int64_t{0}), static_cast<int64_t>(Vpool - 1))];
    k[q] = c < n_children ? orderable(sc) : 0;
  }
  uint32_t taken = 0;
  for (int r = 0; r < W_next; ++r) {
    uint32_t ck = 0, cc = 0xFFFFFFFFu;  // this lane's best child left (lowest c on ties)
#pragma unroll
    for (int q = 0; q < kBeamKeys; ++q) {
      const uint32_t kq = (taken >> q) & 1 ? 0u : k[q];
      if (kq > ck) {
        ck = kq;
        cc = static_cast<uint32_t>(lane + q * kWave);
      }
    }
    uint32_t wk;
    const uint32_t wc = wave_argmax(ck, cc, lane, &wk);
    if (static_cast<int>(wc) % kWave == lane && wk != 0) taken |= 1u << (wc / kWave);
    if (lane == 0) new_frontier[static_cast<int64_t>(b) * W_next + r] = first + static_cast<int>(wc);
  }
  if (lane == 0) pool_size[b] = first + n_children;
}

// Lowest (sequence << 8 | code) over every failing sequence.
__global__ void __launch_bounds__(kThreads) validate_expand_kernel(
    const int32_t* __restrict__ frontier, const int32_t* __restrict__ pool_size, int B, int F,
    int W, int Vpool, int32_t* status) {
  __shared__ int best;
  if (threadIdx.x == 0) best = 0x7FFFFFFF;
  __syncthreads();
  int key = 0x7FFFFFFF;
  for (int64_t e = threadIdx.x; e < static_cast<int64_t>(B) * F; e += kThreads) {
    const int b = static_cast<int>(e / F);
    const int n = pool_size[b];
    int code = 0;
    if (n < 1 || n > Vpool - F * W)
      code = LTD_STATUS_BAD_NNODES;
    else if (frontier[e] < 0 || frontier[e] >= n)
      code = LTD_STATUS_BAD_PARENT;
    if (code != 0) key = min(key, (b << 8) | code);
  }
  if (key != 0x7FFFFFFF) atomicMin(&best, key);
  __syncthreads();
  if (threadIdx.x == 0) *status = (best == 0x7FFFFFFF) ? 0 : (best & 0xFF);
}

}  // namespace

int expand_chunks(int Voc) { return (Voc + kChunk - 1) / kChunk; }

size_t expand_workspace_bytes(int B, int F, int Voc, int W) {
  const size_t nodes = static_cast<size_t>(B) * F * expand_chunks(Voc);
  return nodes * (sizeof(uint64_t) * W + sizeof(float2));
}

hipError_t launch_expand(const float* logits, const int32_t* frontier, int B, int F, int Voc,
                         int W, int W_next, float* scores, int32_t* pool_parents,
                         int32_t* pool_tokens, int32_t* pool_size, int Vpool,
                         int32_t* new_frontier, void* workspace, int32_t* status, bool validate,
                         hipStream_t stream) {
  const int chunks = expand_chunks(Voc);
  auto* keys = static_cast<uint64_t*>(workspace);
  auto* mz = reinterpret_cast<float2*>(keys + static_cast<size_t>(B) * F * chunks * W);
  const int32_t* st = validate ? status : nullptr;
  if (validate) {
    hipLaunchKernelGGL(validate_expand_kernel, dim3(1), dim3(kThreads), 0, stream, frontier,
                       pool_size, B, F, W, Vpool, status);
  }
  const dim3 grid(chunks, F, B);
  if (Voc % 4 == 0)
    hipLaunchKernelGGL(expand_partial_kernel<true>, grid, dim3(kThreads), 0, stream, logits, F,
                       Voc, W, keys, mz, st);
  else
    hipLaunchKernelGGL(expand_partial_kernel<false>, grid, dim3(kThreads), 0, stream, logits, F,
                       Voc, W, keys, mz, st);
  hipLaunchKernelGGL(expand_merge_kernel, dim3(F, B), dim3(kWave), 0, stream, keys, mz, chunks,
                     frontier, F, W, scores, pool_parents, pool_tokens, pool_size, Vpool, st);
  hipLaunchKernelGGL(expand_beam_kernel, dim3(B), dim3(kWave), 0, stream, scores, F, W, W_next,
                     pool_size, Vpool, new_frontier, st);
  return hipGetLastError();
}

}  // namespace ltd
