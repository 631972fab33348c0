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
//                          sum of exp) and its W largest keys, in order.  The
//                          keys are selected by a threshold: each wave ranks
//                          its 64 lane maxima, T is the largest of the four
//                          waves' W-th, every key >= T (at least W, all the
//                          top W among them) goes to LDS, and one wave ranks
//                          those candidates against each other.  Beyond 64
//                          candidates the chunk takes W rounds of a wave
//                          argmax instead;
//   expand_select_kernel   one workgroup per sequence, one wave per frontier
//                          node at a time: the chunk partials give the node's
//                          log-sum-exp (double); its W children are selected
//                          from the chunks' lists the same way (T = the W-th
//                          largest chunk head), scored, and written to the
//                          pool; then every child is ranked against the others
//                          and the W_next best become the next frontier, and
//                          the pool size advances.
//
// The chunk pass reads the logits once (HBM bound: 4 bytes per vocabulary
// entry per frontier node); the selection touches a few KB.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kThreads = 256;
constexpr int kChunk = 4096;
constexpr int kPerThread = kChunk / kThreads;  // 16
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxW = LTD_EXPAND_MAX_W;
constexpr int kSelectWaves = 16;  // waves of the selection workgroup
constexpr int kListPerLane = LTD_EXPAND_MAX_CHUNKS * kMaxW / kWave;  // chunk-list keys a lane
static_assert(LTD_EXPAND_MAX_CHUNKS <= kWave, "one chunk partial a lane in the merge");
static_assert(kThreads / kWave * kMaxW <= kWave, "the four wave lists fit one wave");

__device__ __forceinline__ uint32_t orderable(float v) {
  const uint32_t u = __float_as_uint(v + 0.0f);  // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_orderable(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
__device__ __forceinline__ uint32_t key_index(uint64_t k) {
  return 0xFFFFFFFFu - static_cast<uint32_t>(k);
}

// Exclusive prefix over the wave of a per-lane count below 32, and the wave's
// total: one ballot per bit of the count, counted below each lane by mbcnt.
__device__ __forceinline__ int wave_prefix_small(int cnt, int* total) {
  int pre = 0, tot = 0;
#pragma unroll
  for (int bit = 0; bit < 5; ++bit) {
    const uint64_t bm = __ballot((cnt >> bit) & 1);
    const int below = static_cast<int>(__builtin_amdgcn_mbcnt_hi(
        static_cast<uint32_t>(bm >> 32), __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bm), 0u)));
    pre += below << bit;
    tot += __popcll(bm) << bit;
  }
  *total = tot;
  return pre;
}

// How many of list[0..n) exceed k (LDS, read by every lane alike, two keys a
// 16-byte read: list is 16-byte aligned and list[n] is 0 when n is odd).
__device__ __forceinline__ int count_greater(const uint64_t* list, int n, uint64_t k) {
  const ulonglong2* l2 = reinterpret_cast<const ulonglong2*>(list);
  int c = 0;
#pragma unroll 2
  for (int j = 0; j < (n + 1) / 2; ++j) {
    const ulonglong2 x = l2[j];
    c += (x.x > k ? 1 : 0) + (x.y > k ? 1 : 0);
  }
  return c;
}

// The same count shared by a group of P consecutive lanes (P a power of two
// dividing 64, uniform over the wave): lane `part` of the group counts the
// pairs part, part + P, ...; every lane of the group gets the total.
__device__ __forceinline__ int group_count_greater(const uint64_t* list, int n, uint64_t k, int P,
                                                   int part) {
  const ulonglong2* l2 = reinterpret_cast<const ulonglong2*>(list);
  int c = 0;
  for (int j = part; j < (n + 1) / 2; j += P) {
    const ulonglong2 x = l2[j];
    c += (x.x > k ? 1 : 0) + (x.y > k ? 1 : 0);
  }
  for (int d = 1; d < P; d <<= 1) c += __shfl_xor(c, d, kWave);
  return c;
}

// The largest 32-bit T with at least n of the wave's values >= T (the n-th
// largest value; 0 when fewer than n lanes hold a nonzero value): one ballot
// per bit, from the top.
__device__ __forceinline__ uint32_t wave_nth_largest(uint32_t v, int n) {
  uint32_t t = 0;
#pragma unroll
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    if (__popcll(__ballot(v >= c)) >= n) t = c;
  }
  return t;
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
  __shared__ uint32_t thr_s[kWaves];  // each wave's W-th largest lane maximum
  __shared__ int cnt_s[kWaves];       // candidates per wave
  __shared__ __align__(16) uint64_t cand_s[kWave + 2];
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
  // softmax partial of the chunk (arguments are read before each combine)
  lse_combine(m, z, lane_xor_f<32>(m, lane), lane_xor_f<32>(z, lane));
  lse_combine(m, z, lane_xor_f<16>(m, lane), lane_xor_f<16>(z, lane));
  lse_combine(m, z, lane_xor_f<8>(m, lane), lane_xor_f<8>(z, lane));
  lse_combine(m, z, lane_xor_f<4>(m, lane), lane_xor_f<4>(z, lane));
  lse_combine(m, z, lane_xor_f<2>(m, lane), lane_xor_f<2>(z, lane));
  lse_combine(m, z, lane_xor_f<1>(m, lane), lane_xor_f<1>(z, lane));
  if (lane == 0) wave_mz_s[w] = make_float2(m, z);
  uint64_t* out = ws_keys + ((static_cast<int64_t>(b) * F + f) * chunks + chunk) * W;
  auto write_mz = [&]() {
    float mb = wave_mz_s[0].x, zb = wave_mz_s[0].y;
#pragma unroll
    for (int k = 1; k < kWaves; ++k) lse_combine(mb, zb, wave_mz_s[k].x, wave_mz_s[k].y);
    ws_mz[(static_cast<int64_t>(b) * F + f) * chunks + chunk] = make_float2(mb, zb);
  };

  // Threshold selection.  A wave whose W-th largest lane maximum is T has at
  // least W values >= T, so the chunk's W largest keys all have values >= T
  // (ties included).  The candidates are ranked by their packed 64-bit keys
  // (value bits, complemented index), which are unique.
  const int q_base = base + t * 4;  // index of element q: q_base + (q/4)*1024 + q%4
  uint32_t lm = 0;
#pragma unroll
  for (int q = 0; q < kPerThread; ++q) lm = max(lm, key[q]);
  const uint32_t tw = wave_nth_largest(lm, W);
  if (lane == 0) thr_s[w] = tw;
  __syncthreads();
  uint32_t T = thr_s[0];
#pragma unroll
  for (int k = 1; k < kWaves; ++k) T = max(T, thr_s[k]);
  uint32_t cmask = 0;
#pragma unroll
  for (int q = 0; q < kPerThread; ++q)
    if (key[q] != 0 && key[q] >= T) cmask |= 1u << q;
  int wtot;
  const int pre = wave_prefix_small(__popc(cmask), &wtot);
  if (lane == 0) cnt_s[w] = wtot;
  __syncthreads();
  int off = 0, total = 0;
#pragma unroll
  for (int k = 0; k < kWaves; ++k) {
    off += k < w ? cnt_s[k] : 0;
    total += cnt_s[k];
  }
  if (total <= kWave) {  // uniform: every thread read the same counts
    int p = off + pre;
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
      if ((cmask >> q) & 1) {
        const uint32_t idx = static_cast<uint32_t>(q_base + (q / 4) * kThreads * 4 + (q % 4));
        cand_s[p++] = (static_cast<uint64_t>(key[q]) << 32) | (0xFFFFFFFFu - idx);
      }
    }
    if (t == 0) cand_s[total] = 0;  // the pad of an odd count
    __syncthreads();
    // four lanes rank each candidate
    constexpr int kP = kThreads / kWave;
    const int ci = t / kP;
    const uint64_t c = ci < total ? cand_s[ci] : 0;
    const int r = group_count_greater(cand_s, total, c, kP, t % kP);
    if (t % kP == 0 && ci < total && r < W) out[r] = c;
    if (t >= total && t < W) out[t] = 0;  // a chunk with fewer than W entries
    if (t == 0) write_mz();
    return;
  }

  // More than 64 candidates (whole lanes just above T):
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
    for (int r = 0; r < W; ++r) {
      uint32_t wk;
      const uint32_t wi = wave_argmax(ck2, ci2, lane, &wk);
      if (lane == 0) out[r] = wk == 0 ? 0 : (static_cast<uint64_t>(wk) << 32) | (0xFFFFFFFFu - wi);
      if (wk != 0 && ck2 == wk && ci2 == wi) ck2 = 0;
    }
    if (lane == 0) write_mz();
  }
}

// One workgroup per sequence; wave w takes frontier nodes w, w + waves, ...
// For each: the node's log-sum-exp from the chunk partials (double), then its
// W children from the chunks' sorted lists.  T is the W-th largest chunk head
// (at least W keys are >= T, so the W largest all are); the keys >= T are
// gathered in LDS and ranked against each other, or, beyond 64 of them, taken
// by W rounds of a wave argmax.  After every node, each child is ranked
// against all F*W (score, then lower pool index) and the W_next best become
// the next frontier; the pool size advances.
__global__ void __launch_bounds__(kSelectWaves * kWave) expand_select_kernel(
    const uint64_t* __restrict__ ws_keys, const float2* __restrict__ ws_mz, int chunks,
    const int32_t* __restrict__ frontier, int F, int W, int W_next, float* __restrict__ scores,
    int32_t* __restrict__ pool_parents, int32_t* __restrict__ pool_tokens,
    int32_t* __restrict__ pool_size, int Vpool, int32_t* __restrict__ new_frontier,
    const int32_t* status) {
  __shared__ __align__(16) uint64_t head_s[kSelectWaves][kWave + 2];
  __shared__ __align__(16) uint64_t cand_s[kSelectWaves][kWave + 2];
  __shared__ __align__(16) uint64_t child_s[LTD_EXPAND_MAX_CHILDREN + 2];
  if (halted(status)) return;
  const int b = blockIdx.x;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int waves = blockDim.x / kWave;
  const int64_t pb = static_cast<int64_t>(b) * Vpool;
  const int first = pool_size[b];
  const int n_keys = chunks * W;

  for (int f = w; f < F; f += waves) {
    const int64_t node = static_cast<int64_t>(b) * F + f;
    const uint64_t* lists = ws_keys + node * n_keys;
    // every load up front: the chunk partial and head (one chunk a lane), the
    // lane's share of the lists, the parent's score
    const float2 pm = ws_mz[node * chunks + min(lane, chunks - 1)];
    const uint64_t head_l = lists[min(lane, chunks - 1) * W];
    constexpr int kEarly = 8;  // list keys a lane loads up front (W = 10: 5 needed)
    uint64_t e[kEarly];
#pragma unroll
    for (int k = 0; k < kEarly; ++k) e[k] = lists[min(lane + k * kWave, n_keys - 1)];
    const int32_t fnode = frontier[node];
    const int parent = min(max(fnode, 0), Vpool - 1);
    const double pscore = static_cast<double>(scores[pb + parent]);
    const uint64_t head = lane < chunks ? head_l : 0;

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
    double Z =
        m_l != -INFINITY ? static_cast<double>(pm.y) * exp(static_cast<double>(m_l) - M) : 0.0;
    auto add_xor = [&](uint64_t o) { Z += __longlong_as_double(static_cast<long long>(o)); };
    add_xor(lane_xor_u64<32>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
    add_xor(lane_xor_u64<16>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
    add_xor(lane_xor_u64<8>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
    add_xor(lane_xor_u64<4>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
    add_xor(lane_xor_u64<2>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
    add_xor(lane_xor_u64<1>(static_cast<uint64_t>(__double_as_longlong(Z)), lane));
    const double lse = M + log(Z);

    // child r of the node: its pool entry and its beam key
    auto emit = [&](int r, uint64_t c) {
      const float sc =
          static_cast<float>(pscore + (static_cast<double>(from_orderable(c >> 32)) - lse));
      const int64_t o = static_cast<int64_t>(first) + f * W + r;
      if (o >= 0 && o < Vpool) {  // unvalidated pool sizes stay in bounds
        scores[pb + o] = sc;
        pool_parents[pb + o] = fnode;
        pool_tokens[pb + o] = static_cast<int32_t>(key_index(c));
      }
      child_s[f * W + r] =
          (static_cast<uint64_t>(orderable(sc)) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(f * W + r));
    };

    // T: the W-th largest chunk head (this wave's LDS rows only: a wave's LDS
    // accesses complete in program order)
    head_s[w][lane] = head;
    if (lane == 0) head_s[w][chunks] = 0;  // chunks <= 64; the pad of an odd count
    const int hr = count_greater(head_s[w], chunks, head);
    const uint64_t tb = __ballot(lane < chunks && head != 0 && hr == W - 1);
    uint64_t T = 0;
    if (tb != 0) {
      const int src = __ffsll(static_cast<long long>(tb)) - 1;
      const uint32_t lo = static_cast<uint32_t>(
          __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(head)), src));
      const uint32_t hi = static_cast<uint32_t>(
          __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(head >> 32)), src));
      T = (static_cast<uint64_t>(hi) << 32) | lo;
    }
    int total = 0;
#pragma unroll
    for (int k = 0; k < kListPerLane; ++k) {
      if (k * kWave >= n_keys) break;  // uniform
      const uint64_t ek = k < kEarly ? e[k] : lists[min(lane + k * kWave, n_keys - 1)];
      const bool c = lane + k * kWave < n_keys && ek != 0 && ek >= T;
      const uint64_t bm = __ballot(c);
      const int pos = total + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                  static_cast<uint32_t>(bm >> 32),
                                  __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bm), 0u)));
      if (c && pos < kWave) cand_s[w][pos] = ek;
      total += __popcll(bm);
    }
    if (total <= kWave) {
      if (lane == 0) cand_s[w][total] = 0;
      const uint64_t c = lane < total ? cand_s[w][lane] : 0;
      const int r = count_greater(cand_s[w], total, c);
      if (lane < total && r < W) emit(r, c);
    } else {  // W rounds of a wave argmax over the lane's keys (unique keys: one owner)
      uint32_t taken = 0;
      for (int r = 0; r < W; ++r) {
        uint64_t best = 0;
        int bk = 0;
#pragma unroll 1
        for (int k = 0; k < kListPerLane; ++k) {
          const uint64_t x = ((taken >> k) & 1) || lane + k * kWave >= n_keys
                                 ? 0
                                 : lists[lane + k * kWave];  // L2-resident reloads (rare path)
          if (x > best) {
            best = x;
            bk = k;
          }
        }
        const uint64_t win = wave_max_u64(best, lane);
        if (win != 0 && best == win) taken |= 1u << bk;
        if (lane == 0) emit(r, win);
      }
    }
  }
  __syncthreads();

  // the beam: child c's rank among all F*W children
  const int n_children = F * W;
  if (t == 0) child_s[n_children] = 0;  // the pad of an odd count
  __syncthreads();
  // P lanes count for each child, as many as the workgroup allows
  int P = 1;
  while (P < kWave && n_children * P * 2 <= static_cast<int>(blockDim.x)) P *= 2;
  const int per_round = blockDim.x / P;
  for (int c0 = 0; c0 < n_children; c0 += per_round) {  // uniform trip count
    const int c = c0 + t / P;
    const uint64_t k = c < n_children ? child_s[c] : ~uint64_t{0};
    const int r = group_count_greater(child_s, n_children, k, P, t % P);
    if (t % P == 0 && c < n_children && r < W_next)
      new_frontier[static_cast<int64_t>(b) * W_next + r] = first + c;
  }
  if (t == 0) pool_size[b] = first + n_children;  // every thread read it before the barrier
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
  const int waves = F < kSelectWaves ? F : kSelectWaves;
  hipLaunchKernelGGL(expand_select_kernel, dim3(B), dim3(waves * kWave), 0, stream, keys, mz,
                     chunks, frontier, F, W, W_next, scores, pool_parents, pool_tokens, pool_size,
                     Vpool, new_frontier, st);
  return hipGetLastError();
}

}  // namespace ltd
