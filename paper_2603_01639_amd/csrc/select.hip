// Candidate token selection (section 3.2, "Candidate Token Selection"): from a
// draft pool of up to 1024 candidates, keep the V with the highest cumulative
// score and flatten them into a topologically ordered tree.
//
// One workgroup per sequence, one thread per pool column (the block is the
// pool width rounded up to a power of two, at least one wave):
//
//   1. depth of every candidate by pointer jumping over the parent links in
//      LDS (ceil(log2 depth) rounds, ended as soon as every chain reached the
//      root);
//   2. a rank key per candidate: the order-preserving image of the float32
//      score (-0 folded onto +0) above the depth and pool index complemented
//      (10 bits each), so that a larger key ranks first and
//      ties go to the shallower, then lower-indexed candidate; every key is
//      distinct;
//   3. a bitonic sort of the keys into descending order, one key per thread:
//      partners within a wave are exchanged with lane shuffles, partners in
//      other waves through a double-buffered LDS array (one barrier a stage);
//   4. the first V keys are the kept candidates in rank order.  Within one
//      depth, rank order is already the flattened order (score, then index),
//      so the flattened position is a stable counting sort by depth: the
//      kept candidates with a smaller depth, plus those of the same depth
//      ranked earlier (lane ballots within a wave, per-wave depth counts in
//      LDS across the at most four waves that hold kept candidates);
//   5. the new index of every kept candidate goes to LDS, and each kept
//      candidate writes its pool index, token, depth and re-indexed parent.
//
// The pool is tiny (12 KB at 1011 candidates), so the kernel is bound by its
// chain of barriers and LDS round trips, not by HBM.  Parents are clamped into
// [0, i) before use, so any input stays in bounds and every loop ends; only
// well-formed pools (as validation checks them) give the defined result.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kMaxPool = LTD_MAX_POOL;
constexpr int kOutWaves = LTD_MAX_NODES / kWave;  // waves that can hold kept candidates
constexpr int kIndexBits = 10;                    // pool index and depth are < 1024
constexpr int kLowBits = 2 * kIndexBits;
constexpr uint32_t kLowMask = (1u << kLowBits) - 1;
constexpr uint64_t kRealKey = 1ull << (32 + kLowBits);
static_assert(kMaxPool == 1 << kIndexBits, "pool index must fit the key's index field");

__device__ __forceinline__ uint32_t orderable(float s) {
  const uint32_t u = __float_as_uint(s + 0.0f);  // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  const int lo = __shfl_xor(static_cast<int>(static_cast<uint32_t>(v)), mask, kWave);
  const int hi = __shfl_xor(static_cast<int>(static_cast<uint32_t>(v >> 32)), mask, kWave);
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}

__global__ void __launch_bounds__(kMaxPool) select_kernel(
    const float* __restrict__ scores, const int32_t* __restrict__ pool_parents,
    const int32_t* __restrict__ pool_tokens, const int32_t* __restrict__ pool_size,
    const int32_t* __restrict__ n_select, int Vpool, int Nmax, int n2,
    int32_t* __restrict__ selected, int32_t* __restrict__ parents, int32_t* __restrict__ tokens,
    int32_t* __restrict__ depth, int32_t* __restrict__ n_nodes, const int32_t* status) {
  __shared__ uint64_t key_s[2][kMaxPool];
  __shared__ int32_t anc_s[kMaxPool];
  __shared__ int32_t dep_s[kMaxPool];
  __shared__ int32_t par_s[kMaxPool];
  __shared__ int32_t tok_s[kMaxPool];
  __shared__ int32_t new_id_s[kMaxPool];
  __shared__ int32_t cnt_s[kOutWaves][kMaxPool];
  __shared__ int32_t base_s[kMaxPool];
  __shared__ int32_t wsum_s[kMaxPool / kWave];

  if (halted(status)) return;
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int w = t / kWave;
  const int64_t row = static_cast<int64_t>(b) * Vpool;

  // every load is issued before the sizes arrive
  float sc = 0.f;
  int32_t p = -1, tk = 0;
  if (t < Vpool) {
    sc = scores[row + t];
    p = pool_parents[row + t];
    tk = pool_tokens[row + t];
  }
  const int n = min(max(pool_size[b], 1), Vpool);
  const int V = min(max(n_select[b], 1), min(Nmax, n));
  const bool valid = t < n;
  p = (!valid || t == 0) ? -1 : min(max(p, 0), t - 1);

  par_s[t] = p;
  tok_s[t] = tk;
  anc_s[t] = p;
  dep_s[t] = p >= 0 ? 1 : 0;
  new_id_s[t] = -1;
#pragma unroll
  for (int k = 0; k < kOutWaves; ++k) cnt_s[k][t] = 0;

  // 1. depth: dep_s[i] is the distance from i to anc_s[i] (-1 = past the root)
  int my_dep = p >= 0 ? 1 : 0;
  int my_anc = p;
  for (int r = 0; r <= kIndexBits; ++r) {
    if (!__syncthreads_or(my_anc >= 0)) break;
    int d2 = 0, a2 = -1;
    if (my_anc >= 0) {
      d2 = dep_s[my_anc];
      a2 = anc_s[my_anc];
    }
    __syncthreads();
    if (my_anc >= 0) {
      my_dep += d2;
      my_anc = a2;
      dep_s[t] = my_dep;
      anc_s[t] = my_anc;
    }
  }

  // 2. rank key; padding columns get 0, below every real key (bit 52 is set
  // in every real key)
  uint64_t key = 0;
  if (valid) {
    const uint32_t low = kLowMask - ((static_cast<uint32_t>(my_dep) << kIndexBits) | t);
    key = kRealKey | (static_cast<uint64_t>(orderable(sc)) << kLowBits) | low;
  }

  // 3. bitonic sort, descending
  int buf = 0;
  for (int k = 2; k <= n2; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      uint64_t other;
      if (j >= kWave) {
        key_s[buf][t] = key;
        __syncthreads();
        other = key_s[buf][t ^ j];
        buf ^= 1;
      } else {
        other = shfl_xor_u64(key, j);
      }
      const bool keep_max = ((t & j) == 0) == ((t & k) == 0);
      key = keep_max ? (key > other ? key : other) : (key < other ? key : other);
    }
  }

  // 4. thread t holds the candidate of rank t; the first V are kept
  const bool kept = t < V;
  const uint32_t low = kLowMask - static_cast<uint32_t>(key & kLowMask);
  const int idx = static_cast<int>(low & (kMaxPool - 1));
  const int d = static_cast<int>(low >> kIndexBits);
  int within = 0;  // kept candidates of the same depth ranked earlier in this wave
  uint64_t rem = __ballot(kept);
  while (rem != 0) {
    const int leader = __ffsll(static_cast<unsigned long long>(rem)) - 1;
    const int dd = __shfl(d, leader, kWave);
    const bool same = kept && d == dd;
    const uint64_t m = __ballot(same);
    if (same) within = __popcll(m & ((1ull << lane) - 1));
    if (lane == leader) cnt_s[w][dd] = __popcll(m);
    rem &= ~m;
  }
  __syncthreads();

  // kept candidates with depth below t: exclusive scan of the per-depth totals
  int tot = 0;
#pragma unroll
  for (int k = 0; k < kOutWaves; ++k) tot += cnt_s[k][t];
  int incl = tot;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int v = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += v;
  }
  if (lane == kWave - 1) wsum_s[w] = incl;
  __syncthreads();
  int before = 0;
  for (int k = 0; k < w; ++k) before += wsum_s[k];
  base_s[t] = before + incl - tot;
  __syncthreads();

  int pos = 0;
  if (kept) {
    pos = base_s[d] + within;
    for (int k = 0; k < w; ++k) pos += cnt_s[k][d];
    pos = min(max(pos, 0), V - 1);  // a permutation of [0, V) already; keeps stores in the row
    new_id_s[idx] = pos;
  }
  __syncthreads();

  // 5. outputs in flattened order
  if (kept) {
    const int64_t o = static_cast<int64_t>(b) * Nmax + pos;
    const int pp = par_s[idx];
    parents[o] = pp < 0 ? -1 : new_id_s[pp];
    tokens[o] = tok_s[idx];
    if (selected) selected[o] = idx;
    if (depth) depth[o] = d;
  }
  if (t == 0) n_nodes[b] = V;
}

constexpr int kValidateThreads = 1024;

// Lowest (sequence << 8 | code) over every failing check of every sequence.
__global__ void __launch_bounds__(kValidateThreads) validate_pool_kernel(
    const float* __restrict__ scores, const int32_t* __restrict__ pool_parents,
    const int32_t* __restrict__ pool_size, const int32_t* __restrict__ n_select, int B, int Vpool,
    int Nmax, int32_t* status) {
  __shared__ int best;
  if (threadIdx.x == 0) best = 0x7FFFFFFF;
  __syncthreads();
  int key = 0x7FFFFFFF;
  const int64_t total = static_cast<int64_t>(B) * Vpool;
  for (int64_t e = threadIdx.x; e < total; e += kValidateThreads) {
    const int b = static_cast<int>(e / Vpool);
    const int i = static_cast<int>(e - static_cast<int64_t>(b) * Vpool);
    const int n = pool_size[b];
    int code = 0;
    if (i == 0 && (n < 1 || n > Vpool || n_select[b] < 1 || n_select[b] > Nmax))
      code = LTD_STATUS_BAD_NNODES;
    else if (i < min(n, Vpool)) {
      const int32_t p = pool_parents[e];
      const float s = scores[e];
      if (i == 0 ? p != -1 : (p < 0 || p >= i))
        code = LTD_STATUS_BAD_PARENT;
      else if (s != s || (i > 0 && s > scores[e - i + p]))
        code = LTD_STATUS_BAD_SCORE;
    }
    if (code != 0) key = min(key, (b << 8) | code);
  }
  if (key != 0x7FFFFFFF) atomicMin(&best, key);
  __syncthreads();
  if (threadIdx.x == 0) *status = (best == 0x7FFFFFFF) ? 0 : (best & 0xFF);
}

}  // namespace

int select_block_threads(int Vpool) {
  int n2 = kWave;
  while (n2 < Vpool) n2 <<= 1;
  return n2;
}

hipError_t launch_validate_pool(const float* scores, const int32_t* pool_parents,
                                const int32_t* pool_size, const int32_t* n_select, int B,
                                int Vpool, int Nmax, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(validate_pool_kernel, dim3(1), dim3(kValidateThreads), 0, stream, scores,
                     pool_parents, pool_size, n_select, B, Vpool, Nmax, status);
  return hipGetLastError();
}

hipError_t launch_select(const float* scores, const int32_t* pool_parents,
                         const int32_t* pool_tokens, const int32_t* pool_size,
                         const int32_t* n_select, int B, int Vpool, int Nmax, int32_t* selected,
                         int32_t* parents, int32_t* tokens, int32_t* depth, int32_t* n_nodes,
                         const int32_t* status, hipStream_t stream) {
  const int n2 = select_block_threads(Vpool);
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(n2), 0, stream, scores, pool_parents,
                     pool_tokens, pool_size, n_select, Vpool, Nmax, n2, selected, parents, tokens,
                     depth, n_nodes, status);
  return hipGetLastError();
}

}  // namespace ltd
