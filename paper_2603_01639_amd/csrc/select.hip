// Candidate token selection (section 3.2, "Candidate Token Selection"): from a
// draft pool of up to 1024 candidates, keep the V with the highest cumulative
// score (equal scores: lower pool index first) and list them in pool order as
// a tree with re-indexed parents.
//
// One workgroup per sequence, one thread per pool column (the block is the
// pool width rounded up to a power of two, at least one wave).  No sort is
// needed:
//
//   1. an exact radix select of the V-th largest score over the order-
//      preserving 32-bit image of the float (-0 folded onto +0), 8 bits per
//      pass from the top: each pass histograms the digit of the candidates
//      still tied with the boundary (LDS adds, aggregated per wave over equal
//      digits), one wave scans the 256 bins from the top to find the bucket
//      that holds the V-th candidate, and the select stops as soon as that
//      whole bucket is kept (at most four passes);
//   2. a candidate is kept if it scores above the boundary bucket, or lies in
//      it among the first m by pool index, m being what the bucket still has
//      to give; its flattened position is the number of kept candidates before
//      it in pool order.  Both counts are wave ballots plus per-wave totals
//      (one barrier);
//   3. the new index of every kept candidate goes to LDS, and each kept
//      candidate writes its pool index, token and re-indexed parent (its
//      parent is kept: the kept set is a rooted subtree).
//
// Depth is an optional output, computed by pointer jumping over the parent
// links in LDS only when asked for.
//
// The pool is tiny (12 KB at 1011 candidates), so the kernel is bound by its
// few barriers and LDS round trips, not by HBM.  Parents are clamped into
// [0, i) before use and output positions into [0, V), so any input stays in
// bounds and every loop ends; only well-formed pools (as validation checks
// them) give the defined result.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kMaxPool = LTD_MAX_POOL;
constexpr int kMaxWaves = kMaxPool / kWave;
constexpr int kDigitBits = 8;
constexpr int kBins = 1 << kDigitBits;
constexpr int kPasses = 32 / kDigitBits;
constexpr int kAggregateRounds = 4;  // equal-digit groups a wave folds before plain LDS adds
static_assert(kBins == 4 * kWave, "one wave scans the bins, four per lane");

__device__ __forceinline__ uint32_t orderable(float s) {
  const uint32_t u = __float_as_uint(s + 0.0f);  // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive prefix sum over the 64 lanes of a wave (lane 0 first): a
// Hillis-Steele scan inside each row of 16 lanes with row shifts, then the
// row totals carried across rows with row broadcasts.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15 -> rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31 -> rows 2, 3
  return v;
}

// hist[digit] += 1 for every active lane.  Lanes sharing a digit are folded
// into one add for the first few digits found (the first pass sees only a
// handful of distinct digits, so plain adds would collide), the rest add
// their own 1.
__device__ __forceinline__ void wave_histogram_add(int32_t* hist, int digit, bool active,
                                                   int lane) {
  uint64_t rem = __ballot(active);
  for (int r = 0; r < kAggregateRounds && rem != 0; ++r) {
    const int leader = __ffsll(static_cast<unsigned long long>(rem)) - 1;
    const int dl = __builtin_amdgcn_readlane(digit, leader);
    const uint64_t m = __ballot(active && digit == dl);
    if (lane == leader) atomicAdd(&hist[dl], __popcll(m));
    if (active && digit == dl) active = false;
    rem &= ~m;
  }
  if (active) atomicAdd(&hist[digit], 1);
}

__global__ void __launch_bounds__(kMaxPool) select_kernel(
    const float* __restrict__ scores, const int32_t* __restrict__ pool_parents,
    const int32_t* __restrict__ pool_tokens, const int32_t* __restrict__ pool_size,
    const int32_t* __restrict__ n_select, int Vpool, int Nmax,
    int32_t* __restrict__ selected, int32_t* __restrict__ parents, int32_t* __restrict__ tokens,
    int32_t* __restrict__ depth, int32_t* __restrict__ n_nodes, const int32_t* status) {
  __shared__ int32_t hist_s[kPasses][kBins];
  __shared__ int32_t ctl_s[3];  // boundary digit, still to take from it, its count
  __shared__ int32_t wave_above_s[kMaxWaves];
  __shared__ int32_t wave_equal_s[kMaxWaves];
  __shared__ int32_t new_id_s[kMaxPool];
  __shared__ int32_t anc_s[2][kMaxPool];
  __shared__ int32_t dep_s[2][kMaxPool];

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
  const uint32_t key = orderable(sc);

  for (int i = t; i < kPasses * kBins; i += blockDim.x) (&hist_s[0][0])[i] = 0;
  if (t == 0) {
    ctl_s[0] = 0;
    ctl_s[1] = 1;
    ctl_s[2] = 1;
  }

  // optional depth: dep is the distance from t to anc (-1 = past the root)
  int my_dep = 0;
  if (depth != nullptr) {
    int a = p;
    my_dep = p >= 0 ? 1 : 0;
    anc_s[0][t] = a;
    dep_s[0][t] = my_dep;
    int cur = 0;
    for (int r = 0; r <= 10; ++r) {
      if (!__syncthreads_or(a >= 0)) break;
      if (a >= 0) {
        my_dep += dep_s[cur][a];
        a = anc_s[cur][a];
      }
      anc_s[cur ^ 1][t] = a;
      dep_s[cur ^ 1][t] = my_dep;
      cur ^= 1;
    }
  }
  __syncthreads();

  // 1. radix select: `prefix` holds the boundary bucket's top bits so far,
  // `need` how many candidates that bucket still has to give
  uint32_t prefix = 0;
  int need = V;
  int shift = 32;
  for (int pass = 0; pass < kPasses; ++pass) {
    shift -= kDigitBits;
    const bool in_play = valid && (pass == 0 || (key >> (shift + kDigitBits)) == prefix);
    wave_histogram_add(hist_s[pass], static_cast<int>((key >> shift) & (kBins - 1)), in_play,
                       lane);
    __syncthreads();
    if (w == 0) {
      // lane l owns digits 255-4l (first) down to 252-4l
      const int4 h = *reinterpret_cast<const int4*>(&hist_s[pass][kBins - 4 - 4 * lane]);
      const int sum = h.x + h.y + h.z + h.w;
      const int incl = wave_inclusive_scan(sum);
      int c = incl - sum;  // candidates in higher digits
      if (c < need && need <= incl) {
        const int cnt[4] = {h.w, h.z, h.y, h.x};
        int k = 0;
        while (k < 3 && c + cnt[k] < need) c += cnt[k++];
        ctl_s[0] = kBins - 1 - 4 * lane - k;
        ctl_s[1] = need - c;
        ctl_s[2] = cnt[k];
      }
    }
    __syncthreads();
    prefix = (prefix << kDigitBits) | static_cast<uint32_t>(ctl_s[0]);
    need = ctl_s[1];
    const int bucket = ctl_s[2];
    if (bucket == need) break;  // the whole boundary bucket is kept
  }

  // 2. kept candidates and their positions in pool order
  const uint32_t hi = shift == 0 ? key : key >> shift;
  const bool above = valid && hi > prefix;
  const bool equal = valid && hi == prefix;
  const uint64_t below = (1ull << lane) - 1;
  const uint64_t m_above = __ballot(above);
  const uint64_t m_equal = __ballot(equal);
  if (lane == 0) {
    wave_above_s[w] = __popcll(m_above);
    wave_equal_s[w] = __popcll(m_equal);
  }
  __syncthreads();
  int n_above = __popcll(m_above & below);
  int n_equal = __popcll(m_equal & below);
  for (int k = 0; k < w; ++k) {
    n_above += wave_above_s[k];
    n_equal += wave_equal_s[k];
  }
  const bool kept = above || (equal && n_equal < need);
  const int pos = min(max(n_above + min(n_equal, need), 0), V - 1);
  new_id_s[t] = kept ? pos : -1;
  __syncthreads();

  // 3. outputs
  if (kept) {
    const int64_t o = static_cast<int64_t>(b) * Nmax + pos;
    parents[o] = p < 0 ? -1 : new_id_s[p];
    tokens[o] = tk;
    if (selected) selected[o] = t;
    if (depth) depth[o] = my_dep;
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
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(select_block_threads(Vpool)), 0, stream,
                     scores, pool_parents, pool_tokens, pool_size, n_select, Vpool, Nmax, selected,
                     parents, tokens, depth, n_nodes, status);
  return hipGetLastError();
}

}  // namespace ltd
