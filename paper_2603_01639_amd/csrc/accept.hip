// Greedy acceptance (arXiv 2603.01639, section 3.2, "Draft Tree
// Verification"): the target's prediction at every node, then the longest
// root path of accepted draft tokens and the bonus token.
//
// Two kernels on the stream:
//  1. argmax_partial_kernel: the vocabulary-wide argmax of every node's fp32
//     logits row, split into chunks so that N * chunks workgroups stream the
//     logits at HBM rate.  Each chunk reduces to one packed 64-bit key
//       (order-preserving value bits << 32) | (0xFFFFFFFF - index)
//     whose maximum is the largest value with the lowest index; -0.0 is
//     folded onto +0.0 before packing, so the two compare equal.
//  2. accept_scan_kernel: one workgroup per sequence.  It fetches every chunk
//     key of the sequence in one round of independent loads spread over all
//     threads, issued before the node count arrives (they stay inside the
//     sequence's Nmax * chunks keys), and folds them into per-node maxima in
//     LDS; then, one thread per node, acceptance and depth by pointer doubling
//     over the parent links (ceil(log2 N) rounds), the deepest accepted node
//     (smallest index on ties), and the path by binary lifting from that leaf.
// The kernel boundary is the only synchronisation between the two: on this
// chip a device-scope atomic round trip costs about as much as the whole scan,
// and an agent-scope fence (an L2 write-back) in every argmax workgroup costs
// several times the argmax.
#include <mutex>

#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kArgmaxThreads = 256;
constexpr int kChunk = 16384;                               // logits per workgroup (64 KiB)
constexpr int kVecPerThread = kChunk / 4 / kArgmaxThreads;  // 16-byte loads per thread
constexpr int kScanThreads = LTD_MAX_NODES;                 // one thread per node
constexpr int kKeysPerRound = 8;                            // key loads in flight per thread
constexpr int kLiftLevels = 8;                              // 2^8 = LTD_MAX_NODES

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint64_t pack_key(float v, int idx) {
  if (v == 0.f) v = 0.f;  // -0.0 -> +0.0
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | static_cast<uint32_t>(0xFFFFFFFFu - idx);
}
__device__ __forceinline__ int key_index(uint64_t key) {
  return static_cast<int>(0xFFFFFFFFu - static_cast<uint32_t>(key));
}
__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return b > a ? b : a; }

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v = max_u64(v, __shfl_xor(v, off, kWave));
  return v;
}

template <bool kVec4>
__global__ void __launch_bounds__(kArgmaxThreads) argmax_partial_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ n_nodes, int Nmax, int Voc,
    int chunks, uint64_t* __restrict__ partial, const int32_t* status) {
  const int chunk = blockIdx.x, i = blockIdx.y, b = blockIdx.z;
  if (halted(status)) return;
  if (i >= n_nodes[b]) return;
  const float* row = logits + (static_cast<int64_t>(b) * Nmax + i) * Voc;
  const int lo = chunk * kChunk;
  const int hi = min(Voc, lo + kChunk);
  uint64_t best = 0;
  if (kVec4) {
    // Elements 4f .. 4f+3 of the row for f = lo/4 + tid + 256u.
    const f32x4* row4 = reinterpret_cast<const f32x4*>(row);
    const int f0 = (lo >> 2) + threadIdx.x;
    const int fend = hi >> 2;
    // All loads in flight at once; then the thread's float maximum, and the
    // lowest index holding it (-0.0 == +0.0, and pack_key makes both +0.0),
    // which is the thread's largest packed key: about three operations per
    // element instead of a 64-bit key and maximum each.
    f32x4 x[kVecPerThread];
#pragma unroll
    for (int u = 0; u < kVecPerThread; ++u) {
      const int f = f0 + u * kArgmaxThreads;
      x[u] = f < fend ? __builtin_nontemporal_load(row4 + f)
                      : (f32x4){-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    }
    float vm = -INFINITY;
#pragma unroll
    for (int u = 0; u < kVecPerThread; ++u)
      vm = fmaxf(vm, fmaxf(fmaxf(x[u].x, x[u].y), fmaxf(x[u].z, x[u].w)));
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int u = kVecPerThread - 1; u >= 0; --u) {  // downwards: the lowest index wins
      const int v = (f0 + u * kArgmaxThreads) << 2;
      bi = x[u].w == vm ? v + 3 : bi;
      bi = x[u].z == vm ? v + 2 : bi;
      bi = x[u].y == vm ? v + 1 : bi;
      bi = x[u].x == vm ? v : bi;
    }
    if (bi < hi) best = pack_key(vm, bi);  // (padding past the row is never the lowest)
  } else {
    for (int v = lo + threadIdx.x; v < hi; v += kArgmaxThreads) best = max_u64(best, pack_key(row[v], v));
  }
  __shared__ uint64_t wave_best[kArgmaxThreads / kWave];
  best = wave_max_u64(best);
  if ((threadIdx.x & (kWave - 1)) == 0) wave_best[threadIdx.x / kWave] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t r = wave_best[0];
    for (int w = 1; w < kArgmaxThreads / kWave; ++w) r = max_u64(r, wave_best[w]);
    partial[(static_cast<int64_t>(b) * Nmax + i) * chunks + chunk] = r;
  }
}

__global__ void __launch_bounds__(kScanThreads) accept_scan_kernel(
    const uint64_t* __restrict__ partial, int chunks, const int32_t* __restrict__ draft_tokens,
    const int32_t* __restrict__ parents, const int32_t* __restrict__ n_nodes, int Nmax,
    int32_t* __restrict__ pred_out, int32_t* __restrict__ accepted_nodes,
    int32_t* __restrict__ out_tokens, int32_t* __restrict__ n_accepted, const int32_t* status) {
  __shared__ unsigned long long key_s[LTD_MAX_NODES];
  __shared__ int pred_s[LTD_MAX_NODES];
  __shared__ int tok_s[LTD_MAX_NODES];
  __shared__ int16_t up_s[kLiftLevels][LTD_MAX_NODES];  // 2^r-th ancestor, -1 past the root
  __shared__ int ok_s[2][LTD_MAX_NODES];
  __shared__ int dep_s[2][LTD_MAX_NODES];
  __shared__ int best_s;

  const int b = blockIdx.x;
  const int c = threadIdx.x;
  if (halted(status)) return;
  const int64_t base = static_cast<int64_t>(b) * Nmax;
  // Everything the scan reads is requested in one round, before n is known:
  // the node's token and parent and the first kKeysPerRound * 256 chunk keys
  // of the sequence (key k = node k / chunks, chunk k % chunks; thread c
  // takes keys c + 256 j), all inside the sequence's Nmax rows.
  const int total_max = Nmax * chunks;
  const uint64_t* pk = partial + base * chunks;
  const int c_in = min(c, Nmax - 1);
  const int tok = draft_tokens[base + c_in];
  const int parent = c == 0 ? -1 : parents[base + c_in];
  uint64_t key[kKeysPerRound];
#pragma unroll
  for (int j = 0; j < kKeysPerRound; ++j) {
    const int k = j * kScanThreads + c;
    key[j] = k < total_max ? pk[k] : 0;
  }
  const int n = n_nodes[b];
  key_s[c] = 0;
  if (c == 0) best_s = 0;
  __syncthreads();
  // Fold the keys into per-node maxima with LDS atomics; sequences with more
  // than kKeysPerRound * 256 keys take further rounds.
  const int total = n * chunks;
  for (int k0 = 0; k0 < total; k0 += kKeysPerRound * kScanThreads) {
    if (k0 > 0) {
#pragma unroll
      for (int j = 0; j < kKeysPerRound; ++j) {
        const int k = k0 + j * kScanThreads + c;
        key[j] = k < total ? pk[k] : 0;
      }
    }
#pragma unroll
    for (int j = 0; j < kKeysPerRound; ++j) {
      const int k = k0 + j * kScanThreads + c;
      if (k < total) atomicMax(&key_s[k / chunks], static_cast<unsigned long long>(key[j]));
    }
  }
  __syncthreads();
  if (c < n) {
    const int p = key_index(key_s[c]);
    pred_s[c] = p;
    pred_out[base + c] = p;
    tok_s[c] = tok;
    up_s[0][c] = static_cast<int16_t>(c == 0 ? -1 : parent);
  }
  __syncthreads();

  // valid(c): the draft token equals the target's prediction at the parent.
  // ok(c) = AND of valid over c's root path; depth(c) = its length - 1.
  int cur = 0;
  if (c < n) {
    ok_s[0][c] = (c == 0) ? 1 : (tok_s[c] == pred_s[parent]);
    dep_s[0][c] = (c == 0) ? 0 : 1;
  }
  __syncthreads();
  // Round r folds in the 2^r-th ancestor's values and builds level r + 1 of
  // the ancestor table.  After R rounds each node covers 2^R links of its root
  // path, so ceil(log2 n) rounds (at least one) cover every depth < n, and the
  // levels built are those the lifting below needs for steps < n.
  for (int r = 0; r < kLiftLevels; ++r) {
    if (r > 0 && (1 << r) >= n) break;  // uniform: every thread leaves together
    if (c < n) {
      const int j = up_s[r][c];
      int ok = ok_s[cur][c], dep = dep_s[cur][c];
      if (j >= 0) {
        ok &= ok_s[cur][j];
        dep += dep_s[cur][j];
      }
      ok_s[cur ^ 1][c] = ok;
      dep_s[cur ^ 1][c] = dep;
      if (r + 1 < kLiftLevels) up_s[r + 1][c] = static_cast<int16_t>(j >= 0 ? up_s[r][j] : -1);
    }
    cur ^= 1;
    __syncthreads();
  }

  // Deepest accepted node, smallest index among equals: maximise
  // (depth << 16) | (0xFFFF - index).
  if (c < n && ok_s[cur][c]) atomicMax(&best_s, (dep_s[cur][c] << 16) | (0xFFFF - c));
  __syncthreads();
  const int leaf = 0xFFFF - (best_s & 0xFFFF);
  const int len = (best_s >> 16) + 1;

  // Thread k < len writes the path node at depth k: the (len-1-k)-th ancestor
  // of the leaf, by binary lifting (len - 1 < n needs only the levels built).
  if (c < len) {
    int steps = len - 1 - c, j = leaf;
    for (int r = 0; r < kLiftLevels; ++r)
      if (steps & (1 << r)) j = up_s[r][j];
    accepted_nodes[base + c] = j;
    if (c >= 1) out_tokens[base + c - 1] = tok_s[j];
  }
  if (c == 0) {
    out_tokens[base + len - 1] = pred_s[leaf];
    n_accepted[b] = len;
  }
}

// Scratch of the allocation-free entry point: the argmax partial keys live in
// a file-scope device array instead of a caller workspace.  Each GPU the
// library runs on holds its own copy for the life of the process.  Host code
// never uses the array's name as an address (on the host it only stands for
// the symbol); the device address of each GPU's copy is looked up once, with
// that GPU current, and kept per device.
constexpr size_t kNoAllocScratchBytes = size_t{4} << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxScratchDevices = 64;

// The device address of this GPU's scratch, or nullptr when it cannot be had.
void* noalloc_scratch_ptr() {
  static std::once_flag once[kMaxScratchDevices];
  static void* ptr[kMaxScratchDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return nullptr;
  std::call_once(once[dev], [dev] {
    void* p = nullptr;
    ptr[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess ? p : nullptr;
  });
  return ptr[dev];
}

}  // namespace

size_t accept_noalloc_scratch_bytes() { return kNoAllocScratchBytes; }

void* accept_noalloc_scratch() { return noalloc_scratch_ptr(); }

size_t accept_workspace_bytes(int B, int Nmax, int Voc) {
  const int chunks = (Voc + kChunk - 1) / kChunk;
  return static_cast<size_t>(B) * Nmax * chunks * sizeof(uint64_t);
}

hipError_t launch_accept(const float* logits, const int32_t* draft_tokens, const int32_t* parents,
                         const int32_t* n_nodes, int B, int Nmax, int Voc, int32_t* pred,
                         int32_t* accepted_nodes, int32_t* out_tokens, int32_t* n_accepted,
                         void* workspace, const int32_t* status, hipStream_t stream) {
  const int chunks = (Voc + kChunk - 1) / kChunk;
  uint64_t* partial = static_cast<uint64_t*>(workspace);
  const dim3 grid(chunks, Nmax, B);
  const bool vec4 = (Voc % 4) == 0 && (reinterpret_cast<uintptr_t>(logits) % 16) == 0;
  if (vec4)
    hipLaunchKernelGGL(argmax_partial_kernel<true>, grid, dim3(kArgmaxThreads), 0, stream, logits,
                       n_nodes, Nmax, Voc, chunks, partial, status);
  else
    hipLaunchKernelGGL(argmax_partial_kernel<false>, grid, dim3(kArgmaxThreads), 0, stream,
                       logits, n_nodes, Nmax, Voc, chunks, partial, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_scan_kernel, dim3(B), dim3(kScanThreads), 0, stream, partial, chunks,
                     draft_tokens, parents, n_nodes, Nmax, pred, accepted_nodes, out_tokens,
                     n_accepted, status);
  return hipGetLastError();
}

}  // namespace ltd
