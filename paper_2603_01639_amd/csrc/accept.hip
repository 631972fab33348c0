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
//  2. accept_scan_kernel: one workgroup per sequence, one thread per node.
//     It finishes the argmax from the chunk keys, then computes acceptance
//     and depth with pointer doubling over the parent links (log2 N rounds),
//     picks the deepest accepted node (smallest index on ties), and emits the
//     path by binary lifting from that leaf.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kArgmaxThreads = 256;
constexpr int kChunk = 8192;  // logits per argmax workgroup (32 KiB)
constexpr int kLiftLevels = 8;  // 2^8 = LTD_MAX_NODES

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

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off, kWave);
    v = o > v ? o : v;
  }
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
    const f32x4* row4 = reinterpret_cast<const f32x4*>(row);
#pragma unroll 4
    for (int f = (lo >> 2) + threadIdx.x; f < (hi >> 2); f += kArgmaxThreads) {
      const f32x4 x = __builtin_nontemporal_load(row4 + f);
      const int v = f << 2;
      uint64_t k0 = pack_key(x.x, v), k1 = pack_key(x.y, v + 1);
      uint64_t k2 = pack_key(x.z, v + 2), k3 = pack_key(x.w, v + 3);
      k0 = k1 > k0 ? k1 : k0;
      k2 = k3 > k2 ? k3 : k2;
      k0 = k2 > k0 ? k2 : k0;
      best = k0 > best ? k0 : best;
    }
  } else {
    for (int v = lo + threadIdx.x; v < hi; v += kArgmaxThreads) {
      const uint64_t k = pack_key(row[v], v);
      best = k > best ? k : best;
    }
  }
  __shared__ uint64_t wave_best[kArgmaxThreads / kWave];
  best = wave_max_u64(best);
  if ((threadIdx.x & (kWave - 1)) == 0) wave_best[threadIdx.x / kWave] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t r = wave_best[0];
    for (int w = 1; w < kArgmaxThreads / kWave; ++w) r = wave_best[w] > r ? wave_best[w] : r;
    partial[(static_cast<int64_t>(b) * Nmax + i) * chunks + chunk] = r;
  }
}

__global__ void __launch_bounds__(LTD_MAX_NODES) accept_scan_kernel(
    const uint64_t* __restrict__ partial, int chunks, const int32_t* __restrict__ draft_tokens,
    const int32_t* __restrict__ parents, const int32_t* __restrict__ n_nodes, int Nmax,
    int32_t* __restrict__ pred_out, int32_t* __restrict__ accepted_nodes,
    int32_t* __restrict__ out_tokens, int32_t* __restrict__ n_accepted, const int32_t* status) {
  __shared__ int pred_s[LTD_MAX_NODES];
  __shared__ int tok_s[LTD_MAX_NODES];
  __shared__ int16_t up_s[kLiftLevels][LTD_MAX_NODES];  // 2^r-th ancestor, -1 past the root
  __shared__ int ok_s[2][LTD_MAX_NODES];
  __shared__ int dep_s[2][LTD_MAX_NODES];
  __shared__ int best_s;

  const int b = blockIdx.x;
  const int c = threadIdx.x;
  if (halted(status)) return;
  const int n = n_nodes[b];
  const int64_t base = static_cast<int64_t>(b) * Nmax;

  int parent = -1;
  if (c < n) {
    uint64_t key = 0;
    const uint64_t* pk = partial + (base + c) * chunks;
    for (int j = 0; j < chunks; ++j) key = pk[j] > key ? pk[j] : key;
    const int p = key_index(key);
    pred_s[c] = p;
    pred_out[base + c] = p;
    tok_s[c] = draft_tokens[base + c];
    parent = parents[base + c];
    up_s[0][c] = static_cast<int16_t>(c == 0 ? -1 : parent);
  }
  if (c == 0) best_s = 0;
  __syncthreads();

  // valid(c): the draft token equals the target's prediction at the parent.
  // ok(c) = AND of valid over c's root path; depth(c) = its length - 1.
  int cur = 0;
  if (c < n) {
    ok_s[0][c] = (c == 0) ? 1 : (tok_s[c] == pred_s[parent]);
    dep_s[0][c] = (c == 0) ? 0 : 1;
  }
  __syncthreads();
  for (int r = 0; r < kLiftLevels; ++r) {
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
  // of the leaf, by binary lifting.
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

}  // namespace

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
  hipLaunchKernelGGL(accept_scan_kernel, dim3(B), dim3(LTD_MAX_NODES), 0, stream, partial, chunks,
                     draft_tokens, parents, n_nodes, Nmax, pred, accepted_nodes, out_tokens,
                     n_accepted, status);
  return hipGetLastError();
}

}  // namespace ltd
