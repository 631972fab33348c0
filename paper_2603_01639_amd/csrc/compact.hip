// KV compaction: after acceptance, the accepted root path's K/V rows move to
// the rows right after the prefix and the other candidates are dropped
// (arXiv 2603.01639, section 3.2: the candidates after the first mismatch are
// discarded).
//
// One workgroup per (sequence, layer, kv head, K or V).  Row j of the path
// moves from P + path[j] to P + j.  The path is strictly increasing with
// path[j] >= j, so a destination P + j can only be the source of an earlier
// or the same slot (path[j'] = j needs j' <= j).  Rows are therefore moved in
// ascending passes of R rows: every pass reads all its sources into
// registers, waits at a barrier, then writes; a later pass's sources
// (path[j] >= j >= pass end) lie past every destination already written.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kThreads = 256;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(kThreads) kv_compact_kernel(
    unsigned char* __restrict__ k_cache, unsigned char* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ prefix_len,
    int32_t* __restrict__ new_prefix_len, const int32_t* __restrict__ accepted_nodes,
    const int32_t* __restrict__ n_accepted, int Nmax, int Hkv, int row_bytes, int kv_rows,
    int max_blocks, int64_t layer_stride_bytes, const int32_t* status) {
  const int b = blockIdx.x;
  const int y = blockIdx.y;  // ((layer * Hkv) + g) * 2 + which
  const int which = y & 1;
  const int g = (y >> 1) % Hkv;
  const int layer = (y >> 1) / Hkv;
  if (halted(status)) return;
  // The first pass's path entries are loaded together with P and n (j is
  // clamped below Nmax, so the load is in bounds whatever n is).
  const int32_t* path = accepted_nodes + static_cast<int64_t>(b) * Nmax;
  const int vec_per_row = row_bytes / 16;
  const int rows_per_pass = kThreads / vec_per_row;
  const int rj = threadIdx.x / vec_per_row;
  const int col = threadIdx.x % vec_per_row;
  int pj = path[min(rj, Nmax - 1)];
  const int P = prefix_len[b];
  const int n = n_accepted[b];
  unsigned char* base = (which ? v_cache : k_cache) + layer * layer_stride_bytes;

  for (int j0 = 0; j0 < n; j0 += rows_per_pass) {
    const int j = j0 + rj;
    if (j0 > 0) pj = path[min(j, Nmax - 1)];
    const bool active = rj < rows_per_pass && j < n && pj != j;
    u32x4 v = {0, 0, 0, 0};
    int64_t dst = 0;
    if (active) {
      // cache_row counts elements of a `row_bytes`-wide row with d = row_bytes
      const int64_t src = cache_row(block_table, b, g, P + pj, Hkv, row_bytes, kv_rows, max_blocks);
      dst = cache_row(block_table, b, g, P + j, Hkv, row_bytes, kv_rows, max_blocks);
      v = *reinterpret_cast<const u32x4*>(base + src + col * 16);
    }
    __syncthreads();
    if (active) *reinterpret_cast<u32x4*>(base + dst + col * 16) = v;
    __syncthreads();
  }
  if (y == 0 && threadIdx.x == 0) new_prefix_len[b] = P + n;
}

}  // namespace

hipError_t launch_compact(void* k_cache, void* v_cache, const int32_t* block_table,
                          const int32_t* prefix_len, int32_t* new_prefix_len,
                          const int32_t* accepted_nodes, const int32_t* n_accepted, int B,
                          int Nmax, int Hkv, int row_bytes, int kv_rows, int max_blocks,
                          int num_layers, int64_t layer_stride_bytes, const int32_t* status,
                          hipStream_t stream) {
  const dim3 grid(B, num_layers * Hkv * 2);
  hipLaunchKernelGGL(kv_compact_kernel, grid, dim3(kThreads), 0, stream,
                     static_cast<unsigned char*>(k_cache), static_cast<unsigned char*>(v_cache),
                     block_table, prefix_len, new_prefix_len, accepted_nodes, n_accepted, Nmax,
                     Hkv, row_bytes, kv_rows, max_blocks, layer_stride_bytes, status);
  return hipGetLastError();
}

}  // namespace ltd
