// Device-side checks of data-dependent preconditions (run only when the caller
// asks for validation).  One workgroup scans every sequence and reports the
// code of the lowest failing sequence, checks in code order.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kThreads = 256;

__device__ int check_tree(const int32_t* block_table, const int32_t* prefix_len,
                          const int32_t* parents, const int32_t* n_nodes, int b, int Nmax,
                          int max_prefix, int kv_rows, int max_blocks, int num_blocks,
                          bool check_cache) {
  const int n = n_nodes[b];
  if (n < 1 || n > Nmax) return LTD_STATUS_BAD_NNODES;
  const int32_t* par = parents + static_cast<int64_t>(b) * Nmax;
  if (par[0] != -1) return LTD_STATUS_BAD_PARENT;
  for (int i = 1; i < n; ++i)
    if (par[i] < 0 || par[i] >= i) return LTD_STATUS_BAD_PARENT;
  if (!check_cache) return 0;
  const int P = prefix_len[b];
  const int64_t capacity =
      block_table ? static_cast<int64_t>(kv_rows) * max_blocks : static_cast<int64_t>(kv_rows);
  if (P < 0 || P > max_prefix || static_cast<int64_t>(P) + n > capacity)
    return LTD_STATUS_BAD_PREFIX;
  if (block_table) {
    const int used = (P + n + kv_rows - 1) / kv_rows;
    for (int j = 0; j < used; ++j) {
      const int32_t blk = block_table[static_cast<int64_t>(b) * max_blocks + j];
      if (blk < 0 || blk >= num_blocks) return LTD_STATUS_BAD_BLOCK;
    }
  }
  return 0;
}

__device__ int check_path(const int32_t* block_table, const int32_t* prefix_len,
                          const int32_t* accepted_nodes, const int32_t* n_accepted, int b,
                          int Nmax, int kv_rows, int max_blocks, int num_blocks) {
  const int n = n_accepted[b];
  const int32_t* path = accepted_nodes + static_cast<int64_t>(b) * Nmax;
  if (n < 1 || n > Nmax) return LTD_STATUS_BAD_PATH;
  if (path[0] != 0) return LTD_STATUS_BAD_PATH;
  for (int j = 1; j < n; ++j)
    if (path[j] <= path[j - 1]) return LTD_STATUS_BAD_PATH;
  const int P = prefix_len[b];
  const int64_t capacity =
      block_table ? static_cast<int64_t>(kv_rows) * max_blocks : static_cast<int64_t>(kv_rows);
  if (P < 0 || static_cast<int64_t>(P) + path[n - 1] >= capacity) return LTD_STATUS_BAD_PREFIX;
  if (block_table) {
    const int used = (P + path[n - 1] + kv_rows) / kv_rows;
    for (int j = 0; j < used; ++j) {
      const int32_t blk = block_table[static_cast<int64_t>(b) * max_blocks + j];
      if (blk < 0 || blk >= num_blocks) return LTD_STATUS_BAD_BLOCK;
    }
  }
  return 0;
}

// Lowest (sequence, code) among failing sequences -> *status (0 if none).
__device__ void report(int local_key, int32_t* status) {
  __shared__ int best;
  if (threadIdx.x == 0) best = 0x7FFFFFFF;
  __syncthreads();
  if (local_key != 0x7FFFFFFF) atomicMin(&best, local_key);
  __syncthreads();
  if (threadIdx.x == 0) *status = (best == 0x7FFFFFFF) ? 0 : (best & 0xFF);
}

__global__ void __launch_bounds__(kThreads) validate_tree_kernel(
    const int32_t* block_table, const int32_t* prefix_len, const int32_t* parents,
    const int32_t* n_nodes, int B, int Nmax, int max_prefix, int kv_rows, int max_blocks,
    int num_blocks, int check_cache, int32_t* status) {
  int key = 0x7FFFFFFF;
  for (int b = threadIdx.x; b < B; b += kThreads) {
    const int code = check_tree(block_table, prefix_len, parents, n_nodes, b, Nmax, max_prefix,
                                kv_rows, max_blocks, num_blocks, check_cache != 0);
    if (code != 0 && key == 0x7FFFFFFF) key = (b << 8) | code;
  }
  report(key, status);
}

__global__ void __launch_bounds__(kThreads) validate_path_kernel(
    const int32_t* block_table, const int32_t* prefix_len, const int32_t* accepted_nodes,
    const int32_t* n_accepted, int B, int Nmax, int kv_rows, int max_blocks, int num_blocks,
    int32_t* status) {
  int key = 0x7FFFFFFF;
  for (int b = threadIdx.x; b < B; b += kThreads) {
    const int code = check_path(block_table, prefix_len, accepted_nodes, n_accepted, b, Nmax,
                                kv_rows, max_blocks, num_blocks);
    if (code != 0 && key == 0x7FFFFFFF) key = (b << 8) | code;
  }
  report(key, status);
}

}  // namespace

hipError_t launch_validate_tree(const int32_t* block_table, const int32_t* prefix_len,
                                const int32_t* parents, const int32_t* n_nodes, int B, int Nmax,
                                int max_prefix, int kv_rows, int max_blocks, int num_blocks,
                                bool check_cache, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(validate_tree_kernel, dim3(1), dim3(kThreads), 0, stream, block_table,
                     prefix_len, parents, n_nodes, B, Nmax, max_prefix, kv_rows, max_blocks,
                     num_blocks, check_cache ? 1 : 0, status);
  return hipGetLastError();
}

hipError_t launch_validate_path(const int32_t* block_table, const int32_t* prefix_len,
                                const int32_t* accepted_nodes, const int32_t* n_accepted, int B,
                                int Nmax, int kv_rows, int max_blocks, int num_blocks,
                                int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(validate_path_kernel, dim3(1), dim3(kThreads), 0, stream, block_table,
                     prefix_len, accepted_nodes, n_accepted, B, Nmax, kv_rows, max_blocks,
                     num_blocks, status);
  return hipGetLastError();
}

}  // namespace ltd
