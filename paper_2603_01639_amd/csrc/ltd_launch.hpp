// Host-side launchers shared between the kernel sources and the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ltd {

// validate.hip
hipError_t launch_validate_tree(const int32_t* block_table, const int32_t* prefix_len,
                                const int32_t* parents, const int32_t* n_nodes, int B, int Nmax,
                                int max_prefix, int kv_rows, int max_blocks, int num_blocks,
                                bool check_cache, int32_t* status, hipStream_t stream);
hipError_t launch_validate_path(const int32_t* block_table, const int32_t* prefix_len,
                                const int32_t* accepted_nodes, const int32_t* n_accepted, int B,
                                int Nmax, int kv_rows, int max_blocks, int num_blocks,
                                int32_t* status, hipStream_t stream);

// attn.hip
struct AttnShape {
  int B, Nmax, Hq, Hkv, d, max_prefix, kv_rows, max_blocks, dtype;
};
struct AttnPlan {
  int grid;          // workgroups of the MFMA attention grid (0 on the row-wise path)
  bool mfma;         // bf16 MFMA path (else the row-wise VALU path)
  bool stream;       // stream plan (batches) rather than the split plan (one sequence)
  int split_keys;    // split plan: prefix keys per split (a multiple of the key tile)
  int max_splits;    // split plan: splits of the longest sequence
  int row_tiles;     // split plan: row tiles per (sequence, kv head)
  bool tree_alone;   // split plan: the tree's keys may take a split of their own
  size_t workspace_bytes;
};
AttnPlan plan_attention(const AttnShape& s, int num_cus);
// Workgroups the attention launch uses under a plan (0 on the row-wise path).
int attention_grid(const AttnPlan& p);
hipError_t launch_attention(const AttnShape& s, const AttnPlan& plan, const void* q,
                            const void* k_cache, const void* v_cache, const int32_t* block_table,
                            const int32_t* prefix_len, const int32_t* parents,
                            const int32_t* n_nodes, void* out, float scale, void* workspace,
                            const int32_t* status, hipStream_t stream);

// accept.hip
size_t accept_workspace_bytes(int B, int Nmax, int Voc);
// The allocation-free acceptance: bytes of the per-device scratch array, and
// its device address on the current GPU (nullptr if it cannot be looked up).
size_t accept_noalloc_scratch_bytes();
void* accept_noalloc_scratch();
hipError_t launch_accept(const float* logits, const int32_t* draft_tokens, const int32_t* parents,
                         const int32_t* n_nodes, int B, int Nmax, int Voc, int32_t* pred,
                         int32_t* accepted_nodes, int32_t* out_tokens, int32_t* n_accepted,
                         void* workspace, const int32_t* status, hipStream_t stream);

// compact.hip
hipError_t launch_compact(void* k_cache, void* v_cache, const int32_t* block_table,
                          const int32_t* prefix_len, int32_t* new_prefix_len,
                          const int32_t* accepted_nodes, const int32_t* n_accepted, int B,
                          int Nmax, int Hkv, int row_bytes, int kv_rows, int max_blocks,
                          int num_layers, int64_t layer_stride_bytes, const int32_t* status,
                          hipStream_t stream);

// select.hip
int select_block_threads(int Vpool);
hipError_t launch_validate_pool(const float* scores, const int32_t* pool_parents,
                                const int32_t* pool_size, const int32_t* n_select, int B,
                                int Vpool, int Nmax, int32_t* status, hipStream_t stream);
hipError_t launch_select(const float* scores, const int32_t* pool_parents,
                         const int32_t* pool_tokens, const int32_t* pool_size,
                         const int32_t* n_select, int B, int Vpool, int Nmax, int32_t* selected,
                         int32_t* parents, int32_t* tokens, int32_t* depth, int32_t* n_nodes,
                         const int32_t* status, hipStream_t stream);

// sample.hip
int sampling_chunks(int Voc);
size_t sampling_workspace_bytes(int B, int Nmax, int Voc);
hipError_t launch_sampling(const float* logits, const float* draft_probs,
                           const int32_t* draft_tokens, const int32_t* parents,
                           const int32_t* n_nodes, const float* uniforms, int B, int Nmax,
                           int Voc, float temperature, int32_t* accepted_nodes,
                           int32_t* out_tokens, int32_t* n_accepted, void* workspace,
                           const int32_t* status, hipStream_t stream);

// expand.hip
int expand_chunks(int Voc);
size_t expand_workspace_bytes(int B, int F, int Voc, int W);
hipError_t launch_expand(const float* logits, const int32_t* frontier, int B, int F, int Voc,
                         int W, int W_next, float* scores, int32_t* pool_parents,
                         int32_t* pool_tokens, int32_t* pool_size, int Vpool,
                         int32_t* new_frontier, void* workspace, int32_t* status, bool validate,
                         hipStream_t stream);

// policy.hip
size_t policy_workspace_bytes(int B, int h1, int h2);
hipError_t launch_policy(int layout, const float* scores, const int32_t* pool_size, int Vpool,
                         const int32_t* depth, const int32_t* ctx_len, float pad, int B,
                         int in_dim, const float* w1, const float* b1, int h1, const float* w2,
                         const float* b2, int h2, const float* wo, const float* bo, int n_out,
                         int action_offset, int action_scale, float* logits, int32_t* action,
                         void* workspace, hipStream_t stream);

}  // namespace ltd
