// Launch planning and dispatch for tree attention.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {

hipError_t launch_attn_rowwise(const AttnShape& s, const void* q, const void* k_cache,
                               const void* v_cache, const int32_t* block_table,
                               const int32_t* prefix_len, const int32_t* parents,
                               const int32_t* n_nodes, void* out, float scale,
                               const int32_t* status, hipStream_t stream);

AttnPlan plan_attention(const AttnShape& s, int num_cus) {
  (void)num_cus;
  AttnPlan p{};
  p.rows = (s.Hq / s.Hkv) * s.Nmax;
  p.row_tiles = 1;
  p.tile_rows = p.rows;
  p.split_keys = 0;
  p.max_splits = 1;
  p.mfma = false;
  p.workspace_bytes = 0;
  return p;
}

hipError_t launch_attention(const AttnShape& s, const AttnPlan& plan, const void* q,
                            const void* k_cache, const void* v_cache, const int32_t* block_table,
                            const int32_t* prefix_len, const int32_t* parents,
                            const int32_t* n_nodes, void* out, float scale, void* workspace,
                            const int32_t* status, hipStream_t stream) {
  (void)plan;
  (void)workspace;
  return launch_attn_rowwise(s, q, k_cache, v_cache, block_table, prefix_len, parents, n_nodes,
                             out, scale, status, stream);
}

}  // namespace ltd
