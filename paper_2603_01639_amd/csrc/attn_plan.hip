// Launch planning and dispatch for tree attention: bf16 (head_dim 128 or 64)
// runs on the MFMA kernels, fp32 on the tiled VALU kernel (attn_rowwise.hip).
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {

hipError_t launch_attn_rowwise(const AttnShape& s, const void* q, const void* k_cache,
                               const void* v_cache, const int32_t* block_table,
                               const int32_t* prefix_len, const int32_t* parents,
                               const int32_t* n_nodes, void* out, float scale,
                               const int32_t* status, hipStream_t stream);
bool mfma_supported(const AttnShape& s);
void plan_mfma(const AttnShape& s, int num_cus, AttnPlan* p);
hipError_t launch_attn_mfma(const AttnShape& s, const AttnPlan& p, const void* q,
                            const void* k_cache, const void* v_cache, const int32_t* block_table,
                            const int32_t* prefix_len, const int32_t* parents,
                            const int32_t* n_nodes, void* out, float scale, void* workspace,
                            const int32_t* status, hipStream_t stream);

AttnPlan plan_attention(const AttnShape& s, int num_cus) {
  AttnPlan p{};
  if (mfma_supported(s)) {
    plan_mfma(s, num_cus, &p);
    return p;
  }
  p.grid = 0;
  p.mfma = false;
  p.workspace_bytes = 0;
  return p;
}

hipError_t launch_attention(const AttnShape& s, const AttnPlan& plan, const void* q,
                            const void* k_cache, const void* v_cache, const int32_t* block_table,
                            const int32_t* prefix_len, const int32_t* parents,
                            const int32_t* n_nodes, void* out, float scale, void* workspace,
                            const int32_t* status, hipStream_t stream) {
  if (plan.mfma)
    return launch_attn_mfma(s, plan, q, k_cache, v_cache, block_table, prefix_len, parents,
                            n_nodes, out, scale, workspace, status, stream);
  return launch_attn_rowwise(s, q, k_cache, v_cache, block_table, prefix_len, parents, n_nodes,
                             out, scale, status, stream);
}

}  // namespace ltd
