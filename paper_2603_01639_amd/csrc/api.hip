// The C ABI of ltd_verify (declared in ltd_verify.h): argument checks, launch
// plans and kernel dispatch.  No allocation, no synchronisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>

#include "ltd_launch.hpp"
#include "ltd_verify.h"

namespace {

constexpr int kMaxDevices = 64;

int device_cu_count() {
  static std::once_flag once[kMaxDevices];
  static int cus[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  std::call_once(once[dev], [dev] {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cus[dev] = n;
  });
  return cus[dev];
}

bool attn_args_ok(int B, int Nmax, int Hq, int Hkv, int d, int max_prefix, int dtype) {
  (void)d;
  (void)dtype;
  return B >= 0 && Nmax >= 1 && Nmax <= LTD_MAX_NODES && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0 &&
         max_prefix >= 0;
}

bool attn_supported(int d, int dtype) {
  return (dtype == LTD_DTYPE_F32 || dtype == LTD_DTYPE_BF16) && (d == 64 || d == 128);
}

ltd::AttnShape make_shape(int B, int Nmax, int Hq, int Hkv, int d, int max_prefix, int kv_rows,
                          int max_blocks, int dtype) {
  return ltd::AttnShape{B, Nmax, Hq, Hkv, d, max_prefix, kv_rows, max_blocks, dtype};
}

}  // namespace

extern "C" {

const char* ltd_version(void) { return "ltd_verify 0.1 (gfx950)"; }

size_t ltd_tree_verify_attn_workspace_size(int B, int Nmax, int Hq, int Hkv, int d, int max_prefix,
                                           int dtype) {
  if (!attn_args_ok(B, Nmax, Hq, Hkv, d, max_prefix, dtype) || !attn_supported(d, dtype)) return 0;
  // The largest need over the layouts: a contiguous cache, and a paged one
  // with one-row blocks (the smallest blocks shorten the split plan's splits
  // the most, and send a batch from the stream plan to the split plan).
  const ltd::AttnShape contiguous =
      make_shape(B, Nmax, Hq, Hkv, d, max_prefix, max_prefix + Nmax, 0, dtype);
  const ltd::AttnShape tiny_blocks = make_shape(B, Nmax, Hq, Hkv, d, max_prefix, 1, 1, dtype);
  const int cus = device_cu_count();
  return std::max(ltd::plan_attention(contiguous, cus).workspace_bytes,
                  ltd::plan_attention(tiny_blocks, cus).workspace_bytes);
}

int ltd_tree_verify_attn_grid(int B, int Nmax, int Hq, int Hkv, int d, int max_prefix, int dtype,
                              int kv_rows, int paged) {
  if (!attn_args_ok(B, Nmax, Hq, Hkv, d, max_prefix, dtype) || !attn_supported(d, dtype) ||
      kv_rows < 1)
    return -1;
  const ltd::AttnShape s =
      make_shape(B, Nmax, Hq, Hkv, d, max_prefix, kv_rows, paged ? 1 : 0, dtype);
  return ltd::attention_grid(ltd::plan_attention(s, device_cu_count()));
}

int ltd_tree_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* block_table, const int32_t* prefix_len,
                         const int32_t* parents, const int32_t* n_nodes, void* out, int B, int Nmax,
                         int Hq, int Hkv, int d, int max_prefix, int kv_rows, int max_blocks,
                         int num_blocks, float scale, int dtype, void* workspace,
                         size_t workspace_bytes, int validate, int32_t* status, void* stream) {
  if (!attn_args_ok(B, Nmax, Hq, Hkv, d, max_prefix, dtype) || kv_rows < 1) return LTD_EINVAL;
  if (!(scale > 0.f) || !std::isfinite(scale)) return LTD_EINVAL;
  if (!attn_supported(d, dtype)) return LTD_EUNSUPPORTED;
  if (block_table && (max_blocks < 1 || num_blocks < 1)) return LTD_EINVAL;
  if (validate && !status) return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!q || !k_cache || !v_cache || !prefix_len || !parents || !n_nodes || !out) return LTD_EINVAL;
  const ltd::AttnShape s = make_shape(B, Nmax, Hq, Hkv, d, max_prefix, kv_rows, max_blocks, dtype);
  const ltd::AttnPlan plan = ltd::plan_attention(s, device_cu_count());
  if (plan.workspace_bytes > 0 && (!workspace || workspace_bytes < plan.workspace_bytes))
    return LTD_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (validate) {
    if (ltd::launch_validate_tree(block_table, prefix_len, parents, n_nodes, B, Nmax, max_prefix,
                                  kv_rows, max_blocks, num_blocks, true, status, st) != hipSuccess)
      return LTD_EHIP;
  }
  if (ltd::launch_attention(s, plan, q, k_cache, v_cache, block_table, prefix_len, parents,
                            n_nodes, out, scale, workspace, validate ? status : nullptr,
                            st) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

size_t ltd_tree_accept_workspace_size(int B, int Nmax, int Voc) {
  if (B < 0 || Nmax < 1 || Nmax > LTD_MAX_NODES || Voc < 1) return 0;
  return ltd::accept_workspace_bytes(B, Nmax, Voc);
}

int ltd_tree_accept(const float* logits, const int32_t* draft_tokens, const int32_t* parents,
                    const int32_t* n_nodes, int B, int Nmax, int Voc, int32_t* pred,
                    int32_t* accepted_nodes, int32_t* out_tokens, int32_t* n_accepted,
                    void* workspace, size_t workspace_bytes, int validate, int32_t* status,
                    void* stream) {
  if (B < 0 || Nmax < 1 || Nmax > LTD_MAX_NODES || Voc < 1) return LTD_EINVAL;
  if (validate && !status) return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!logits || !draft_tokens || !parents || !n_nodes || !pred || !accepted_nodes ||
      !out_tokens || !n_accepted)
    return LTD_EINVAL;
  const size_t need = ltd::accept_workspace_bytes(B, Nmax, Voc);
  if (!workspace || workspace_bytes < need) return LTD_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (validate) {
    if (ltd::launch_validate_tree(nullptr, nullptr, parents, n_nodes, B, Nmax, 0, 1, 0, 0, false,
                                  status, st) != hipSuccess)
      return LTD_EHIP;
  }
  if (ltd::launch_accept(logits, draft_tokens, parents, n_nodes, B, Nmax, Voc, pred,
                         accepted_nodes, out_tokens, n_accepted, workspace,
                         validate ? status : nullptr, st) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

size_t ltd_tree_accept_noalloc_max_bytes(void) { return ltd::accept_noalloc_scratch_bytes(); }

int ltd_tree_accept_noalloc(const float* logits, const int32_t* draft_tokens,
                            const int32_t* parents, const int32_t* n_nodes, int B, int Nmax,
                            int Voc, int32_t* pred, int32_t* accepted_nodes, int32_t* out_tokens,
                            int32_t* n_accepted, int validate, int32_t* status, void* stream) {
  if (B < 0 || Nmax < 1 || Nmax > LTD_MAX_NODES || Voc < 1) return LTD_EINVAL;
  if (validate && !status) return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!logits || !draft_tokens || !parents || !n_nodes || !pred || !accepted_nodes ||
      !out_tokens || !n_accepted)
    return LTD_EINVAL;
  if (ltd::accept_workspace_bytes(B, Nmax, Voc) > ltd::accept_noalloc_scratch_bytes())
    return LTD_EWORKSPACE;
  void* scratch = ltd::accept_noalloc_scratch();
  if (!scratch) return LTD_EHIP;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (validate) {
    if (ltd::launch_validate_tree(nullptr, nullptr, parents, n_nodes, B, Nmax, 0, 1, 0, 0, false,
                                  status, st) != hipSuccess)
      return LTD_EHIP;
  }
  if (ltd::launch_accept(logits, draft_tokens, parents, n_nodes, B, Nmax, Voc, pred,
                         accepted_nodes, out_tokens, n_accepted, scratch,
                         validate ? status : nullptr, st) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

int ltd_kv_compact(void* k_cache, void* v_cache, const int32_t* block_table,
                   const int32_t* prefix_len, int32_t* new_prefix_len,
                   const int32_t* accepted_nodes, const int32_t* n_accepted, int B, int Nmax,
                   int Hkv, int d, int kv_rows, int max_blocks, int num_blocks, int num_layers,
                   int64_t layer_stride_elems, int dtype, int validate, int32_t* status,
                   void* stream) {
  if (B < 0 || Nmax < 1 || Nmax > LTD_MAX_NODES || Hkv < 1 || d < 1 || kv_rows < 1 ||
      num_layers < 1 || layer_stride_elems < 0)
    return LTD_EINVAL;
  if (dtype != LTD_DTYPE_F32 && dtype != LTD_DTYPE_BF16) return LTD_EUNSUPPORTED;
  const int elem = dtype == LTD_DTYPE_F32 ? 4 : 2;
  const int row_bytes = d * elem;
  if (row_bytes % 16 != 0 || row_bytes > 16 * 256) return LTD_EUNSUPPORTED;
  if (block_table && (max_blocks < 1 || num_blocks < 1)) return LTD_EINVAL;
  if (validate && !status) return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!k_cache || !v_cache || !prefix_len || !new_prefix_len || !accepted_nodes || !n_accepted)
    return LTD_EINVAL;
  if (new_prefix_len == prefix_len) return LTD_EINVAL;
  if (num_layers > 1 && layer_stride_elems == 0) return LTD_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (validate) {
    if (ltd::launch_validate_path(block_table, prefix_len, accepted_nodes, n_accepted, B, Nmax,
                                  kv_rows, max_blocks, num_blocks, status, st) != hipSuccess)
      return LTD_EHIP;
  }
  if (ltd::launch_compact(k_cache, v_cache, block_table, prefix_len, new_prefix_len,
                          accepted_nodes, n_accepted, B, Nmax, Hkv, row_bytes, kv_rows, max_blocks,
                          num_layers, layer_stride_elems * elem, validate ? status : nullptr,
                          st) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

int ltd_select_candidates(const float* scores, const int32_t* pool_parents,
                          const int32_t* pool_tokens, const int32_t* pool_size,
                          const int32_t* n_select, int B, int Vpool, int Nmax, int32_t* selected,
                          int32_t* parents, int32_t* tokens, int32_t* depth, int32_t* n_nodes,
                          int validate, int32_t* status, void* stream) {
  if (B < 0 || Vpool < 1 || Vpool > LTD_MAX_POOL || Nmax < 1 || Nmax > LTD_MAX_NODES)
    return LTD_EINVAL;
  if (validate && !status) return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!scores || !pool_parents || !pool_tokens || !pool_size || !n_select || !parents ||
      !tokens || !n_nodes)
    return LTD_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (validate) {
    if (ltd::launch_validate_pool(scores, pool_parents, pool_size, n_select, B, Vpool, Nmax,
                                  status, st) != hipSuccess)
      return LTD_EHIP;
  }
  if (ltd::launch_select(scores, pool_parents, pool_tokens, pool_size, n_select, B, Vpool, Nmax,
                         selected, parents, tokens, depth, n_nodes, validate ? status : nullptr,
                         st) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

size_t ltd_tree_accept_sampling_workspace_size(int B, int Nmax, int Voc) {
  if (B < 0 || Nmax < 1 || Nmax > LTD_MAX_NODES || Voc < 1 ||
      ltd::sampling_chunks(Voc) > LTD_SAMPLING_MAX_CHUNKS)
    return 0;
  return ltd::sampling_workspace_bytes(B, Nmax, Voc);
}

int ltd_tree_accept_sampling(const float* logits, const float* draft_probs,
                             const int32_t* draft_tokens, const int32_t* parents,
                             const int32_t* n_nodes, const float* uniforms, int B, int Nmax,
                             int Voc, float temperature, int32_t* accepted_nodes,
                             int32_t* out_tokens, int32_t* n_accepted, void* workspace,
                             size_t workspace_bytes, int validate, int32_t* status, void* stream) {
  if (B < 0 || Nmax < 1 || Nmax > LTD_MAX_NODES || Voc < 1 ||
      ltd::sampling_chunks(Voc) > LTD_SAMPLING_MAX_CHUNKS || !(temperature > 0.f) ||
      !std::isfinite(temperature))
    return LTD_EINVAL;
  if (validate && !status) return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!logits || !draft_probs || !draft_tokens || !parents || !n_nodes || !uniforms ||
      !accepted_nodes || !out_tokens || !n_accepted)
    return LTD_EINVAL;
  if (!workspace || workspace_bytes < ltd::sampling_workspace_bytes(B, Nmax, Voc))
    return LTD_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (validate) {
    if (ltd::launch_validate_tree(nullptr, nullptr, parents, n_nodes, B, Nmax, 0, 1, 0, 0, false,
                                  status, st) != hipSuccess)
      return LTD_EHIP;
  }
  if (ltd::launch_sampling(logits, draft_probs, draft_tokens, parents, n_nodes, uniforms, B, Nmax,
                           Voc, temperature, accepted_nodes, out_tokens, n_accepted, workspace,
                           validate ? status : nullptr, st) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

namespace {
bool expand_args_ok(int B, int F, int Voc, int W) {
  return B >= 0 && F >= 1 && W >= 1 && W <= LTD_EXPAND_MAX_W && Voc >= W &&
         ltd::expand_chunks(Voc) <= LTD_EXPAND_MAX_CHUNKS && F * W <= LTD_EXPAND_MAX_CHILDREN;
}
}  // namespace

size_t ltd_draft_expand_workspace_size(int B, int F, int Voc, int W) {
  if (!expand_args_ok(B, F, Voc, W)) return 0;
  return ltd::expand_workspace_bytes(B, F, Voc, W);
}

int ltd_draft_expand(const float* logits, const int32_t* frontier, int B, int F, int Voc, int W,
                     int W_next, float* scores, int32_t* pool_parents, int32_t* pool_tokens,
                     int32_t* pool_size, int Vpool, int32_t* new_frontier, void* workspace,
                     size_t workspace_bytes, int validate, int32_t* status, void* stream) {
  if (Voc < 1 || F < 1 || W < 1 || F > LTD_EXPAND_MAX_CHILDREN || !expand_args_ok(B, F, Voc, W) ||
      W_next < 1 || W_next > F * W || Vpool < 1)
    return LTD_EINVAL;
  if (validate && !status) return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!logits || !frontier || !scores || !pool_parents || !pool_tokens || !pool_size ||
      !new_frontier)
    return LTD_EINVAL;
  if (!workspace || workspace_bytes < ltd::expand_workspace_bytes(B, F, Voc, W))
    return LTD_EWORKSPACE;
  if (ltd::launch_expand(logits, frontier, B, F, Voc, W, W_next, scores, pool_parents,
                         pool_tokens, pool_size, Vpool, new_frontier, workspace, status,
                         validate != 0, static_cast<hipStream_t>(stream)) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

size_t ltd_policy_workspace_size(int B, int h1, int h2) {
  if (B < 0 || h1 < 1 || h1 > LTD_POLICY_MAX_HIDDEN || h2 < 0 || h2 > LTD_POLICY_MAX_HIDDEN)
    return 0;
  return ltd::policy_workspace_bytes(B, h1, h2);
}

int ltd_policy_forward(int layout, const float* scores, const int32_t* pool_size, int Vpool,
                       const int32_t* depth, const int32_t* ctx_len, float pad, int B, int in_dim,
                       const float* w1, const float* b1, int h1, const float* w2, const float* b2,
                       int h2, const float* wo, const float* bo, int n_out, int action_offset,
                       int action_scale, float* logits, int32_t* action, void* workspace,
                       size_t workspace_bytes, void* stream) {
  if ((layout != LTD_POLICY_SIZE && layout != LTD_POLICY_DEPTH) || B < 0 || Vpool < 1 ||
      in_dim < 3 || in_dim > LTD_POLICY_MAX_IN || h1 < 1 || h1 > LTD_POLICY_MAX_HIDDEN || h2 < 0 ||
      h2 > LTD_POLICY_MAX_HIDDEN || n_out < 1 || n_out > LTD_POLICY_MAX_OUT)
    return LTD_EINVAL;
  if (B == 0) return LTD_OK;
  if (!scores || !pool_size || !depth || !ctx_len || !w1 || !b1 || !wo || !bo || !logits ||
      !action || (h2 > 0 && (!w2 || !b2)))
    return LTD_EINVAL;
  if (!workspace || workspace_bytes < ltd::policy_workspace_bytes(B, h1, h2))
    return LTD_EWORKSPACE;
  if (ltd::launch_policy(layout, scores, pool_size, Vpool, depth, ctx_len, pad, B, in_dim, w1, b1,
                         h1, w2, b2, h2, wo, bo, n_out, action_offset, action_scale, logits, action,
                         workspace, static_cast<hipStream_t>(stream)) != hipSuccess)
    return LTD_EHIP;
  return LTD_OK;
}

}  // extern "C"
