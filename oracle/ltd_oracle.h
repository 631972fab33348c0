/*
 * CPU oracle for the tree-verification step of Learning-to-Draft speculative
 * decoding (arXiv 2603.01639).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the slow, plain, fp64 statement of
 * what the GPU path computes.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it.  It shares no source, header or
 * helper with the HIP library, and the HIP library never calls it.
 *
 * All pointers are HOST pointers.  Layouts match the HIP library's contract:
 *   q            [B][Nmax][Hq][d]           f32 or bf16 (stored as uint16 bit patterns)
 *   k/v cache    contiguous [B][Hkv][cap][d]  (block_table == NULL)
 *                paged      [num_blocks][Hkv][block_size][d] with
 *                           block_table [B][max_blocks]
 *   parents      [B][Nmax]  parents[b][0] = -1, 0 <= parents[b][i] < i
 *   out          [B][Nmax][Hq][d]  fp64; rows i >= n_nodes[b] are left untouched
 *   node_mask    [B][Nmax] uint8 or NULL: when given, only nodes with a nonzero
 *                entry are computed (sampled checks of large workloads)
 *
 * Return values: 0 on success, a negative LTDO_E* code for a malformed call,
 * or a positive LTDO_STATUS_* code for malformed data (nothing is written then).
 */
#ifndef LTD_ORACLE_H
#define LTD_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LTDO_EINVAL (-1)
#define LTDO_EUNSUPPORTED (-2)

#define LTDO_DTYPE_F32 0
#define LTDO_DTYPE_BF16 1

#define LTDO_STATUS_BAD_NNODES 1
#define LTDO_STATUS_BAD_PARENT 2
#define LTDO_STATUS_BAD_PREFIX 3
#define LTDO_STATUS_BAD_BLOCK 4
#define LTDO_STATUS_BAD_PATH 5
#define LTDO_STATUS_BAD_SCORE 6

/* Tree attention (paper section 3.2: candidates flattened with a tree
 * attention mask, verified in one target pass).  Node i of sequence b attends
 * to the prefix rows [0, P_b) and to the tree rows P_b + j for every j on its
 * own root path; q head h reads kv head h / (Hq / Hkv). */
int ltd_oracle_tree_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* block_table, const int32_t* prefix_len,
                                const int32_t* parents, const int32_t* n_nodes,
                                const uint8_t* node_mask, double* out, int B, int Nmax, int Hq,
                                int Hkv, int d, int kv_rows, int max_blocks, int num_blocks,
                                double scale, int dtype);

/* Greedy acceptance (paper section 3.2, "Draft Tree Verification"): per-node
 * target argmax, then the longest root path whose draft tokens all equal the
 * target prediction at their parent, then the bonus token. */
int ltd_oracle_tree_accept(const float* logits, const int32_t* draft_tokens,
                           const int32_t* parents, const int32_t* n_nodes, int B, int Nmax,
                           int Voc, int32_t* pred, int32_t* accepted_nodes,
                           int32_t* out_tokens, int32_t* n_accepted);

/* KV compaction: the accepted path's rows move to [P_b, P_b + n_accepted[b]);
 * new_prefix_len[b] = P_b + n_accepted[b].  elem_bytes is 2 or 4. */
int ltd_oracle_kv_compact(void* k_cache, void* v_cache, const int32_t* block_table,
                          const int32_t* prefix_len, int32_t* new_prefix_len,
                          const int32_t* accepted_nodes, const int32_t* n_accepted, int B,
                          int Nmax, int Hkv, int d, int kv_rows, int max_blocks, int num_blocks,
                          int num_layers, int64_t layer_stride_elems, int elem_bytes);

/* Candidate token selection (paper section 3.2, "Candidate Token
 * Selection"): from a draft tree of pool_size[b] candidates (pool_parents
 * [B][Vpool], pool_parents[b][0] = -1 and 0 <= pool_parents[b][i] < i; a
 * cumulative score per candidate, larger = more probable, never above its
 * parent's), keep the V = min(n_select[b], pool_size[b]) candidates ranked
 * first by (score descending, pool index ascending), and flatten them in pool
 * order.  Outputs [B][Nmax] (entries past V untouched): selected = pool index
 * of node k, parents in the new order (-1 for the root), tokens, depth;
 * n_nodes[b] = V. */
int ltd_oracle_select_candidates(const float* scores, const int32_t* pool_parents,
                                 const int32_t* pool_tokens, const int32_t* pool_size,
                                 const int32_t* n_select, int B, int Vpool, int Nmax,
                                 int32_t* selected, int32_t* parents, int32_t* tokens,
                                 int32_t* depth, int32_t* n_nodes);

/* Acceptance by recursive rejection sampling at temperature T > 0 (the
 * paper's T = 1 setting; the rule is the baseline's, not printed in the
 * paper).  Same tree arguments and path/token outputs as
 * ltd_oracle_tree_accept; draft_probs [B][Nmax][Voc] holds, for every node
 * with children, the draft distribution its children were drawn from
 * (without replacement, in ascending node order); uniforms [B][Nmax][2] in
 * [0, 1): [c][0] decides child c, [u][1] the bonus token drawn at u.  Optional
 * final_dist [B][Voc] receives the distribution the bonus was drawn from and
 * min_margin [B] the smallest relative gap of an accept test. */
int ltd_oracle_tree_accept_sampling(const float* logits, const float* draft_probs,
                                    const int32_t* draft_tokens, const int32_t* parents,
                                    const int32_t* n_nodes, const float* uniforms, int B, int Nmax,
                                    int Voc, double temperature, int32_t* accepted_nodes,
                                    int32_t* out_tokens, int32_t* n_accepted, double* final_dist,
                                    double* min_margin);

/* One round of draft tree expansion (paper section 3.2, "Draft Tree
 * Generation").  logits [B][F][Voc]: draft logits at the F frontier nodes,
 * whose pool indices are frontier [B][F].  Appends F*W children per sequence
 * to the pool ([B][Vpool] scores, parents, tokens) at pool_size[b] onwards:
 * for each frontier node in order, its W tokens of largest logit (equal
 * logits: lower token index first), each scored parent score + log-softmax
 * of its logit (double, stored as float).  Then new_frontier [B][W_next] =
 * the W_next new children of highest score (equal: lower pool index first),
 * best first, and pool_size[b] += F*W.  Returns a status code when a pool
 * would overflow or a frontier index is not in the pool. */
int ltd_oracle_draft_expand(const float* logits, const int32_t* frontier, int B, int F, int Voc,
                            int W, int W_next, float* scores, int32_t* pool_parents,
                            int32_t* pool_tokens, int32_t* pool_size, int Vpool,
                            int32_t* new_frontier);

/* Threads the oracle's parallel loops use (OpenMP), for reporting. */
int ltd_oracle_num_threads(void);
/* Threads for the next parallel regions (n >= 1; timing only: results do not
 * depend on it). */
void ltd_oracle_set_num_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
