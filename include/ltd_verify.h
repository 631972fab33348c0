/*
 * ltd_verify: the tree-verification step of Learning-to-Draft speculative
 * decoding (arXiv 2603.01639, section 3.2) on AMD Instinct MI355X (gfx950).
 *
 * One verification step of a draft-and-verify cycle is three calls on one
 * stream, with no host synchronisation between them:
 *
 *   ltd_tree_verify_attn  the target model's attention over its KV-cache prefix
 *                         plus the N flattened draft-tree candidates, each
 *                         candidate seeing only the prefix and its own ancestors
 *                         (the tree attention mask of section 3.2, "Candidate
 *                         Token Selection" / "Draft Tree Verification");
 *   ltd_tree_accept       the target's prediction at every node (vocabulary
 *                         argmax of its logits) and greedy acceptance: the
 *                         longest root path whose draft tokens all equal the
 *                         prediction at their parent, plus the target's token at
 *                         the first mismatch (section 3.2, "Draft Tree
 *                         Verification");
 *   ltd_kv_compact        the accepted path's K/V rows move next to the prefix
 *                         and the rest of the candidates are discarded (same
 *                         paragraph: the remainder after the first error is
 *                         dropped).
 *
 * The steps before it have calls of their own:
 *
 *   ltd_draft_expand      one round of the draft tree's beam expansion
 *                         (section 3.2, "Draft Tree Generation");
 *   ltd_policy_forward    the size and depth policies' decisions (section 4,
 *                         appendix A.2);
 *   ltd_select_candidates the V most probable candidates of the draft tree's
 *                         pool, flattened into the tree the three calls above
 *                         verify (section 3.2, "Candidate Token Selection").
 *
 * Conventions for every call
 * --------------------------
 * - All array pointers are DEVICE pointers, owned by the caller.  The library
 *   never allocates, frees or synchronises; every call is asynchronous on
 *   `stream` (a hipStream_t passed as void*, NULL = the default stream).
 * - Return value: LTD_OK, or a negative LTD_E* code when the call itself is
 *   malformed (nothing is launched then).  These checks use only the scalar
 *   arguments and pointer nullness.
 * - Data-dependent checks (tree shape, prefix bounds, block ids, paths) run on
 *   the device only when `validate != 0`: a validation kernel writes an
 *   LTD_STATUS_* code to `*status` (0 when the data is well formed) and, when
 *   it is nonzero, the step's kernels write nothing.  The code reported is the
 *   one of the lowest failing sequence index, with checks in the order the
 *   codes are numbered.  With `validate == 0`, malformed data is undefined
 *   behaviour and `status` may be NULL.
 * - Trees: N counts the root.  parents[b][0] = -1 and 0 <= parents[b][i] < i
 *   (a topological order); node 0 is the root (the previous cycle's bonus
 *   token).  Tree node i of sequence b sits at logical cache row P_b + i.
 * - Calls on different streams that touch the same buffers race; calls that
 *   share a workspace must be stream-ordered.
 */
#ifndef LTD_VERIFY_H
#define LTD_VERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LTD_OK 0
#define LTD_EINVAL (-1)       /* null pointer or out-of-range scalar argument */
#define LTD_EUNSUPPORTED (-2) /* dtype or head_dim the kernels do not implement */
#define LTD_EWORKSPACE (-3)   /* workspace missing or smaller than the query says */
#define LTD_EHIP (-4)         /* a HIP runtime call or kernel launch failed */

#define LTD_DTYPE_F32 0  /* IEEE binary32 */
#define LTD_DTYPE_BF16 1 /* bfloat16 */

#define LTD_STATUS_OK 0
#define LTD_STATUS_BAD_NNODES 1 /* n_nodes[b] outside [1, Nmax] */
#define LTD_STATUS_BAD_PARENT 2 /* parents[b][0] != -1 or parents[b][i] outside [0, i) */
#define LTD_STATUS_BAD_PREFIX 3 /* prefix_len[b] < 0, > max_prefix, or rows past capacity */
#define LTD_STATUS_BAD_BLOCK 4  /* a block id the sequence uses is outside [0, num_blocks) */
#define LTD_STATUS_BAD_PATH 5   /* accepted path not 0 = p_0 < p_1 < ..., or n_accepted out of range */
#define LTD_STATUS_BAD_SCORE 6  /* a pool score is NaN or above its parent's */

#define LTD_MAX_NODES 256 /* largest Nmax (the paper's size policy spans V in [20, 240]) */
#define LTD_MAX_POOL 1024 /* largest draft pool (1 + W + (D-2) W^2 = 1011 at W = 10, D = 12) */

#define LTD_SAMPLING_MAX_CHUNKS 64  /* sampling vocabulary up to 64 * 4096 = 262144 entries */

#define LTD_EXPAND_MAX_W 16          /* children per frontier node (the paper's W is 10) */
#define LTD_EXPAND_MAX_CHUNKS 64     /* vocabulary up to 64 * 4096 = 262144 entries */
#define LTD_EXPAND_MAX_CHILDREN 256  /* F * W per round */

#define LTD_POLICY_SIZE 0          /* state [D, L, score of every pool candidate, pad ...] */
#define LTD_POLICY_DEPTH 1         /* state [scores of the newest in_dim-2 candidates, D, L] */
#define LTD_POLICY_MAX_IN 1024     /* state width (the size policy's is 2 + 1011) */
#define LTD_POLICY_MAX_HIDDEN 1024 /* hidden width (the paper's widest layer) */
#define LTD_POLICY_MAX_OUT 64      /* output logits (12 size actions, 2 depth actions) */

/*
 * Tree attention (section 3.2: candidates flattened with a tree attention
 * mask, verified in one target pass).
 *
 * For every sequence b, node i < n_nodes[b] and query head h (kv head
 * g = h / (Hq / Hkv)):
 *     out[b][i][h] = softmax_t(scale * <q[b][i][h], K[b][g][t]>) . V[b][g][t]
 * over the visible rows t = {0, ..., P_b - 1} u {P_b + j : j on the root path of
 * node i, i included}.  Accumulation is fp32; out has the input dtype.  On
 * the bf16 path the exponent of each weight is formed in fp32 as
 * s*c - m*c (c = scale * log2(e), m a running row maximum), exact to about
 * |m*c| * 2^-24: scaled scores up to ~1e5 in magnitude keep the bf16 output
 * accuracy (max-abs error ~1e-2 against exact arithmetic).
 *
 *   q           [B][Nmax][Hq][d] (dtype): the tree nodes' queries (position
 *               encoding already applied by the caller).
 *   k_cache,    contiguous (block_table == NULL): [B][Hkv][kv_rows][d], kv_rows
 *   v_cache     = capacity per sequence;
 *               paged: [num_blocks][Hkv][kv_rows][d], kv_rows = block size,
 *               logical row r of sequence b in block block_table[b][r / kv_rows].
 *               The tree's own K/V rows must already be written at P_b .. P_b+n-1.
 *   block_table [B][max_blocks] int32 or NULL.
 *   prefix_len  [B] int32, P_b >= 0.  max_prefix >= every P_b (host bound used
 *               to size the launch; checked on the device when validate != 0).
 *   parents     [B][Nmax] int32, n_nodes [B] int32 in [1, Nmax].
 *   out         [B][Nmax][Hq][d] (dtype); rows i >= n_nodes[b] are not written.
 *   Hq % Hkv == 0, d in {64, 128}, 1 <= Nmax <= LTD_MAX_NODES.
 *   scale       softmax scale, finite and > 0 (1/sqrt(d) for standard
 *               attention); anything else is LTD_EINVAL.
 *   workspace   device scratch of at least ltd_tree_verify_attn_workspace_size()
 *               bytes for the same (B, Nmax, Hq, Hkv, d, max_prefix, dtype) (that
 *               size covers every cache layout; it is 0 on the fp32 path,
 *               and workspace may then be NULL); it holds the partial results
 *               of units cut between workgroups, needs no initialisation and
 *               is garbage afterwards.
 */
size_t ltd_tree_verify_attn_workspace_size(int B, int Nmax, int Hq, int Hkv, int d, int max_prefix,
                                           int dtype);

int ltd_tree_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* block_table, const int32_t* prefix_len,
                         const int32_t* parents, const int32_t* n_nodes, void* out, int B, int Nmax,
                         int Hq, int Hkv, int d, int max_prefix, int kv_rows, int max_blocks,
                         int num_blocks, float scale, int dtype, void* workspace,
                         size_t workspace_bytes, int validate, int32_t* status, void* stream);

/*
 * Greedy acceptance (section 3.2, "Draft Tree Verification").
 *
 *   logits        [B][Nmax][Voc] fp32: the target's logits at every node.
 *   draft_tokens  [B][Nmax] int32; draft_tokens[b][0] is the root token.
 *   parents, n_nodes as for attention.
 * Outputs (entries past n_nodes[b] / n_accepted[b] are not written):
 *   pred           [B][Nmax] int32: argmax_v logits[b][i][v]; ties go to the
 *                  lowest v and -0.0 equals +0.0 (NaN logits are undefined).
 *   accepted_nodes [B][Nmax] int32: the accepted root path, root first
 *                  (accepted_nodes[b][0] = 0).  Node c is accepted when its
 *                  parent is and draft_tokens[b][c] == pred[b][parent(c)]; the
 *                  path ends at the deepest accepted node, the smallest index
 *                  among equally deep ones.
 *   out_tokens     [B][Nmax] int32: draft tokens of the accepted non-root path
 *                  nodes, then the bonus token pred[b][leaf].
 *   n_accepted     [B] int32: path length = number of emitted tokens (L_A).
 *   workspace      at least ltd_tree_accept_workspace_size(B, Nmax, Voc) bytes.
 */
size_t ltd_tree_accept_workspace_size(int B, int Nmax, int Voc);

int ltd_tree_accept(const float* logits, const int32_t* draft_tokens, const int32_t* parents,
                    const int32_t* n_nodes, int B, int Nmax, int Voc, int32_t* pred,
                    int32_t* accepted_nodes, int32_t* out_tokens, int32_t* n_accepted,
                    void* workspace, size_t workspace_bytes, int validate, int32_t* status,
                    void* stream);

/*
 * Greedy acceptance without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results and validation as
 * ltd_tree_accept, minus the workspace: the argmax partials go to a scratch
 * array that the library holds on each GPU for the life of the process
 * (ltd_tree_accept_noalloc_max_bytes() bytes, 4 MiB).  The call allocates
 * nothing and frees nothing.
 *
 * Limits: ltd_tree_accept_workspace_size(B, Nmax, Voc) must not exceed
 * ltd_tree_accept_noalloc_max_bytes() (B * Nmax * ceil(Voc / 16384) * 8 bytes;
 * e.g. B = 16, Nmax = 256 and Voc = 262144 use 1 MiB), else LTD_EWORKSPACE and
 * nothing is launched.  LTD_EHIP if the scratch's device address cannot be
 * looked up on the current GPU.
 * Every call on one GPU shares that GPU's scratch and keeps the last call's
 * contents there (no call depends on them): calls that overlap on one GPU
 * (different streams without ordering between them) race and give undefined
 * results.
 */
size_t ltd_tree_accept_noalloc_max_bytes(void);

int ltd_tree_accept_noalloc(const float* logits, const int32_t* draft_tokens,
                            const int32_t* parents, const int32_t* n_nodes, int B, int Nmax,
                            int Voc, int32_t* pred, int32_t* accepted_nodes, int32_t* out_tokens,
                            int32_t* n_accepted, int validate, int32_t* status, void* stream);

/*
 * Acceptance at temperature T > 0 (the paper's T = 1 setting; its rule is
 * the baseline's, not printed in the paper): recursive rejection sampling
 * over each node's children, which must have been drawn without replacement
 * from the node's draft distribution, in ascending node order.
 *
 * At node u, with target P = softmax(logits[u] / T) and draft distribution
 * Q = draft_probs[u] / sum(draft_probs[u]), child c (token x) is accepted
 * when uniforms[c][0] * Q(x) < P(x), i.e. with probability min(1, P/Q), and
 * the walk moves to c.  On rejection P becomes max(P - Q, 0) renormalised and
 * Q drops x.  When no child is accepted (or u is a leaf) the bonus token is
 * the inverse-CDF sample of P at uniforms[u][1].  The emitted tokens are then
 * distributed exactly as the target's own sampling.
 *
 *   logits       [B][Nmax][Voc] float32, target logits at every node.
 *   draft_probs  [B][Nmax][Voc] float32, read only for nodes with children
 *                (non-negative, positive sum).
 *   draft_tokens [B][Nmax] int32 in [0, Voc); siblings distinct.
 *   uniforms     [B][Nmax][2] float32 in [0, 1).
 *   temperature  finite and > 0, else LTD_EINVAL.
 *   Outputs as ltd_tree_accept: accepted_nodes, out_tokens (the accepted
 *   drafts, then the bonus), n_accepted.  Entries past n_accepted untouched.
 *   Voc <= 4096 * LTD_SAMPLING_MAX_CHUNKS.
 *   workspace: ltd_tree_accept_sampling_workspace_size(B, Nmax, Voc) bytes.
 * Decisions are taken on float32 element arithmetic with double sums, so they
 * can differ from an exact evaluation only where a uniform lies within about
 * 1e-6 (relative) of its threshold.  The draft mass left after each rejection
 * is summed over the tokens not rejected, so it stays exact to double
 * rounding however little of it is left.
 */
size_t ltd_tree_accept_sampling_workspace_size(int B, int Nmax, int Voc);

int ltd_tree_accept_sampling(const float* logits, const float* draft_probs,
                             const int32_t* draft_tokens, const int32_t* parents,
                             const int32_t* n_nodes, const float* uniforms, int B, int Nmax,
                             int Voc, float temperature, int32_t* accepted_nodes,
                             int32_t* out_tokens, int32_t* n_accepted, void* workspace,
                             size_t workspace_bytes, int validate, int32_t* status, void* stream);

/*
 * KV compaction (the candidates after the first mismatch are discarded,
 * section 3.2, "Draft Tree Verification").
 *
 * For every sequence b, layer l < num_layers and kv head: logical row
 * P_b + accepted_nodes[b][j] moves to row P_b + j for j < n_accepted[b], all
 * reads before the writes they could overlap; then
 * new_prefix_len[b] = P_b + n_accepted[b].  Rows >= P_b + n_accepted[b] keep
 * whatever they held.  K and V of layer l start layer_stride_elems elements
 * after layer l-1; each layer has the attention call's layout.
 *
 *   k_cache, v_cache  device caches (modified in place).
 *   prefix_len        [B] int32 (read); new_prefix_len [B] int32 (written;
 *                     must not alias prefix_len).
 *   accepted_nodes    [B][Nmax], n_accepted [B]: as written by ltd_tree_accept.
 *   d * element size must be a multiple of 16 bytes.
 */
int ltd_kv_compact(void* k_cache, void* v_cache, const int32_t* block_table,
                   const int32_t* prefix_len, int32_t* new_prefix_len,
                   const int32_t* accepted_nodes, const int32_t* n_accepted, int B, int Nmax,
                   int Hkv, int d, int kv_rows, int max_blocks, int num_blocks, int num_layers,
                   int64_t layer_stride_elems, int dtype, int validate, int32_t* status,
                   void* stream);

/* Workgroups of the attention launch for a shape and cache layout
 * (kv_rows = capacity or block size, paged != 0 for a block table).  A bf16
 * call (head_dim 128 or 64) runs on the matrix-core kernels: a batch lays all
 * its (sequence, kv head, row tile) units' key tiles end to end and gives each
 * of that many workgroups (a power of two) an equal share; a single sequence
 * cuts each unit into KV splits.  Units cut between workgroups are merged by a
 * second kernel.  0 when the call runs on the fp32 vector kernel instead,
 * -1 on bad args.
 * Introspection for tests and benchmarks. */
int ltd_tree_verify_attn_grid(int B, int Nmax, int Hq, int Hkv, int d, int max_prefix, int dtype,
                              int kv_rows, int paged);

/*
 * Candidate token selection (section 3.2, "Candidate Token Selection"): of a
 * draft tree's candidate pool, keep the V = min(n_select[b], pool_size[b])
 * candidates with the highest cumulative path score and flatten them into a
 * tree in the form the verification calls take.
 *
 * Ranking: score descending; equal scores (-0.0 equals +0.0) rank the lower
 * pool index first.  Since the pool lists a parent before its children and a
 * child never scores above its parent, the kept candidates form a rooted
 * subtree.  They are flattened in pool order, so every parent precedes its
 * children (and a pool listed level by level comes out depth-major).
 *
 *   scores        [B][Vpool] float32: cumulative log-probability of each
 *                 candidate (any order-preserving image of its path
 *                 probability); never above its parent's, never NaN.
 *   pool_parents  [B][Vpool] int32: pool_parents[b][0] = -1 (the root) and
 *                 0 <= pool_parents[b][i] < i.
 *   pool_tokens   [B][Vpool] int32: the candidate tokens (copied, not read).
 *   pool_size     [B] int32 in [1, Vpool]; columns past it are never read.
 *   n_select      [B] int32 in [1, Nmax]: the verification size asked for
 *                 (the size policy's action).
 *   Vpool         1 <= Vpool <= LTD_MAX_POOL; 1 <= Nmax <= LTD_MAX_NODES.
 *   Outputs [B][Nmax] int32, rows k < V written, the rest untouched:
 *   selected      pool index of flattened node k (may be NULL);
 *   parents       parent of node k in the flattened order (-1 for the root);
 *                 the tree the verification calls take;
 *   tokens        token of node k (the verification's draft tokens);
 *   depth         depth of node k (the root is 0; may be NULL, which saves
 *                 the pass that computes it);
 *   n_nodes       [B] int32: V.
 * With validate != 0, malformed data is reported as LTD_STATUS_BAD_NNODES
 * (pool_size or n_select out of range), LTD_STATUS_BAD_PARENT or
 * LTD_STATUS_BAD_SCORE, and then nothing is written.  No workspace.
 */
int ltd_select_candidates(const float* scores, const int32_t* pool_parents,
                          const int32_t* pool_tokens, const int32_t* pool_size,
                          const int32_t* n_select, int B, int Vpool, int Nmax, int32_t* selected,
                          int32_t* parents, int32_t* tokens, int32_t* depth, int32_t* n_nodes,
                          int validate, int32_t* status, void* stream);

/*
 * One round of draft tree expansion (section 3.2, "Draft Tree Generation":
 * each leaf gets the W most probable tokens of its draft distribution as
 * children; the W children of highest cumulative path probability become the
 * next leaves).  The draft model's logits at the F frontier nodes are the
 * input; the children are appended to the candidate pool that
 * ltd_select_candidates and the policies read.
 *
 *   logits        [B][F][Voc] float32: draft logits at frontier node f.
 *   frontier      [B][F] int32: the frontier nodes' pool indices.
 *   scores, pool_parents, pool_tokens  [B][Vpool]: the pool, appended to.
 *   pool_size     [B] int32: read, then advanced by F*W.
 *   new_frontier  [B][W_next] int32: the next frontier (pool indices).
 * For frontier node f, in order, its children are the W tokens of largest
 * logit (equal logits: lower token index first), stored at pool_size + f*W
 * + r with parent frontier[f] and score = parent's score + log-softmax of the
 * logit (float32; the log-sum-exp is accumulated in double).  new_frontier
 * is the W_next new children of highest score, best first (equal scores:
 * lower pool index first).  A first round from the root has F = 1; after
 * D - 1 rounds of width W the pool holds 1 + W + (D-2) W^2 candidates.
 * Limits: 1 <= W <= LTD_EXPAND_MAX_W, W <= Voc <= 4096 * LTD_EXPAND_MAX_CHUNKS,
 * 1 <= F*W <= LTD_EXPAND_MAX_CHILDREN, 1 <= W_next <= F*W.
 * workspace: ltd_draft_expand_workspace_size(B, F, Voc, W) bytes.
 * With validate != 0: LTD_STATUS_BAD_NNODES if pool_size[b] < 1 or the
 * children would pass Vpool, LTD_STATUS_BAD_PARENT if a frontier index is
 * not in the pool; then nothing is written.
 */
size_t ltd_draft_expand_workspace_size(int B, int F, int Voc, int W);

int ltd_draft_expand(const float* logits, const int32_t* frontier, int B, int F, int Voc, int W,
                     int W_next, float* scores, int32_t* pool_parents, int32_t* pool_tokens,
                     int32_t* pool_size, int Vpool, int32_t* new_frontier, void* workspace,
                     size_t workspace_bytes, int validate, int32_t* status, void* stream);

/*
 * Draft-policy inference (section 4: the state vector of draft depth D,
 * context length L and candidate scores; appendix A.2: the size and depth
 * policies are fully connected ReLU networks with hidden widths [1024, 256]
 * and [1024], 12 and 2 actions, the action being the most likely one).
 *
 * The state of sequence b is built from its draft pool (no separate pass):
 *   LTD_POLICY_SIZE   [D_b, L_b, scores[b][0 .. min(n_b, F)), pad ...]
 *   LTD_POLICY_DEPTH  [pad ..., scores[b][n_b - F .. n_b), D_b, L_b]
 * with n_b = pool_size[b] and F = in_dim - 2 (the depth layout takes the last
 * F candidates, i.e. the newest expansion once the pool holds W^2 of them).
 * Then h1 = relu(w1 s + b1), optionally h2 = relu(w2 h1 + b2) (h2 > 0), and
 * logits = wo h + bo; action[b] = action_offset + action_scale * argmax
 * (lowest index on ties), so the size policy's V = 20 + 20 a can be written
 * straight into ltd_select_candidates' n_select.
 *
 *   scores [B][Vpool] float32, pool_size/depth/ctx_len [B] int32 (read).
 *   w1 [h1][in_dim], b1 [h1]; w2 [h2][h1], b2 [h2] (NULL when h2 = 0);
 *   wo [n_out][h2 or h1], bo [n_out]: float32, row-major (a row per unit).
 *   logits [B][n_out] float32, action [B] int32 (written).
 *   workspace: ltd_policy_workspace_size(B, h1, h2) bytes (hidden activations).
 * Limits: 3 <= in_dim <= LTD_POLICY_MAX_IN, 1 <= h1 <= LTD_POLICY_MAX_HIDDEN,
 * 0 <= h2 <= LTD_POLICY_MAX_HIDDEN, 1 <= n_out <= LTD_POLICY_MAX_OUT;
 * anything else, or a bad layout, is LTD_EINVAL.  Accumulation is float32 in
 * a fixed order (deterministic).
 */
size_t ltd_policy_workspace_size(int B, int h1, int h2);

int ltd_policy_forward(int layout, const float* scores, const int32_t* pool_size, int Vpool,
                       const int32_t* depth, const int32_t* ctx_len, float pad, int B, int in_dim,
                       const float* w1, const float* b1, int h1, const float* w2, const float* b2,
                       int h2, const float* wo, const float* bo, int n_out, int action_offset,
                       int action_scale, float* logits, int32_t* action, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Library version string. */
const char* ltd_version(void);

#ifdef __cplusplus
}
#endif
#endif /* LTD_VERIFY_H */
