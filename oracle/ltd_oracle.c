/*
 * CPU oracle for the tree-verification step of Learning-to-Draft speculative
 * decoding (arXiv 2603.01639).  TEST INFRASTRUCTURE ONLY: loaded by the test
 * suite, the smoke check and the benchmark's CPU-baseline leg, never by the
 * GPU library.  It shares no code with the HIP path.
 *
 * Every function here writes out the plain definition of the step it stands
 * for, in fp64, with no blocking, splitting, online softmax or fusion:
 *
 *   tree attention   paper section 3.2 ("Candidate Token Selection": the V
 *                    candidates are flattened into one sequence with a tree
 *                    attention mask; "Draft Tree Verification": one target pass
 *                    checks them all in parallel).  The mask lets a candidate
 *                    see the context prefix and its own ancestors only, so a
 *                    node's output is ordinary attention of its query over
 *                    prefix + root path.
 *   acceptance       paper section 3.2 ("Draft Tree Verification"): tokens are
 *                    accepted up to the first mismatch with the target's own
 *                    prediction; the target's prediction at the first error
 *                    (the bonus token) is appended.
 *   compaction       the rejected candidates are discarded (same paragraph);
 *                    the accepted rows are moved next to the prefix.
 *   selection        paper section 3.2 ("Candidate Token Selection"): of the
 *                    draft tree's candidates, the V with the highest predicted
 *                    (cumulative path) probability are kept and flattened.
 *   sampling         acceptance at temperature T > 0, the paper's second
 *                    setting (its experiments report T = 0 and T = 1; the rule
 *                    is the one its baseline inherits, not printed in the
 *                    paper): recursive rejection sampling over each node's
 *                    children, which were drawn without replacement from the
 *                    draft distribution.
 *   expansion        paper section 3.2 ("Draft Tree Generation"): each leaf
 *                    of the current level gets the W most probable tokens of
 *                    its draft distribution as children; of all children, the
 *                    W with the highest cumulative path probability become
 *                    the next leaves.
 *
 * Readings of points the paper leaves open (softmax scale, node order, whether
 * V counts the root, tie rules, where tree K/V live) are fixed by the caller's
 * arguments or stated at the function that applies them.
 */
#include "ltd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int ltd_oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads for the next parallel regions (n >= 1); no effect without OpenMP. */
void ltd_oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* bf16 is the top half of an IEEE binary32; widening is exact. */
static double bf16_bits_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

static double load_elem(const void* base, int64_t idx, int dtype) {
  if (dtype == LTDO_DTYPE_F32) return (double)((const float*)base)[idx];
  return bf16_bits_to_double(((const uint16_t*)base)[idx]);
}

/* Element offset of cache row `row` (logical position in sequence b), kv head
 * g.  Contiguous: [B][Hkv][cap][d].  Paged: [num_blocks][Hkv][block_size][d]
 * with the physical block taken from block_table[b][row / block_size]. */
static int64_t cache_row_offset(const int32_t* block_table, int b, int g, int row, int Hkv,
                                int d, int kv_rows, int max_blocks) {
  if (block_table == NULL) {
    return (((int64_t)b * Hkv + g) * kv_rows + row) * (int64_t)d;
  }
  int64_t blk = block_table[(int64_t)b * max_blocks + row / kv_rows];
  return ((blk * Hkv + g) * kv_rows + row % kv_rows) * (int64_t)d;
}

/* Checks shared by attention: tree shape, prefix bounds and block ids.
 * Returns 0 or an LTDO_STATUS_* code. */
static int check_tree_and_cache(const int32_t* block_table, const int32_t* prefix_len,
                                const int32_t* parents, const int32_t* n_nodes, int B, int Nmax,
                                int kv_rows, int max_blocks, int num_blocks) {
  for (int b = 0; b < B; ++b) {
    int n = n_nodes[b];
    if (n < 1 || n > Nmax) return LTDO_STATUS_BAD_NNODES;
    const int32_t* par = parents + (int64_t)b * Nmax;
    if (par[0] != -1) return LTDO_STATUS_BAD_PARENT;
    for (int i = 1; i < n; ++i)
      if (par[i] < 0 || par[i] >= i) return LTDO_STATUS_BAD_PARENT;
    int P = prefix_len[b];
    int64_t capacity = block_table ? (int64_t)kv_rows * max_blocks : kv_rows;
    if (P < 0 || (int64_t)P + n > capacity) return LTDO_STATUS_BAD_PREFIX;
    if (block_table) {
      int used = (P + n + kv_rows - 1) / kv_rows;
      for (int j = 0; j < used; ++j) {
        int32_t blk = block_table[(int64_t)b * max_blocks + j];
        if (blk < 0 || blk >= num_blocks) return LTDO_STATUS_BAD_BLOCK;
      }
    }
  }
  return 0;
}

int ltd_oracle_tree_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* block_table, const int32_t* prefix_len,
                                const int32_t* parents, const int32_t* n_nodes,
                                const uint8_t* node_mask, double* out, int B, int Nmax, int Hq,
                                int Hkv, int d, int kv_rows, int max_blocks, int num_blocks,
                                double scale, int dtype) {
  if (!q || !k_cache || !v_cache || !prefix_len || !parents || !n_nodes || !out)
    return LTDO_EINVAL;
  if (B < 0 || Nmax < 1 || Hq < 1 || Hkv < 1 || d < 1 || kv_rows < 1 || Hq % Hkv != 0)
    return LTDO_EINVAL;
  if (block_table && (max_blocks < 1 || num_blocks < 1)) return LTDO_EINVAL;
  if (dtype != LTDO_DTYPE_F32 && dtype != LTDO_DTYPE_BF16) return LTDO_EUNSUPPORTED;
  int st = check_tree_and_cache(block_table, prefix_len, parents, n_nodes, B, Nmax, kv_rows,
                                max_blocks, num_blocks);
  if (st) return st;

  const int group = Hq / Hkv; /* GQA: q head h reads kv head h / group */
  int failed = 0;

#pragma omp parallel
  {
    /* Per-thread scratch: the node's root path and one score per visible key. */
    int max_keys = 0;
    for (int b = 0; b < B; ++b)
      if (prefix_len[b] + n_nodes[b] > max_keys) max_keys = prefix_len[b] + n_nodes[b];
    int* path = (int*)malloc(sizeof(int) * (size_t)Nmax);
    int* key_rows = (int*)malloc(sizeof(int) * (size_t)(max_keys > 0 ? max_keys : 1));
    double* score = (double*)malloc(sizeof(double) * (size_t)(max_keys > 0 ? max_keys : 1));
    double* acc = (double*)malloc(sizeof(double) * (size_t)d);
    if (!path || !key_rows || !score || !acc) {
#pragma omp atomic write
      failed = 1;
    }

#pragma omp for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b) {
      for (int i = 0; i < Nmax; ++i) {
        if (failed || i >= n_nodes[b]) continue;
        if (node_mask && !node_mask[(int64_t)b * Nmax + i]) continue;
        const int P = prefix_len[b];
        const int32_t* par = parents + (int64_t)b * Nmax;

        /* Visible keys of node i: every prefix row, then the tree rows of its
         * ancestors (the root path, walked from i up to the root). */
        int n_keys = 0;
        for (int t = 0; t < P; ++t) key_rows[n_keys++] = t;
        int path_len = 0;
        for (int j = i; j != -1; j = par[j]) path[path_len++] = j;
        for (int a = 0; a < path_len; ++a) key_rows[n_keys++] = P + path[a];

        for (int h = 0; h < Hq; ++h) {
          const int g = h / group;
          const int64_t q_off = (((int64_t)b * Nmax + i) * Hq + h) * d;

          /* s_t = scale * <q, k_t> for every visible key t */
          double m = -INFINITY;
          for (int t = 0; t < n_keys; ++t) {
            int64_t k_off = cache_row_offset(block_table, b, g, key_rows[t], Hkv, d, kv_rows,
                                             max_blocks);
            double dot = 0.0;
            for (int e = 0; e < d; ++e)
              dot += load_elem(q, q_off + e, dtype) * load_elem(k_cache, k_off + e, dtype);
            score[t] = scale * dot;
            if (score[t] > m) m = score[t];
          }

          /* softmax weights exp(s_t - max) and the weighted sum of V rows */
          double denom = 0.0;
          for (int e = 0; e < d; ++e) acc[e] = 0.0;
          for (int t = 0; t < n_keys; ++t) {
            double w = exp(score[t] - m);
            denom += w;
            int64_t v_off = cache_row_offset(block_table, b, g, key_rows[t], Hkv, d, kv_rows,
                                             max_blocks);
            for (int e = 0; e < d; ++e) acc[e] += w * load_elem(v_cache, v_off + e, dtype);
          }
          double* o = out + q_off;
          for (int e = 0; e < d; ++e) o[e] = acc[e] / denom;
        }
      }
    }
    free(path);
    free(key_rows);
    free(score);
    free(acc);
  }
  return failed ? LTDO_EINVAL : 0;
}

/* argmax over one node's logits; ties go to the lowest vocabulary index.
 * Plain IEEE comparison, so -0.0 and +0.0 compare equal.  NaN is outside the
 * contract. */
static int32_t argmax_row(const float* row, int Voc) {
  int32_t best = 0;
  float best_val = row[0];
  for (int v = 1; v < Voc; ++v) {
    if (row[v] > best_val) {
      best_val = row[v];
      best = v;
    }
  }
  return best;
}

int ltd_oracle_tree_accept(const float* logits, const int32_t* draft_tokens,
                           const int32_t* parents, const int32_t* n_nodes, int B, int Nmax,
                           int Voc, int32_t* pred, int32_t* accepted_nodes,
                           int32_t* out_tokens, int32_t* n_accepted) {
  if (!logits || !draft_tokens || !parents || !n_nodes || !pred || !accepted_nodes ||
      !out_tokens || !n_accepted)
    return LTDO_EINVAL;
  if (B < 0 || Nmax < 1 || Voc < 1) return LTDO_EINVAL;
  for (int b = 0; b < B; ++b) {
    int n = n_nodes[b];
    if (n < 1 || n > Nmax) return LTDO_STATUS_BAD_NNODES;
    const int32_t* par = parents + (int64_t)b * Nmax;
    if (par[0] != -1) return LTDO_STATUS_BAD_PARENT;
    for (int i = 1; i < n; ++i)
      if (par[i] < 0 || par[i] >= i) return LTDO_STATUS_BAD_PARENT;
  }

  /* 1. The target's own prediction at every node. */
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < Nmax; ++i)
      if (i < n_nodes[b])
        pred[(int64_t)b * Nmax + i] = argmax_row(logits + ((int64_t)b * Nmax + i) * Voc, Voc);

  for (int b = 0; b < B; ++b) {
    const int n = n_nodes[b];
    const int32_t* par = parents + (int64_t)b * Nmax;
    const int32_t* tok = draft_tokens + (int64_t)b * Nmax;
    const int32_t* pr = pred + (int64_t)b * Nmax;
    char* ok = (char*)malloc((size_t)n);
    int* depth = (int*)malloc(sizeof(int) * (size_t)n);
    if (!ok || !depth) {
      free(ok);
      free(depth);
      return LTDO_EINVAL;
    }

    /* 2-3. A draft token is accepted when it equals the target's prediction at
     * its parent and its parent was accepted; the root (the previous cycle's
     * bonus token) is always accepted.  parent < child, so index order visits
     * parents first. */
    ok[0] = 1;
    depth[0] = 0;
    for (int c = 1; c < n; ++c) {
      ok[c] = ok[par[c]] && (tok[c] == pr[par[c]]);
      depth[c] = depth[par[c]] + 1;
    }

    /* 4. The accepted leaf is the deepest accepted node (the longest accepted
     * root path); among equally deep ones, the smallest node index. */
    int leaf = 0;
    for (int c = 1; c < n; ++c)
      if (ok[c] && depth[c] > depth[leaf]) leaf = c;

    /* 5. The path is the leaf's ancestors, root first. */
    int len = depth[leaf] + 1;
    int32_t* path = accepted_nodes + (int64_t)b * Nmax;
    for (int j = leaf, k = len - 1; j != -1; j = par[j], --k) path[k] = j;

    /* 6. Emitted tokens: the accepted drafts after the root, then the bonus
     * (the target's prediction at the leaf).  Their count is the acceptance
     * length L_A, equal to the path length. */
    int32_t* ot = out_tokens + (int64_t)b * Nmax;
    for (int k = 1; k < len; ++k) ot[k - 1] = tok[path[k]];
    ot[len - 1] = pr[leaf];
    n_accepted[b] = len;

    free(ok);
    free(depth);
  }
  return 0;
}

int ltd_oracle_kv_compact(void* k_cache, void* v_cache, const int32_t* block_table,
                          const int32_t* prefix_len, int32_t* new_prefix_len,
                          const int32_t* accepted_nodes, const int32_t* n_accepted, int B,
                          int Nmax, int Hkv, int d, int kv_rows, int max_blocks, int num_blocks,
                          int num_layers, int64_t layer_stride_elems, int elem_bytes) {
  if (!k_cache || !v_cache || !prefix_len || !new_prefix_len || !accepted_nodes || !n_accepted)
    return LTDO_EINVAL;
  if (new_prefix_len == prefix_len) return LTDO_EINVAL;
  if (B < 0 || Nmax < 1 || Hkv < 1 || d < 1 || kv_rows < 1 || num_layers < 1) return LTDO_EINVAL;
  if (elem_bytes != 2 && elem_bytes != 4) return LTDO_EUNSUPPORTED;
  if (block_table && (max_blocks < 1 || num_blocks < 1)) return LTDO_EINVAL;

  int64_t capacity = block_table ? (int64_t)kv_rows * max_blocks : kv_rows;
  for (int b = 0; b < B; ++b) {
    int n = n_accepted[b];
    const int32_t* path = accepted_nodes + (int64_t)b * Nmax;
    if (n < 1 || n > Nmax) return LTDO_STATUS_BAD_PATH;
    if (path[0] != 0) return LTDO_STATUS_BAD_PATH;
    for (int j = 1; j < n; ++j)
      if (path[j] <= path[j - 1]) return LTDO_STATUS_BAD_PATH;
    int P = prefix_len[b];
    if (P < 0 || (int64_t)P + path[n - 1] >= capacity) return LTDO_STATUS_BAD_PREFIX;
    if (block_table) {
      int used = (P + path[n - 1] + kv_rows) / kv_rows;
      for (int j = 0; j < used; ++j) {
        int32_t blk = block_table[(int64_t)b * max_blocks + j];
        if (blk < 0 || blk >= num_blocks) return LTDO_STATUS_BAD_BLOCK;
      }
    }
  }

  const size_t row_bytes = (size_t)d * (size_t)elem_bytes;
  unsigned char* tmp = (unsigned char*)malloc(row_bytes * (size_t)Nmax);
  if (!tmp) return LTDO_EINVAL;
  for (int b = 0; b < B; ++b) {
    const int P = prefix_len[b];
    const int n = n_accepted[b];
    const int32_t* path = accepted_nodes + (int64_t)b * Nmax;
    for (int layer = 0; layer < num_layers; ++layer) {
      for (int which = 0; which < 2; ++which) {
        unsigned char* base = (unsigned char*)(which == 0 ? k_cache : v_cache) +
                              (size_t)(layer * layer_stride_elems) * (size_t)elem_bytes;
        for (int g = 0; g < Hkv; ++g) {
          /* Read every accepted row first, then write them back in path
           * order, so a destination that is also a later source is safe. */
          for (int j = 0; j < n; ++j) {
            int64_t off = cache_row_offset(block_table, b, g, P + path[j], Hkv, d, kv_rows,
                                           max_blocks);
            memcpy(tmp + (size_t)j * row_bytes, base + (size_t)off * (size_t)elem_bytes,
                   row_bytes);
          }
          for (int j = 0; j < n; ++j) {
            int64_t off = cache_row_offset(block_table, b, g, P + j, Hkv, d, kv_rows, max_blocks);
            memcpy(base + (size_t)off * (size_t)elem_bytes, tmp + (size_t)j * row_bytes,
                   row_bytes);
          }
        }
      }
    }
    new_prefix_len[b] = P + n;
  }
  free(tmp);
  return 0;
}

/* ---- candidate token selection (section 3.2, "Candidate Token Selection").
 * The paper keeps the V candidates of the draft tree with the highest overall
 * (cumulative path) probability.  Readings of what it leaves open: equal
 * scores are ranked by pool index, lower first (the pool lists a parent before
 * its children and a child never scores above its parent, so a parent always
 * ranks before its children and the kept set is a rooted subtree); the kept
 * candidates are flattened in pool order, which puts every parent before its
 * children (and, for a pool listed level by level, is depth-major). */
typedef struct {
  float score;
  int index;
} cand_t;

static int by_rank(const void* pa, const void* pb) {
  const cand_t* a = (const cand_t*)pa;
  const cand_t* b = (const cand_t*)pb;
  if (a->score != b->score) return a->score > b->score ? -1 : 1;
  return (a->index > b->index) - (a->index < b->index);
}

static int by_pool_order(const void* pa, const void* pb) {
  const cand_t* a = (const cand_t*)pa;
  const cand_t* b = (const cand_t*)pb;
  return (a->index > b->index) - (a->index < b->index);
}

int ltd_oracle_select_candidates(const float* scores, const int32_t* pool_parents,
                                 const int32_t* pool_tokens, const int32_t* pool_size,
                                 const int32_t* n_select, int B, int Vpool, int Nmax,
                                 int32_t* selected, int32_t* parents, int32_t* tokens,
                                 int32_t* depth, int32_t* n_nodes) {
  if (B < 0 || Vpool < 1 || Nmax < 1) return LTDO_EINVAL;
  /* data checks first, for every sequence, so nothing is written on failure */
  for (int b = 0; b < B; ++b) {
    const int pn = pool_size[b];
    if (pn < 1 || pn > Vpool || n_select[b] < 1 || n_select[b] > Nmax)
      return LTDO_STATUS_BAD_NNODES;
    const int32_t* par = pool_parents + (int64_t)b * Vpool;
    const float* sc = scores + (int64_t)b * Vpool;
    if (par[0] != -1) return LTDO_STATUS_BAD_PARENT;
    for (int i = 1; i < pn; ++i)
      if (par[i] < 0 || par[i] >= i) return LTDO_STATUS_BAD_PARENT;
    for (int i = 0; i < pn; ++i) {
      if (isnan(sc[i])) return LTDO_STATUS_BAD_SCORE;
      if (i > 0 && sc[i] > sc[par[i]]) return LTDO_STATUS_BAD_SCORE;
    }
  }
  cand_t* c = (cand_t*)malloc(sizeof(cand_t) * (size_t)Vpool);
  int* dep = (int*)malloc(sizeof(int) * (size_t)Vpool);
  int* new_id = (int*)malloc(sizeof(int) * (size_t)Vpool);
  if (!c || !dep || !new_id) {
    free(c);
    free(dep);
    free(new_id);
    return LTDO_EINVAL;
  }
  for (int b = 0; b < B; ++b) {
    const int pn = pool_size[b];
    const int32_t* par = pool_parents + (int64_t)b * Vpool;
    const float* sc = scores + (int64_t)b * Vpool;
    /* depth: the root is 0, a child one more than its parent (parents come
     * first in the pool) */
    for (int i = 0; i < pn; ++i) dep[i] = i == 0 ? 0 : dep[par[i]] + 1;
    for (int i = 0; i < pn; ++i) {
      c[i].score = sc[i];
      c[i].index = i;
    }
    /* the V candidates ranked first */
    qsort(c, (size_t)pn, sizeof(cand_t), by_rank);
    const int V = n_select[b] < pn ? n_select[b] : pn;
    /* flattened in pool order */
    qsort(c, (size_t)V, sizeof(cand_t), by_pool_order);
    for (int i = 0; i < pn; ++i) new_id[i] = -1;
    for (int k = 0; k < V; ++k) new_id[c[k].index] = k;
    const int64_t o = (int64_t)b * Nmax;
    for (int k = 0; k < V; ++k) {
      const int j = c[k].index;
      selected[o + k] = j;
      parents[o + k] = j == 0 ? -1 : new_id[par[j]];
      tokens[o + k] = pool_tokens[(int64_t)b * Vpool + j];
      depth[o + k] = dep[j];
    }
    n_nodes[b] = V;
  }
  free(c);
  free(dep);
  free(new_id);
  return 0;
}

/* ---- one round of draft tree expansion (section 3.2, "Draft Tree
 * Generation").  For frontier node f of sequence b, with draft logits l over
 * the vocabulary: log p(v) = l_v - log(sum_u exp(l_u)) (in double); its W
 * children are the W tokens of largest logit (equal logits: lower token
 * index first), in that order, and a child's score is its parent's score plus
 * log p(token), stored as float.  Children are appended to the pool frontier
 * by frontier; then the W_next children of highest stored score (equal
 * scores: lower pool index first) become the next frontier, in that order. */
int ltd_oracle_draft_expand(const float* logits, const int32_t* frontier, int B, int F, int Voc,
                            int W, int W_next, float* scores, int32_t* pool_parents,
                            int32_t* pool_tokens, int32_t* pool_size, int Vpool,
                            int32_t* new_frontier) {
  if (B < 0 || F < 1 || Voc < 1 || W < 1 || W > Voc || W_next < 1 || W_next > F * W || Vpool < 1)
    return LTDO_EINVAL;
  for (int b = 0; b < B; ++b) {
    if (pool_size[b] < 1 || pool_size[b] + F * W > Vpool) return LTDO_STATUS_BAD_NNODES;
    for (int f = 0; f < F; ++f)
      if (frontier[(int64_t)b * F + f] < 0 || frontier[(int64_t)b * F + f] >= pool_size[b])
        return LTDO_STATUS_BAD_PARENT;
  }
  const size_t n_taken = (size_t)(F * W > Voc ? F * W : Voc);
  unsigned char* taken = (unsigned char*)malloc(n_taken);
  if (!taken) return LTDO_EINVAL;
  for (int b = 0; b < B; ++b) {
    const int64_t pb = (int64_t)b * Vpool;
    const int first = pool_size[b];
    for (int f = 0; f < F; ++f) {
      const float* row = logits + ((int64_t)b * F + f) * Voc;
      const int parent = frontier[(int64_t)b * F + f];
      double m = -INFINITY;
      for (int v = 0; v < Voc; ++v)
        if (row[v] > m) m = row[v];
      double z = 0.0;
      for (int v = 0; v < Voc; ++v) z += exp((double)row[v] - m);
      const double lse = m + log(z);
      memset(taken, 0, (size_t)Voc);
      for (int r = 0; r < W; ++r) {
        /* the largest logit not taken yet, lowest index on ties */
        int best = -1;
        for (int v = 0; v < Voc; ++v)
          if (!taken[v] && (best < 0 || row[v] > row[best])) best = v;
        taken[best] = 1;
        const int c = first + f * W + r;
        pool_parents[pb + c] = parent;
        pool_tokens[pb + c] = best;
        scores[pb + c] = (float)((double)scores[pb + parent] + ((double)row[best] - lse));
      }
    }
    /* beam: the W_next children of highest score */
    const int n_children = F * W;
    memset(taken, 0, n_taken);
    for (int r = 0; r < W_next; ++r) {
      int best = -1;
      for (int c = 0; c < n_children; ++c)
        if (!taken[c] && (best < 0 || scores[pb + first + c] > scores[pb + first + best])) best = c;
      taken[best] = 1;
      new_frontier[(int64_t)b * W_next + r] = first + best;
    }
    pool_size[b] = first + n_children;
  }
  free(taken);
  return 0;
}

/* ---- acceptance by recursive rejection sampling at temperature T > 0.
 * Written as the literal recursion over explicit distributions, in double.
 * At node u the target distribution is P = softmax(logits[u] / T) and the
 * draft distribution Q = draft_probs[u] / sum(draft_probs[u]).  Children are
 * tried in ascending node index (the order they were drawn).  Child c with
 * token x is accepted when uniforms[c][0] * Q(x) < P(x) (probability
 * min(1, P(x)/Q(x))); the walk then continues at c.  On rejection, P becomes
 * max(P - Q, 0) renormalised (unchanged if that has no mass) and Q loses x
 * and is renormalised.  When no child is accepted (or u is a leaf) the bonus
 * token is drawn from the current P by inverse CDF at uniforms[u][1]: the
 * smallest v whose cumulative mass exceeds uniforms[u][1] * sum(P) (the last
 * v with mass if rounding leaves none).  Optional outputs: final_dist [B][Voc]
 * (the distribution the bonus was drawn from) and min_margin [B] (the
 * smallest |r Q(x) - P(x)| / max(P(x), r Q(x)) over the accept tests taken). */
int ltd_oracle_tree_accept_sampling(const float* logits, const float* draft_probs,
                                    const int32_t* draft_tokens, const int32_t* parents,
                                    const int32_t* n_nodes, const float* uniforms, int B, int Nmax,
                                    int Voc, double temperature, int32_t* accepted_nodes,
                                    int32_t* out_tokens, int32_t* n_accepted, double* final_dist,
                                    double* min_margin) {
  if (B < 0 || Nmax < 1 || Voc < 1 || !(temperature > 0.0)) return LTDO_EINVAL;
  for (int b = 0; b < B; ++b) {
    const int n = n_nodes[b];
    if (n < 1 || n > Nmax) return LTDO_STATUS_BAD_NNODES;
    const int32_t* par = parents + (int64_t)b * Nmax;
    if (par[0] != -1) return LTDO_STATUS_BAD_PARENT;
    for (int i = 1; i < n; ++i)
      if (par[i] < 0 || par[i] >= i) return LTDO_STATUS_BAD_PARENT;
  }
  double* P = (double*)malloc(sizeof(double) * (size_t)Voc);
  double* Q = (double*)malloc(sizeof(double) * (size_t)Voc);
  if (!P || !Q) {
    free(P);
    free(Q);
    return LTDO_EINVAL;
  }
  for (int b = 0; b < B; ++b) {
    const int n = n_nodes[b];
    const int32_t* par = parents + (int64_t)b * Nmax;
    const int32_t* tok = draft_tokens + (int64_t)b * Nmax;
    const float* ur = uniforms + (int64_t)b * Nmax * 2;
    int32_t* path = accepted_nodes + (int64_t)b * Nmax;
    int32_t* ot = out_tokens + (int64_t)b * Nmax;
    double margin = INFINITY;
    int len = 0;
    int u = 0;
    path[len++] = 0;
    for (;;) {
      const float* lu = logits + ((int64_t)b * Nmax + u) * Voc;
      double m = -INFINITY;
      for (int v = 0; v < Voc; ++v)
        if (lu[v] > m) m = lu[v];
      double z = 0.0;
      for (int v = 0; v < Voc; ++v) {
        P[v] = exp(((double)lu[v] - m) / temperature);
        z += P[v];
      }
      for (int v = 0; v < Voc; ++v) P[v] /= z;
      int has_child = 0;
      for (int c = u + 1; c < n; ++c)
        if (par[c] == u) has_child = 1;
      if (has_child) {
        const float* qu = draft_probs + ((int64_t)b * Nmax + u) * Voc;
        double qs = 0.0;
        for (int v = 0; v < Voc; ++v) qs += qu[v];
        for (int v = 0; v < Voc; ++v) Q[v] = qu[v] / qs;
      }
      int next = -1;
      for (int c = u + 1; c < n && next < 0; ++c) {
        if (par[c] != u) continue;
        const int x = tok[c];
        const double r = ur[2 * c];
        const double lhs = r * Q[x];
        const double den = lhs > P[x] ? lhs : P[x];
        if (den > 0) {
          const double mg = fabs(lhs - P[x]) / den;
          if (mg < margin) margin = mg;
        }
        if (lhs < P[x]) {
          next = c;
          break;
        }
        /* rejected: residual target, draft without x */
        double s = 0.0;
        for (int v = 0; v < Voc; ++v) s += P[v] > Q[v] ? P[v] - Q[v] : 0.0;
        if (s > 0.0)
          for (int v = 0; v < Voc; ++v) P[v] = (P[v] > Q[v] ? P[v] - Q[v] : 0.0) / s;
        Q[x] = 0.0;
        double qs = 0.0;
        for (int v = 0; v < Voc; ++v) qs += Q[v];
        if (qs > 0.0)
          for (int v = 0; v < Voc; ++v) Q[v] /= qs;
      }
      if (next >= 0) {
        path[len++] = next;
        u = next;
        continue;
      }
      /* bonus token from P by inverse CDF */
      double total = 0.0;
      for (int v = 0; v < Voc; ++v) total += P[v];
      const double target = (double)ur[2 * u + 1] * total;
      int bonus = -1, last = 0;
      double cum = 0.0;
      for (int v = 0; v < Voc; ++v) {
        if (P[v] > 0.0) last = v;
        cum += P[v];
        if (cum > target && P[v] > 0.0) {
          bonus = v;
          break;
        }
      }
      if (bonus < 0) bonus = last;
      for (int j = 1; j < len; ++j) ot[j - 1] = tok[path[j]];
      ot[len - 1] = bonus;
      if (final_dist)
        for (int v = 0; v < Voc; ++v) final_dist[(int64_t)b * Voc + v] = P[v];
      break;
    }
    n_accepted[b] = len;
    if (min_margin) min_margin[b] = margin;
  }
  free(P);
  free(Q);
  return 0;
}
