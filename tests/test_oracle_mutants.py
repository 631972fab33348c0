"""The oracle's pins are sensitive: plant plausible mistakes in a copy of the
oracle's C source, build each mutant on the CPU, and check that at least one
pin fails for every mutant.  (Mistakes are planted in the oracle only.)"""
import os
import subprocess

import numpy as np
import pytest

import oracle
import test_oracle_accept as TA
import test_oracle_attention as TT
import test_oracle_compact as TC
import test_oracle_select as TS
import test_oracle_expand as TE
import test_oracle_sampling as TSa

SRC = os.path.join(os.path.dirname(oracle.__file__), "ltd_oracle.c")

ATTN_PINS = [
    lambda: TT.test_every_tree_up_to_6_nodes_matches_root_path_attention(4),
    lambda: TT.test_random_trees_up_to_32_nodes(1),
    lambda: TT.test_matches_library_sdpa_with_closure_mask(2),
    lambda: TT.test_single_node_is_decode_attention(),
    lambda: TT.test_paged_layout_equals_contiguous(),
]
ACCEPT_PINS = [
    lambda: TA.test_worked_examples(),
    lambda: TA.test_exhaustive_small_trees_all_patterns(5),
    lambda: TA.test_argmax_ties_and_signed_zero_match_numpy(),
    lambda: TA.test_greedy_equivalence_on_toy_lm(0),
]
COMPACT_PINS = [
    lambda: TC.test_contiguous_matches_explicit_gather([0, 1, 3, 6]),
    lambda: TC.test_contiguous_matches_explicit_gather([0, 4, 5, 9, 11]),
    lambda: TC.test_attention_after_compaction_equals_attention_over_path(),
    lambda: TC.test_paged_multilayer_bf16_moves_the_same_rows(),
]
SELECT_PINS = [
    lambda: TS.test_worked_examples(),
    lambda: TS.test_exhaustive_small_pools(4),
    lambda: TS.test_matches_the_generators_own_selection(6, 10, 60),
    lambda: TS.test_star_pool_is_a_stable_argsort(),
    lambda: TS.test_validation_codes(),
]

EXPAND_PINS = [
    lambda: TE.test_replays_the_generators_beam(4, 4, 50),
    lambda: TE.test_matches_torch_log_softmax_topk(),
    lambda: TE.test_ties(),
]

SAMPLING_PINS = [
    lambda: TSa.test_worked_examples(),
    lambda: TSa.test_losslessness_on_a_toy_model(),
    lambda: TSa.test_draft_equal_to_target_accepts_the_first_child(),
    lambda: TSa.test_lone_root_is_inverse_cdf_sampling(),
]

# (name, original text, mutated text, pins expected to notice)
MUTANTS = [
    ("tree part dropped (node sees only itself)",
     "for (int a = 0; a < path_len; ++a) key_rows", "for (int a = 0; a < 1; ++a) key_rows", ATTN_PINS),
    ("mask uses parent instead of ancestors",
     "for (int a = 0; a < path_len; ++a) key_rows",
     "for (int a = 0; a < (path_len < 2 ? path_len : 2); ++a) key_rows", ATTN_PINS),
    ("last prefix row dropped", "for (int t = 0; t < P; ++t) key_rows",
     "for (int t = 0; t + 1 < P; ++t) key_rows", ATTN_PINS),
    ("GQA head mapping interleaved", "const int g = h / group;", "const int g = h % Hkv;", ATTN_PINS),
    ("scale ignored", "score[t] = scale * dot;", "score[t] = dot;", ATTN_PINS),
    ("V read at the wrong row", "int64_t v_off = cache_row_offset(block_table, b, g, key_rows[t],",
     "int64_t v_off = cache_row_offset(block_table, b, g, key_rows[t] ? key_rows[t] - 1 : 0,",
     ATTN_PINS),
    ("paged offset ignores the block table",
     "int64_t blk = block_table[(int64_t)b * max_blocks + row / kv_rows];",
     "int64_t blk = b * max_blocks + row / kv_rows;", ATTN_PINS),
    ("parent acceptance not required", "ok[c] = ok[par[c]] && (tok[c] == pr[par[c]]);",
     "ok[c] = (tok[c] == pr[par[c]]);", ACCEPT_PINS),
    ("token compared with own prediction", "ok[c] = ok[par[c]] && (tok[c] == pr[par[c]]);",
     "ok[c] = ok[par[c]] && (tok[c] == pr[c]);", ACCEPT_PINS),
    ("argmax ties go to the last index", "if (row[v] > best_val) {", "if (row[v] >= best_val) {",
     ACCEPT_PINS),
    ("leaf ties go to the largest index", "if (ok[c] && depth[c] > depth[leaf]) leaf = c;",
     "if (ok[c] && depth[c] >= depth[leaf]) leaf = c;", ACCEPT_PINS),
    ("bonus taken at the parent", "ot[len - 1] = pr[leaf];",
     "ot[len - 1] = pr[leaf ? par[leaf] : 0];", ACCEPT_PINS),
    ("compaction copies row by row in reverse order without staging",
     "for (int j = 0; j < n; ++j) {\n"
     "            int64_t off = cache_row_offset(block_table, b, g, P + path[j], Hkv, d, kv_rows,\n"
     "                                           max_blocks);\n"
     "            memcpy(tmp + (size_t)j * row_bytes, base + (size_t)off * (size_t)elem_bytes,\n"
     "                   row_bytes);",
     "for (int j = n - 1; j >= 0; --j) {\n"
     "            int64_t off = cache_row_offset(block_table, b, g, P + path[j], Hkv, d, kv_rows,\n"
     "                                           max_blocks);\n"
     "            memcpy(tmp + (size_t)j * row_bytes, base + (size_t)off * (size_t)elem_bytes,\n"
     "                   row_bytes);\n"
     "            int64_t dst = cache_row_offset(block_table, b, g, P + j, Hkv, d, kv_rows, max_blocks);\n"
     "            memcpy(base + (size_t)dst * (size_t)elem_bytes, tmp + (size_t)j * row_bytes, row_bytes);",
     COMPACT_PINS),
    ("compaction shifts by one row", "int64_t off = cache_row_offset(block_table, b, g, P + j, Hkv",
     "int64_t off = cache_row_offset(block_table, b, g, P + j + 1, Hkv", COMPACT_PINS),
    ("selection ties go to the higher index",
     "if (a->score != b->score) return a->score > b->score ? -1 : 1;\n"
     "  return (a->index > b->index) - (a->index < b->index);",
     "if (a->score != b->score) return a->score > b->score ? -1 : 1;\n"
     "  return (a->index < b->index) - (a->index > b->index);", SELECT_PINS),
    ("selection keeps the lowest scores",
     "if (a->score != b->score) return a->score > b->score ? -1 : 1;\n  return (a->index",
     "if (a->score != b->score) return a->score < b->score ? -1 : 1;\n  return (a->index",
     SELECT_PINS),
    ("flattened in rank order", "qsort(c, (size_t)V, sizeof(cand_t), by_pool_order);",
     "(void)by_pool_order;", SELECT_PINS),
    ("flattened in reverse pool order",
     "static int by_pool_order(const void* pa, const void* pb) {\n"
     "  const cand_t* a = (const cand_t*)pa;\n  const cand_t* b = (const cand_t*)pb;\n"
     "  return (a->index > b->index) - (a->index < b->index);",
     "static int by_pool_order(const void* pa, const void* pb) {\n"
     "  const cand_t* a = (const cand_t*)pa;\n  const cand_t* b = (const cand_t*)pb;\n"
     "  return (a->index < b->index) - (a->index > b->index);", SELECT_PINS),
    ("parents left as pool indices", "parents[o + k] = j == 0 ? -1 : new_id[par[j]];",
     "parents[o + k] = j == 0 ? -1 : par[j];", SELECT_PINS),
    ("one candidate too few", "const int V = n_select[b] < pn ? n_select[b] : pn;",
     "const int V = n_select[b] <= pn ? n_select[b] - (n_select[b] > 1) : pn;", SELECT_PINS),
    ("depth not incremented", "dep[i] = i == 0 ? 0 : dep[par[i]] + 1;",
     "dep[i] = i == 0 ? 0 : dep[par[i]];", SELECT_PINS),
    ("sampling: residual not renormalised",
     "for (int v = 0; v < Voc; ++v) P[v] = (P[v] > Q[v] ? P[v] - Q[v] : 0.0) / s;",
     "for (int v = 0; v < Voc; ++v) P[v] = (P[v] > Q[v] ? P[v] - Q[v] : 0.0);", SAMPLING_PINS),
    ("sampling: draft keeps a rejected token", "        Q[x] = 0.0;\n", "\n", SAMPLING_PINS),
    ("sampling: acceptance test inverted", "        if (lhs < P[x]) {", "        if (lhs > P[x]) {",
     SAMPLING_PINS),
    ("sampling: residual of the draft over the target",
     "for (int v = 0; v < Voc; ++v) P[v] = (P[v] > Q[v] ? P[v] - Q[v] : 0.0) / s;",
     "for (int v = 0; v < Voc; ++v) P[v] = (Q[v] > P[v] ? Q[v] - P[v] : 0.0) / s;", SAMPLING_PINS),
    ("sampling: temperature ignored", "P[v] = exp(((double)lu[v] - m) / temperature);",
     "P[v] = exp((double)lu[v] - m);", SAMPLING_PINS),
    ("sampling: no residual after a rejection",
     "        if (s > 0.0)\n          for (int v = 0; v < Voc; ++v) P[v] = (P[v] > Q[v] ? P[v] - Q[v] : 0.0) / s;",
     "", SAMPLING_PINS),
    ("expansion scores the raw logit", "((double)row[best] - lse)", "((double)row[best])",
     EXPAND_PINS),
    ("expansion drops the parent's score", "(float)((double)scores[pb + parent] + ((double)row[best] - lse))",
     "(float)((double)row[best] - lse)", EXPAND_PINS),
    ("children are the least likely tokens", "if (!taken[v] && (best < 0 || row[v] > row[best])) best = v;",
     "if (!taken[v] && (best < 0 || row[v] < row[best])) best = v;", EXPAND_PINS),
    ("equal logits go to the higher token index",
     "if (!taken[v] && (best < 0 || row[v] > row[best])) best = v;",
     "if (!taken[v] && (best < 0 || row[v] >= row[best])) best = v;", EXPAND_PINS),
    ("beam keeps the lowest scores",
     "if (!taken[c] && (best < 0 || scores[pb + first + c] > scores[pb + first + best])) best = c;",
     "if (!taken[c] && (best < 0 || scores[pb + first + c] < scores[pb + first + best])) best = c;",
     EXPAND_PINS),
    ("beam ties go to the higher pool index",
     "if (!taken[c] && (best < 0 || scores[pb + first + c] > scores[pb + first + best])) best = c;",
     "if (!taken[c] && (best < 0 || scores[pb + first + c] >= scores[pb + first + best])) best = c;",
     EXPAND_PINS),
    ("a child scoring above its parent accepted",
     "if (i > 0 && sc[i] > sc[par[i]]) return LTDO_STATUS_BAD_SCORE;",
     "if (i > 0 && sc[i] > sc[par[i]] + 1.0f) return LTDO_STATUS_BAD_SCORE;", SELECT_PINS),
]


def _build_mutant(tmp_path, idx, orig, mutated):
    src = open(SRC).read()
    assert src.count(orig) >= 1, f"mutation anchor not found: {orig!r}"
    msrc = src.replace(orig, mutated, 1)
    cpath = tmp_path / f"mutant{idx}.c"
    cpath.write_text(msrc)
    so = tmp_path / f"mutant{idx}.so"
    inc = os.path.dirname(SRC)
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-I", inc, "-o",
                    str(so), str(cpath), "-lm"], check=True)
    return str(so)


def _pins_pass(pins):
    for pin in pins:
        try:
            pin()
        except (AssertionError, oracle.OracleError):
            return False
    return True


def test_unmutated_oracle_passes_every_pin():
    assert _pins_pass(ATTN_PINS + ACCEPT_PINS + COMPACT_PINS + SELECT_PINS + EXPAND_PINS +
                      SAMPLING_PINS)


@pytest.mark.parametrize("idx", range(len(MUTANTS)), ids=[m[0] for m in MUTANTS])
def test_every_mutant_is_caught(idx, tmp_path, monkeypatch):
    name, orig, mutated, pins = MUTANTS[idx]
    so = _build_mutant(tmp_path, idx, orig, mutated)
    monkeypatch.setattr(oracle, "_lib", oracle.load_library(so))
    np.seterr(all="ignore")
    assert not _pins_pass(pins), f"pins did not notice: {name}"


# ---- the policy oracle (numpy): the same idea, planted in a copy of its source
import importlib.util  # noqa: E402

import test_oracle_policy as TP  # noqa: E402
from oracle import policy as _policy  # noqa: E402

POLICY_PINS = [
    lambda: TP.test_worked_examples(),
    lambda: TP.test_matches_torch_linear_relu_stack((7, 5, 3)),
    lambda: TP.test_zero_weights_give_the_bias_and_the_action_map(),
    lambda: TP.test_state_layouts(),
]
POLICY_MUTANTS = [
    ("ReLU missing", "h = np.maximum(h, 0.0)", "h = h"),
    ("bias dropped", "h = h @ np.asarray(w, np.float64).T + np.asarray(bias, np.float64)",
     "h = h @ np.asarray(w, np.float64).T"),
    ("ReLU on the logits too", "if k + 1 < len(layers):", "if True:"),
    ("argmax ties to the last index", "np.argmax(h, axis=1)",
     "(h.shape[1] - 1 - np.argmax(h[:, ::-1], axis=1))"),
    ("size-policy scalars swapped", "out[b, 0] = depth[b]\n            out[b, 1] = ctx_len[b]",
     "out[b, 0] = ctx_len[b]\n            out[b, 1] = depth[b]"),
    ("depth window misses the newest score", "out[b, n_feat - k:n_feat] = scores[b, n - k:n]",
     "out[b, n_feat - k:n_feat] = scores[b, max(n - k - 1, 0):max(n - 1, k)]"),
]


def test_unmutated_policy_oracle_passes_every_pin():
    for pin in POLICY_PINS:
        pin()


@pytest.mark.parametrize("idx", range(len(POLICY_MUTANTS)), ids=[m[0] for m in POLICY_MUTANTS])
def test_every_policy_mutant_is_caught(idx, tmp_path, monkeypatch):
    name, orig, mutated = POLICY_MUTANTS[idx]
    src = open(_policy.__file__).read()
    assert src.count(orig) >= 1, f"mutation anchor not found: {orig!r}"
    path = tmp_path / f"policy_mutant{idx}.py"
    path.write_text(src.replace(orig, mutated, 1))
    spec = importlib.util.spec_from_file_location(f"policy_mutant{idx}", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    monkeypatch.setattr(TP, "OP", mod)
    caught = False
    for pin in POLICY_PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught = True
            break
    assert caught, f"pins did not notice: {name}"
