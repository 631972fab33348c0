"""Pins for the oracle's greedy acceptance (CPU only).

* hand-derived worked examples (tests/golden/accept_examples.json);
* exhaustive: every tree with N <= 6 times every accept/reject pattern of its
  draft tokens, against an enumerator that lists all root paths;
* argmax special cases against numpy.argmax (ties -> lowest index, -0 == +0);
* greedy equivalence: verifying a draft tree on a toy LM emits exactly the
  tokens that token-by-token greedy decoding emits (section 3.2, "Draft Tree
  Verification": accept up to the first mismatch, append the target's token).
"""
import json
import os

import numpy as np
import pytest

import oracle
from brute import ToyLM, accept_by_enumeration, all_parent_arrays, root_path

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "accept_examples.json")


def _onehot_logits(pred, vocab):
    lg = np.zeros((len(pred), vocab), np.float32)
    lg[np.arange(len(pred)), pred] = 1.0
    return lg


def test_worked_examples():
    g = json.load(open(GOLDEN))
    par = np.array(g["tree"]["parents"], np.int32)
    tok = np.array(g["tree"]["draft_tokens"], np.int32)
    for i, anc in enumerate(g["ancestors"]):
        assert root_path(par, i) == anc
    for ex in g["examples"]:
        lg = _onehot_logits(ex["pred"], 16)
        pred, acc, toks, n = oracle.tree_accept(lg[None], tok[None], par[None], np.array([7], np.int32))
        assert pred[0].tolist() == ex["pred"], ex["name"]
        k = ex["n_accepted"]
        assert n[0] == k, ex["name"]
        assert acc[0, :k].tolist() == ex["accepted_nodes"], ex["name"]
        assert toks[0, :k].tolist() == ex["out_tokens"], ex["name"]


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 6])
def test_exhaustive_small_trees_all_patterns(n):
    """Batch every (tree, pattern) pair into one call.  pred[u] = 100 + u; a
    'valid' node copies its parent's pred, an invalid one takes a token no
    node predicts.  Several valid siblings give duplicate sibling tokens."""
    cases = []
    for par in all_parent_arrays(n):
        for mask in range(1 << (n - 1)):
            valid = [True] + [bool(mask >> (c - 1) & 1) for c in range(1, n)]
            pred = np.array([100 + u for u in range(n)], np.int32)
            tok = np.array([7] + [pred[par[c]] if valid[c] else 1 for c in range(1, n)], np.int32)
            cases.append((par, pred, tok))
    B = len(cases)
    vocab = 100 + n
    logits = np.stack([_onehot_logits(p, vocab) for _, p, _ in cases])
    parents = np.stack([c[0] for c in cases])
    tokens = np.stack([c[2] for c in cases])
    pred, acc, toks, nacc = oracle.tree_accept(logits, tokens, parents, np.full(B, n, np.int32))
    for b, (par, pr, tok) in enumerate(cases):
        path, emitted = accept_by_enumeration(pr, tok, par)
        k = len(path)
        assert nacc[b] == k
        assert acc[b, :k].tolist() == path
        assert toks[b, :k].tolist() == emitted


def test_argmax_ties_and_signed_zero_match_numpy():
    rng = np.random.default_rng(3)
    rows = [
        np.array([-0.0, 0.0, -1.0], np.float32),
        np.array([-1.0, 0.0, -0.0, 0.0], np.float32),
        np.array([2.0, 5.0, 5.0, 1.0, 5.0], np.float32),
        np.array([-3.0, -2.0, -2.0, -7.0], np.float32),
        np.array([np.float32(-np.inf), -1e30, -1e30], np.float32),
        rng.integers(-3, 4, size=257).astype(np.float32),
    ]
    V = max(len(r) for r in rows)
    logits = np.full((len(rows), 1, V), -np.inf, np.float32)
    for i, r in enumerate(rows):
        logits[i, 0, :len(r)] = r
    n = len(rows)
    pred, *_ = oracle.tree_accept(logits, np.zeros((n, 1), np.int32), np.full((n, 1), -1, np.int32),
                                  np.ones(n, np.int32))
    for i, r in enumerate(rows):
        assert pred[i, 0] == int(np.argmax(r)), i


def _tree_with_greedy_branch(rng, greedy, k, distractors, vocab):
    """Root + chain of the first k greedy tokens + random distractor nodes.

    Distractor tokens differ from the greedy token of the same parent, so the
    accepted path is exactly the greedy chain (siblings stay distinct)."""
    parents = [-1]
    tokens = [None]  # root token filled by the caller
    chain = [0]
    for j in range(k):
        parents.append(chain[-1])
        tokens.append(greedy[j])
        chain.append(len(parents) - 1)
    for _ in range(distractors):
        p = int(rng.integers(0, len(parents)))
        used = {tokens[c] for c in range(1, len(parents)) if parents[c] == p}
        if p in chain and chain.index(p) < len(greedy):
            used.add(greedy[chain.index(p)])
        choices = [t for t in range(vocab) if t not in used]
        parents.append(p)
        tokens.append(int(rng.choice(choices)))
    # renumber into a random topological order
    n = len(parents)
    placed, order = {0}, [0]
    while len(order) < n:
        ready = [i for i in range(n) if i not in placed and parents[i] in placed]
        pick = ready[rng.integers(0, len(ready))]
        placed.add(pick)
        order.append(pick)
    new_of = {o: i for i, o in enumerate(order)}
    par2 = np.array([-1] + [new_of[parents[o]] for o in order[1:]], np.int32)
    tok2 = [tokens[o] for o in order]
    return par2, tok2


def _verify_on_toy_lm(lm, prompt, par, tok):
    """Tree verification with the oracle: prefix K/V = prompt[:-1], root =
    prompt[-1]; node i sits at position P + depth(i); per-node logits come
    from the oracle's attention output through the toy LM's head."""
    P = len(prompt) - 1
    n = len(par)
    depth = [len(root_path(par, i)) - 1 for i in range(n)]
    tok = list(tok)
    tok[0] = prompt[-1]
    cap = P + n
    kc = np.zeros((1, lm.Hkv, cap, lm.d), np.float32)
    vc = np.zeros_like(kc)
    for p in range(P):
        _, k, v = lm.qkv(prompt[p], p)
        kc[0, :, p], vc[0, :, p] = k, v
    q = np.zeros((1, n, lm.Hq, lm.d), np.float32)
    for i in range(n):
        qi, k, v = lm.qkv(tok[i], P + depth[i])
        q[0, i] = qi
        kc[0, :, P + i], vc[0, :, P + i] = k, v
    att = oracle.tree_verify_attn(q, kc, vc, np.array([P], np.int32), par[None],
                                  np.array([n], np.int32), Hkv=lm.Hkv, dtype=oracle.DTYPE_F32)[0]
    logits = np.stack([lm.logits_from_attention(tok[i], P + depth[i], att[i]) for i in range(n)])
    return oracle.tree_accept(logits[None], np.array([tok], np.int32), par[None],
                              np.array([n], np.int32))


@pytest.mark.parametrize("seed", range(6))
def test_greedy_equivalence_on_toy_lm(seed):
    lm = ToyLM(seed)
    rng = np.random.default_rng(1000 + seed)
    prompt = [int(t) for t in rng.integers(0, lm.vocab, size=int(rng.integers(3, 12)))]
    steps = 8
    greedy, margin = lm.greedy(prompt, steps)
    assert margin > 1e-6  # no near-ties: both sides decide the same argmax
    for k in range(0, steps):
        par, tok = _tree_with_greedy_branch(rng, greedy, k, distractors=int(rng.integers(0, 12)),
                                            vocab=lm.vocab)
        pred, acc, toks, nacc = _verify_on_toy_lm(lm, prompt, par, tok)
        assert nacc[0] == k + 1
        assert toks[0, :k + 1].tolist() == greedy[:k + 1]
    # a chain tree made of the whole greedy continuation accepts all of it
    par = np.arange(-1, steps, dtype=np.int32)
    pred, acc, toks, nacc = _verify_on_toy_lm(lm, prompt, par, [0] + greedy)
    assert nacc[0] == steps + 1
    assert toks[0, :steps].tolist() == greedy


def test_bad_parents_rejected():
    lg = np.zeros((1, 3, 4), np.float32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.tree_accept(lg, np.zeros((1, 3), np.int32), np.array([[-1, 1, 0]], np.int32),
                           np.array([3], np.int32))
    assert e.value.code == oracle.STATUS_BAD_PARENT
    with pytest.raises(oracle.OracleError) as e:
        oracle.tree_accept(lg, np.zeros((1, 3), np.int32), np.array([[-1, 0, 0]], np.int32),
                           np.array([4], np.int32))
    assert e.value.code == oracle.STATUS_BAD_NNODES
