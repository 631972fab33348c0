"""Pins for the oracle's acceptance by recursive rejection sampling (CPU).

The paper runs its experiments at T = 0 and T = 1 and does not print the
T > 0 acceptance rule; the oracle follows the published recursive rejection
sampling for drafts drawn without replacement.  What pins it is the property
that rule exists for: the emitted tokens are distributed exactly as the
target model's own sampling.  The pins:

* statistical losslessness on a toy model (vocabulary 6, T = 0.7): over
  200000 independent verifications with fresh drafts and uniforms, the first
  emitted token follows the root's target distribution, and the second
  follows the target conditioned on the first (every |z| < 5);
* hand-derived worked examples (tests/golden/sampling_examples.json);
* special cases: a draft equal to the target always accepts the first child;
  a lone root samples its target by inverse CDF exactly as numpy's
  searchsorted over the cumulative sum does.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "sampling_examples.json")


def _softmax(l, T):
    e = np.exp((l - l.max(-1, keepdims=True)) / T)
    return e / e.sum(-1, keepdims=True)


def _draw_without_replacement(rng, probs, k):
    """k draws without replacement, in draw order, for each row of probs: the
    order of the k largest of log p + Gumbel noise (the Gumbel-top-k identity
    for sequential sampling without replacement)."""
    g = np.log(probs) - np.log(-np.log(rng.random(probs.shape)))
    return np.argsort(-g, axis=-1, kind="stable")[..., :k]


def toy_batch(rng, n_trials, V=6, T=0.7, n_children=3):
    """A root with n_children drafts drawn without replacement from the root's
    draft distribution; each child has 2 drafts of its own drawn from the
    draft distribution of its token.  Targets depend on the token path only
    (a toy language model): root logits L0, a child with token x has L1[x]."""
    L0 = rng.normal(size=V) * 1.5
    L1 = rng.normal(size=(V, V)) * 1.5
    Q0 = _softmax(rng.normal(size=V), 1.0)
    Q1 = _softmax(rng.normal(size=(V, V)), 1.0)
    N = 1 + n_children + 2 * n_children
    parents = np.array([-1] + [0] * n_children + [1 + i // 2 for i in range(2 * n_children)],
                       np.int32)
    B = n_trials
    tok = np.zeros((B, N), np.int32)
    logits = np.zeros((B, N, V), np.float32)
    q = np.zeros((B, N, V), np.float32)
    logits[:, 0] = L0
    q[:, 0] = Q0
    xs = _draw_without_replacement(rng, np.tile(Q0, (B, 1)), n_children)
    tok[:, 1:1 + n_children] = xs
    for i in range(n_children):
        c = 1 + i
        logits[:, c] = L1[xs[:, i]]
        q[:, c] = Q1[xs[:, i]]
        gs = _draw_without_replacement(rng, Q1[xs[:, i]], 2)
        for j in range(2):
            gc = 1 + n_children + 2 * i + j
            tok[:, gc] = gs[:, j]
            logits[:, gc] = rng.normal(size=(B, V))  # deeper targets are not checked
    uni = rng.random((B, N, 2)).astype(np.float32)
    par = np.tile(parents, (B, 1))
    return dict(logits=logits, q=q, tok=tok, par=par, n=np.full(B, N, np.int32), uni=uni, T=T,
                P0=_softmax(L0, T), P1=_softmax(L1, T))


def test_gumbel_draws_match_numpys_sequential_choice():
    """The vectorised draw is numpy's sequential choice without replacement in
    distribution: compare the frequencies of the ordered first two draws."""
    rng = np.random.default_rng(9)
    p = _softmax(rng.normal(size=5), 1.0)
    g = _draw_without_replacement(rng, np.tile(p, (60000, 1)), 2)
    c = np.array([rng.choice(5, size=2, replace=False, p=p) for _ in range(60000)])
    fg = np.bincount(g[:, 0] * 5 + g[:, 1], minlength=25) / 60000
    fc = np.bincount(c[:, 0] * 5 + c[:, 1], minlength=25) / 60000
    assert np.abs(fg - fc).max() < 0.01


def _z_ok(counts, probs, label):
    n = counts.sum()
    expect = n * probs
    sd = np.sqrt(n * probs * (1 - probs)) + 1e-12
    z = (counts - expect) / sd
    assert np.abs(z).max() < 5, (label, z)


def test_losslessness_on_a_toy_model():
    rng = np.random.default_rng(1)
    tb = toy_batch(rng, 200000)
    acc, toks, n_acc, _ = oracle.tree_accept_sampling(tb["logits"], tb["q"], tb["tok"], tb["par"],
                                                      tb["n"], tb["uni"], temperature=tb["T"])
    V = tb["P0"].size
    first = toks[:, 0]
    _z_ok(np.bincount(first, minlength=V), tb["P0"], "first token")
    two = n_acc >= 2
    assert two.mean() > 0.3  # the drafts are accepted often enough to test the second token
    for y in range(V):
        sel = two & (first == y)
        if sel.sum() > 2000:
            _z_ok(np.bincount(toks[sel, 1], minlength=V), tb["P1"][y], f"second token after {y}")


def test_worked_examples():
    g = json.load(open(GOLDEN))
    for ex in g["examples"]:
        logits = np.log(np.array([g["root_p"]] + g["leaf_p"], np.float32))[None]
        q = np.array([g["root_q"], [1, 1, 1], [1, 1, 1]], np.float32)[None]
        tok = np.array([[7] + ex["tokens"]], np.int32)
        par = np.array([[-1, 0, 0]], np.int32)
        uni = np.zeros((1, 3, 2), np.float32)
        uni[0, 1:, 0] = ex["r_child"]
        uni[0, :, 1] = ex["r_bonus"]
        acc, toks, n, _ = oracle.tree_accept_sampling(logits, q, tok, par, np.array([3], np.int32),
                                                      uni, temperature=1.0)
        k = ex["n_accepted"]
        assert n[0] == k, ex["name"]
        assert acc[0, :k].tolist() == ex["accepted_nodes"], ex["name"]
        assert toks[0, :k].tolist() == ex["out_tokens"], ex["name"]


def test_draft_equal_to_target_accepts_the_first_child():
    rng = np.random.default_rng(2)
    V, B = 50, 400
    L = rng.normal(size=(B, 4, V)).astype(np.float32)
    T = 0.9
    q = _softmax(L.astype(np.float64), T).astype(np.float32)
    tok = rng.integers(0, V, size=(B, 4)).astype(np.int32)
    par = np.tile(np.array([-1, 0, 0, 1], np.int32), (B, 1))
    uni = rng.random((B, 4, 2)).astype(np.float32) * 0.999
    acc, toks, n, _ = oracle.tree_accept_sampling(L, q, tok, par, np.full(B, 4, np.int32), uni,
                                                  temperature=T)
    assert (acc[:, 1] == 1).all() and (acc[:, 2] == 3).all() and (n == 3).all()


def test_lone_root_is_inverse_cdf_sampling():
    rng = np.random.default_rng(3)
    B, V = 300, 1000
    L = (rng.normal(size=(B, 1, V)) * 2).astype(np.float32)
    uni = rng.random((B, 1, 2)).astype(np.float32)
    acc, toks, n, _ = oracle.tree_accept_sampling(L, np.ones_like(L), np.zeros((B, 1), np.int32),
                                                  np.full((B, 1), -1, np.int32),
                                                  np.ones(B, np.int32), uni, temperature=1.3)
    P = _softmax(L[:, 0].astype(np.float64), 1.3)
    cdf = np.cumsum(P, axis=1)
    want = [int(np.searchsorted(cdf[b], uni[b, 0, 1] * cdf[b, -1], side="right")) for b in range(B)]
    assert (n == 1).all() and toks[:, 0].tolist() == want
