"""Pins for the oracle's candidate token selection (CPU only).

Section 3.2 ("Candidate Token Selection") keeps the V candidates of the draft
tree with the highest cumulative path probability and flattens them with a
tree mask.  Readings: equal scores rank the lower pool index first; the kept
candidates are flattened in pool order.  The pins:

* hand-derived worked examples with ties across and within depths, a pool
  not listed level by level, a child equal to its parent, signed zero and -inf
  (tests/golden/select_examples.json);
* the generator's own independent selection (workloads.tree_eagle) on the
  paper's pool shapes, where scores are distinct (same kept set, same tree);
* special cases that reduce to library routines: a star pool is numpy's
  stable argsort, and with distinct scores the kept set is numpy's top-V;
* exhaustive small pools (every tree with N <= 6, every 0/1 score decrement
  pattern, every V) and random pools with heavy ties, against the defining
  properties: V = min(n_select, pool size) candidates, ancestor-closed, no
  left-out candidate ranks before a kept one, listed in pool order, parents
  re-indexed to the same candidates, true depths;
* validation codes.
"""
import json
import os

import numpy as np
import pytest

import oracle
from brute import all_parent_arrays, root_path
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_examples.json")


def _pack(pars, scores, toks=None, Vpool=None):
    """List of per-sequence pools -> padded [B, Vpool] arrays (junk padding)."""
    B = len(pars)
    Vpool = Vpool or max(len(p) for p in pars)
    P = np.full((B, Vpool), Vpool + 3, np.int32)
    S = np.full((B, Vpool), np.float32(7.0), np.float32)
    T = np.full((B, Vpool), -9, np.int32)
    for b in range(B):
        n = len(pars[b])
        P[b, :n] = pars[b]
        S[b, :n] = scores[b]
        T[b, :n] = toks[b] if toks is not None else 1000 + np.arange(n)
    return S, P, T, np.array([len(p) for p in pars], np.int32)


def _true_depth(par):
    return [len(root_path(par, i)) - 1 for i in range(len(par))]


def _ranks_before(u, s, sc):
    """Does pool candidate u rank before s (the selection order's definition:
    higher score, then lower pool index)?"""
    if sc[u] != sc[s]:
        return sc[u] > sc[s]
    return u < s


def check_selection(par, sc, tok, n_select, got):
    """The defining properties of one sequence's result."""
    sel, newpar, newtok, newdep, nn = got
    n = len(par)
    V = min(n_select, n)
    dep = _true_depth(par)
    assert nn == V
    assert (sel[V:] == -1).all() and (newpar[V:] == -1).all()
    kept = [int(x) for x in sel[:V]]
    assert len(set(kept)) == V and all(0 <= x < n for x in kept)
    S = set(kept)
    for x in kept:  # a rooted subtree
        assert par[x] == -1 or par[x] in S
    for s in kept:  # nothing left out ranks before anything kept
        for u in range(n):
            if u not in S:
                assert not _ranks_before(u, s, sc), (u, s)
    assert kept == sorted(kept)
    assert kept[0] == 0 and newpar[0] == -1
    for k in range(1, V):
        assert 0 <= newpar[k] < k
        assert kept[newpar[k]] == par[kept[k]]
    assert newtok[:V].tolist() == [int(tok[x]) for x in kept]
    assert newdep[:V].tolist() == [dep[x] for x in kept]


def _run(S, P, T, sizes, nsel, Nmax):
    return oracle.select_candidates(S, P, T, sizes, np.asarray(nsel, np.int32), Nmax)


def test_worked_examples():
    g = json.load(open(GOLDEN))
    par = np.array(g["pool"]["parents"], np.int32)
    sc = np.array([float(x) for x in g["pool"]["scores"]], np.float32)
    tok = np.array(g["pool"]["tokens"], np.int32)
    assert _true_depth(par) == g["pool"]["depth"]
    assert np.signbit(sc[1]) and not np.signbit(sc[0])
    for ex in g["examples"]:
        Nmax = max(ex["n_select"], 16)
        sel, np_, nt, nd, nn = _run(sc[None], par[None], tok[None], np.array([len(par)], np.int32),
                                    [ex["n_select"]], Nmax)
        V = len(ex["selected"])
        assert nn[0] == V, ex["name"]
        assert sel[0, :V].tolist() == ex["selected"], ex["name"]
        assert np_[0, :V].tolist() == ex["parents"], ex["name"]
        assert nt[0, :V].tolist() == ex["tokens"], ex["name"]
        assert nd[0, :V].tolist() == ex["depth"], ex["name"]
        assert (sel[0, V:] == -1).all()


@pytest.mark.parametrize("depth,width,n", [(6, 10, 60), (4, 4, 24), (12, 10, 240), (8, 10, 100),
                                           (3, 5, 31), (1, 10, 1)])
def test_matches_the_generators_own_selection(depth, width, n):
    """workloads.tree_eagle cuts the same pool with its own code; where the
    float32 scores are distinct both keep the same candidates and build the
    same tree (it lists them by (level, score), the oracle in pool order, so
    nodes are matched by their distinct scores)."""
    for seed in range(3):
        pool = W.draft_pool(W.rng_for(seed), depth, width, 1000)
        tree = W.tree_eagle(W.rng_for(seed), n, depth, width, 1000)
        sc32 = pool.scores.astype(np.float32)
        assert len(np.unique(sc32)) == len(sc32)
        S, P, T, sizes = _pack([pool.parents], [sc32], [pool.tokens])
        sel, par, tok, dep, nn = _run(S, P, T, sizes, [n], n)
        assert nn[0] == n
        got = {float(pool.scores[j]): (float(pool.scores[sel[0, par[0, k]]]) if k else None,
                                       int(tok[0, k]), int(dep[0, k]))
               for k, j in enumerate(sel[0])}
        want = {float(tree.scores[k]): (float(tree.scores[tree.parents[k]]) if k else None,
                                        int(tree.tokens[k]), len(root_path(tree.parents, k)) - 1)
                for k in range(n)}
        assert got == want
        assert dep[0].tolist() == pool.level[sel[0]].tolist()


def test_star_pool_is_a_stable_argsort():
    """Root plus n-1 children: the kept children are the first V-1 of numpy's
    stable descending argsort (ties -> lower index), listed in pool order."""
    rng = np.random.default_rng(5)
    n = 40
    par = W.tree_star(n)
    sc = np.concatenate([[0.0], -rng.integers(0, 6, size=n - 1)]).astype(np.float32)
    S, P, T, sizes = _pack([par], [sc])
    for V in (1, 2, 7, 39, 40, 55):
        sel, npar, _, dep, nn = _run(S, P, T, sizes, [V], max(V, n))
        children = 1 + np.argsort(-sc[1:], kind="stable")
        want = [0] + sorted(children[:min(V, n) - 1].tolist())
        assert sel[0, :nn[0]].tolist() == want
        assert (npar[0, 1:nn[0]] == 0).all() and (dep[0, 1:nn[0]] == 1).all()


def test_chain_pool_keeps_its_first_v_links():
    n = 30
    par = W.tree_chain(n)
    sc = -np.arange(n, dtype=np.float32) * 0.25
    sc[10:14] = sc[9]  # equal to the parent: depth decides
    S, P, T, sizes = _pack([par], [sc])
    for V in (1, 5, 12, 30, 31):
        sel, npar, _, dep, nn = _run(S, P, T, sizes, [V], 32)
        k = min(V, n)
        assert sel[0, :k].tolist() == list(range(k))
        assert npar[0, :k].tolist() == [-1] + list(range(k - 1))
        assert dep[0, :k].tolist() == list(range(k))


def test_distinct_scores_keep_numpys_top_v():
    """With distinct scores the kept set is the V largest (numpy argpartition)."""
    rng = np.random.default_rng(8)
    for n, V in ((411, 60), (1011, 240), (211, 140), (64, 64)):
        par = W.tree_uniform_parent(rng, n)
        dec = rng.random(n).astype(np.float64) + 1e-3
        sc = np.zeros(n)
        for i in range(1, n):
            sc[i] = sc[par[i]] - dec[i]
        sc = sc.astype(np.float32)
        assert len(np.unique(sc)) == n
        S, P, T, sizes = _pack([par], [sc])
        sel, *_ = _run(S, P, T, sizes, [V], 256)
        top = np.argpartition(-sc, V - 1)[:V] if V < n else np.arange(n)
        assert sorted(sel[0, :V].tolist()) == sorted(top.tolist())


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 6])
def test_exhaustive_small_pools(n):
    """Every tree with n nodes x every 0/1 decrement pattern (0 = a child equal
    to its parent) x every V in 1..n+1, one batched call per V."""
    pars, scs = [], []
    for par in all_parent_arrays(n):
        for mask in range(1 << (n - 1)):
            dec = [0] + [(mask >> (c - 1)) & 1 for c in range(1, n)]
            sc = np.zeros(n, np.float32)
            for i in range(1, n):
                sc[i] = sc[par[i]] - dec[i]
            pars.append(np.array(par, np.int32))
            scs.append(sc)
    S, P, T, sizes = _pack(pars, scs)
    for V in range(1, n + 2):
        got = _run(S, P, T, sizes, [V] * len(pars), n + 1)
        for b in range(len(pars)):
            check_selection(pars[b], scs[b], T[b], V, [g[b] for g in got])


@pytest.mark.parametrize("seed", range(4))
def test_random_pools_with_heavy_ties(seed):
    rng = np.random.default_rng(100 + seed)
    pars, scs, nsel = [], [], []
    for _ in range(12):
        n = int(rng.integers(1, 300))
        par = W.tree_uniform_parent(rng, n)
        sc = np.zeros(n, np.float32)
        for i in range(1, n):
            step = rng.choice([0.0, 0.5, 1.0, np.inf], p=[0.3, 0.3, 0.35, 0.05])
            sc[i] = sc[par[i]] - np.float32(step)
        if n > 1 and seed % 2:
            sc[1:] = np.where(sc[1:] == 0, np.float32(-0.0), sc[1:])
        pars.append(par)
        scs.append(sc)
        nsel.append(int(rng.integers(1, 257)))
    S, P, T, sizes = _pack(pars, scs, Vpool=W.MAX_POOL)
    got = _run(S, P, T, sizes, nsel, 256)
    for b in range(len(pars)):
        check_selection(pars[b], scs[b], T[b], nsel[b], [g[b] for g in got])


def test_generated_batches():
    for mk in (W.select_8b, W.select_deep, W.select_batch16):
        sb = mk()
        got = _run(sb.scores, sb.pool_parents, sb.pool_tokens, sb.pool_size, sb.n_select, sb.Nmax)
        for b in range(sb.B):
            n = sb.pool_size[b]
            check_selection(sb.pool_parents[b, :n], sb.scores[b, :n], sb.pool_tokens[b, :n],
                            int(sb.n_select[b]), [g[b] for g in got])


def _status(S, P, T, sizes, nsel, Nmax):
    try:
        _run(S, P, T, sizes, nsel, Nmax)
        return 0
    except oracle.OracleError as e:
        return e.code


def test_validation_codes():
    par = W.tree_uniform_parent(np.random.default_rng(2), 20)
    sc = -np.arange(20, dtype=np.float32)
    for i in range(1, 20):
        sc[i] = sc[par[i]] - 1
    S, P, T, sizes = _pack([par, par], [sc, sc], Vpool=24)
    assert _status(S, P, T, sizes, [5, 5], 8) == 0
    bad = sizes.copy(); bad[1] = 0
    assert _status(S, P, T, bad, [5, 5], 8) == oracle.STATUS_BAD_NNODES
    bad[1] = 25
    assert _status(S, P, T, bad, [5, 5], 8) == oracle.STATUS_BAD_NNODES
    assert _status(S, P, T, sizes, [5, 9], 8) == oracle.STATUS_BAD_NNODES
    assert _status(S, P, T, sizes, [0, 5], 8) == oracle.STATUS_BAD_NNODES
    P2 = P.copy(); P2[1, 0] = 0
    assert _status(S, P2, T, sizes, [5, 5], 8) == oracle.STATUS_BAD_PARENT
    P2 = P.copy(); P2[0, 7] = 7
    assert _status(S, P2, T, sizes, [5, 5], 8) == oracle.STATUS_BAD_PARENT
    S2 = S.copy(); S2[1, 3] = np.nan
    assert _status(S2, P, T, sizes, [5, 5], 8) == oracle.STATUS_BAD_SCORE
    S2 = S.copy(); c = 11; S2[0, c] = S2[0, par[c]] + 0.5
    assert _status(S2, P, T, sizes, [5, 5], 8) == oracle.STATUS_BAD_SCORE
    # the padding past a pool's size is never read
    S2 = S.copy(); S2[:, 20:] = np.nan
    P2 = P.copy(); P2[:, 20:] = 99
    assert _status(S2, P2, T, sizes, [5, 5], 8) == 0
