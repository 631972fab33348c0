"""Pins for the oracle's draft tree expansion (CPU only).

Section 3.2 ("Draft Tree Generation"): each leaf gets the W most probable
tokens of its draft distribution as children, scored by cumulative path
log-probability, and the W children of highest score become the next leaves;
the pool grows to 1 + W + (D-2) W^2 candidates.  The pins:

* replaying the generator's own beam (workloads.draft_pool, written
  independently) from logits that carry its recorded draws: same parents,
  tokens and leaves, scores within float32 rounding, and the pool size
  formula;
* a different library: torch log_softmax + topk (float64) on random rows;
* hand-built ties: equal logits go to the lower token index, equal child
  scores to the lower pool index;
* validation codes.
"""
import numpy as np
import pytest

import oracle
import workloads as W


def _empty_pool(B, Vpool):
    return (np.zeros((B, Vpool), np.float32), np.full((B, Vpool), -1, np.int32),
            np.zeros((B, Vpool), np.int32), np.ones(B, np.int32))


def _row_for(draw, vocab):
    """Logits whose softmax is the draw's W + 1 Dirichlet components: the W
    child tokens and one more token carry log p, every other token -inf."""
    _, full, toks = draw
    row = np.full(vocab, -np.inf, np.float32)
    row[toks] = np.log(full[:len(toks)]).astype(np.float32)
    extra = next(v for v in range(vocab) if v not in set(toks.tolist()))
    row[extra] = np.float32(np.log(full[len(toks)]))
    return row


@pytest.mark.parametrize("depth,width,vocab", [(6, 10, 4000), (4, 4, 50), (12, 5, 300), (2, 3, 10),
                                               (3, 10, 128256)])
def test_replays_the_generators_beam(depth, width, vocab):
    pool = W.draft_pool(W.rng_for(depth * 100 + width), depth, width, vocab)
    n = len(pool.parents)
    assert n == W.pool_size(depth, width)
    scores, par, tok, size = _empty_pool(1, n)
    tok[0, 0] = pool.tokens[0]
    draws = list(pool.draws)
    frontier = np.zeros((1, 1), np.int32)
    k = 0
    for rnd in range(depth - 1):
        F = frontier.shape[1]
        rows = np.stack([_row_for(draws[k + f], vocab) for f in range(F)])
        assert [draws[k + f][0] for f in range(F)] == frontier[0].tolist()
        k += F
        scores, par, tok, size, frontier = oracle.draft_expand(
            rows[None], frontier, scores, par, tok, size, W=width, W_next=width)
    assert k == len(draws) and size[0] == n
    np.testing.assert_array_equal(par[0], pool.parents)
    np.testing.assert_array_equal(tok[0], pool.tokens)
    np.testing.assert_allclose(scores[0], pool.scores, rtol=0, atol=1e-5 * depth)


def test_matches_torch_log_softmax_topk():
    import torch
    rng = np.random.default_rng(3)
    B, F, Voc, Wd = 2, 3, 5000, 7
    logits = rng.normal(size=(B, F, Voc)).astype(np.float32) * 3
    scores, par, tok, size = _empty_pool(B, 64)
    scores[:, :5] = rng.normal(size=(B, 5)).astype(np.float32) - 2
    size[:] = 5
    frontier = np.array([[4, 0, 2], [1, 3, 3]], np.int32)
    s2, p2, t2, n2, nf = oracle.draft_expand(logits, frontier, scores, par, tok, size, W=Wd,
                                             W_next=6)
    lsm = torch.log_softmax(torch.from_numpy(logits.astype(np.float64)), dim=-1)
    top = torch.topk(lsm, Wd, dim=-1)
    for b in range(B):
        child_scores = []
        for f in range(F):
            sl = slice(5 + f * Wd, 5 + (f + 1) * Wd)
            assert t2[b, sl].tolist() == top.indices[b, f].tolist()
            assert (p2[b, sl] == frontier[b, f]).all()
            want = scores[b, frontier[b, f]].astype(np.float64) + top.values[b, f].numpy()
            np.testing.assert_allclose(s2[b, sl], want, rtol=0, atol=1e-5)
            child_scores += s2[b, sl].tolist()
        beam = torch.topk(torch.tensor(child_scores), 6).indices.numpy() + 5
        assert nf[b].tolist() == beam.tolist()
        assert n2[b] == 5 + F * Wd


def test_ties():
    """Equal logits: the lower token index first.  Equal child scores: the
    lower pool index first."""
    logits = np.full((1, 2, 6), -5.0, np.float32)
    logits[0, 0, [4, 1, 3]] = 2.0  # three-way tie
    logits[0, 1, [5, 0, 2]] = 2.0  # the same values in another order
    scores, par, tok, size = _empty_pool(1, 16)
    size[:] = 3
    frontier = np.array([[2, 1]], np.int32)
    s2, p2, t2, n2, nf = oracle.draft_expand(logits, frontier, scores, par, tok, size, W=2,
                                             W_next=3)
    assert t2[0, 3:7].tolist() == [1, 3, 0, 2]
    assert p2[0, 3:7].tolist() == [2, 2, 1, 1]
    assert len(set(s2[0, 3:7].tolist())) == 1  # all four children tie
    assert nf[0].tolist() == [3, 4, 5]


def test_validation_codes():
    logits = np.zeros((1, 1, 8), np.float32)
    scores, par, tok, size = _empty_pool(1, 5)
    with pytest.raises(oracle.OracleError) as e:
        oracle.draft_expand(logits, np.array([[0]], np.int32), scores, par, tok, size, W=5, W_next=1)
    assert e.value.code == oracle.STATUS_BAD_NNODES  # 1 + 5 > 5
    with pytest.raises(oracle.OracleError) as e:
        oracle.draft_expand(logits, np.array([[1]], np.int32), scores, par, tok, size, W=2, W_next=1)
    assert e.value.code == oracle.STATUS_BAD_PARENT  # node 1 is not in a pool of size 1
