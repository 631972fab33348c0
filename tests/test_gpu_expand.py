"""GPU parity of one round of draft tree expansion against the oracle.

Children (parents, tokens) are decided on the float32 logits alone and must
match exactly.  Child scores: the kernel sums exp() in float32 over chunks of
4096 (relative error a few 1e-7 per chunk, merged in double), so its
log-sum-exp is within 1e-5 of the oracle's double one; with the float32
rounding of the result a score may differ by 2e-5 + 2^-23 |score|.  The next
frontier must match exactly wherever the oracle's W_next-th and next-best
child differ by more than twice that; a near-tie may pick either."""
import numpy as np
import pytest

import gpu_util as U
import oracle
import paper_2603_01639_amd as ltd
import workloads as W
import test_oracle_expand as TE

pytestmark = pytest.mark.gpu


def _tol(s):
    return 2e-5 + np.abs(s) * 2.0 ** -23


def _gpu_round(logits, frontier, pool, W_, W_next, validate=False, status=None):
    import torch
    scores, par, tok, size = (U.to_dev(a) for a in pool)
    nf = torch.full((logits.shape[0], W_next), -1, dtype=torch.int32, device="cuda")
    ltd.draft_expand(U.to_dev(logits), U.to_dev(frontier), scores, par, tok, size, nf, W=W_,
                     validate=validate, status=status)
    torch.cuda.synchronize()
    return tuple(U.to_host(x) for x in (scores, par, tok, size, nf))


def _compare(got, want, first, label):
    gs, gp, gt, gn, gf = got
    ws, wp, wt, wn, wf = want
    np.testing.assert_array_equal(gn, wn, err_msg=label)
    B = gs.shape[0]
    for b in range(B):
        sl = slice(first[b], wn[b])
        np.testing.assert_array_equal(gp[b, sl], wp[b, sl], err_msg=f"{label} parents b={b}")
        np.testing.assert_array_equal(gt[b, sl], wt[b, sl], err_msg=f"{label} tokens b={b}")
        assert (np.abs(gs[b, sl] - ws[b, sl]) <= _tol(ws[b, sl])).all(), f"{label} scores b={b}"
        # untouched before the new children
        np.testing.assert_array_equal(gp[b, :first[b]], wp[b, :first[b]])
        children = np.sort(ws[b, sl])[::-1]
        k = gf.shape[1]
        margin = children[k - 1] - children[k] if k < len(children) else np.inf
        if margin > 2 * _tol(children[k - 1]):
            np.testing.assert_array_equal(gf[b], wf[b], err_msg=f"{label} frontier b={b}")
        else:
            assert set(gf[b].tolist()) <= set(range(first[b], wn[b]))


def test_replays_the_generators_beam_on_the_gpu():
    """Rounds of width 10 to depth 6 over a 4000-token vocabulary, each round
    on the GPU and in the oracle from the same start."""
    for depth, width, vocab in ((6, 10, 4000), (4, 4, 50), (12, 5, 300)):
        pool = W.draft_pool(W.rng_for(depth * 100 + width), depth, width, vocab)
        n = len(pool.parents)
        start = TE._empty_pool(1, n)
        start[2][0, 0] = pool.tokens[0]
        gpu_state, cpu_state = start, start
        gf = cf = np.zeros((1, 1), np.int32)
        k = 0
        for rnd in range(depth - 1):
            F = cf.shape[1]
            rows = np.stack([TE._row_for(pool.draws[k + f], vocab) for f in range(F)])[None]
            k += F
            U.log(f"[expand] replay D={depth} W={width} round {rnd} F={F}")
            first = cpu_state[3].copy()
            got = _gpu_round(rows, gf, gpu_state, width, width)
            want = oracle.draft_expand(rows, cf, *cpu_state, W=width, W_next=width)
            _compare(got, want, first, f"replay D{depth} round {rnd}")
            gpu_state, cpu_state = got[:4], want[:4]
            gf, cf = got[4], want[4]
        np.testing.assert_array_equal(gpu_state[1][0], pool.parents)
        np.testing.assert_array_equal(gpu_state[2][0], pool.tokens)


@pytest.mark.parametrize("B,F,Voc,Wd,W_next", [
    (1, 1, 128256, 10, 10), (1, 10, 128256, 10, 10), (4, 10, 152064, 10, 10), (2, 3, 4097, 4, 7),
    (3, 16, 262144, 16, 16), (2, 1, 16, 16, 5), (1, 5, 10, 1, 3), (2, 7, 4095, 3, 21),
    (2, 40, 5000, 4, 12), (1, 256, 100, 1, 64)])
def test_random_logits(B, F, Voc, Wd, W_next):
    rng = np.random.default_rng(Voc + F * 100 + Wd)
    logits = (rng.standard_normal((B, F, Voc)) * 2).astype(np.float32)
    Vpool = max(30, F + 1) + F * Wd + 5
    scores = (-rng.random((B, Vpool)) * 10).astype(np.float32)
    par = rng.integers(-1, 5, size=(B, Vpool)).astype(np.int32)
    tok = rng.integers(0, 100, size=(B, Vpool)).astype(np.int32)
    size = rng.integers(F, max(31, F + 2), size=B).astype(np.int32)
    frontier = np.stack([rng.choice(size[b], F, replace=False) for b in range(B)]).astype(np.int32)
    U.log(f"[expand] random B={B} F={F} Voc={Voc} W={Wd} W_next={W_next}")
    pool = (scores, par, tok, size)
    got = _gpu_round(logits, frontier, pool, Wd, W_next)
    want = oracle.draft_expand(logits, frontier, *pool, W=Wd, W_next=W_next)
    _compare(got, want, size, f"random Voc={Voc}")


def test_tied_logits():
    """Integer logits with many equal values: the lower token index wins, in
    every chunk and across chunks."""
    rng = np.random.default_rng(7)
    B, F, Voc = 2, 4, 20000
    logits = rng.integers(-3, 3, size=(B, F, Voc)).astype(np.float32)
    logits[0, 0, :] = 1.0  # one row entirely tied
    pool = TE._empty_pool(B, 64)
    pool[3][:] = 5
    frontier = np.array([[0, 1, 2, 3], [4, 2, 0, 1]], np.int32)
    U.log("[expand] tied logits")
    got = _gpu_round(logits, frontier, pool, 10, 10)
    want = oracle.draft_expand(logits, frontier, *pool, W=10, W_next=10)
    _compare(got, want, pool[3], "ties")
    assert got[2][0, 5:15].tolist() == list(range(10))


def test_crowded_thresholds():
    """Rows built so that many keys pass the selection thresholds: in node 0,
    ten runs of four consecutive tokens in every 1024-token block of the first
    4096-token chunk carry large, nearly equal values (so whole runs sit just
    above the chunk's threshold); in node 1 the ten largest values of each of
    the first ten chunks are all larger than the tenth-largest chunk maximum.
    Both are exact against the oracle."""
    rng = np.random.default_rng(17)
    B, F, Voc, W = 1, 2, 50000, 10
    logits = rng.standard_normal((B, F, Voc)).astype(np.float32)
    for t in range(10):
        for j in range(4):
            for e in range(4):
                logits[0, 0, j * 1024 + t * 4 + e] = 100 + t * 0.01 + (j * 4 + e) * 1e-4
    for c in range(10):
        pos = c * 4096 + rng.choice(4096, 10, replace=False)
        logits[0, 1, pos] = 50 + c * 0.01 + np.arange(10) * 1e-4
    pool = TE._empty_pool(B, 64)
    pool[3][:] = 5
    frontier = np.array([[0, 3]], np.int32)
    U.log("[expand] crowded thresholds")
    got = _gpu_round(logits, frontier, pool, W, W)
    want = oracle.draft_expand(logits, frontier, *pool, W=W, W_next=W)
    _compare(got, want, pool[3], "crowded")


def test_validation():
    import torch
    logits = np.zeros((2, 2, 100), np.float32)
    pool = TE._empty_pool(2, 12)
    pool[3][:] = [3, 3]
    for label, frontier, size, code in (
            ("overflow", [[0, 1], [0, 1]], [3, 5], oracle.STATUS_BAD_NNODES),
            ("frontier outside", [[0, 3], [0, 1]], [3, 3], oracle.STATUS_BAD_PARENT),
            ("empty pool", [[0, 1], [0, 1]], [0, 3], oracle.STATUS_BAD_NNODES)):
        frontier = np.array(frontier, np.int32)
        p = (pool[0], pool[1], pool[2], np.array(size, np.int32))
        with pytest.raises(oracle.OracleError) as e:
            oracle.draft_expand(logits, frontier, *p, W=4, W_next=2)
        assert e.value.code == code
        U.log(f"[expand] validation {label}")
        st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        got = _gpu_round(logits, frontier, p, 4, 2, validate=True, status=st)
        assert int(st.item()) == code, label
        np.testing.assert_array_equal(got[3], p[3])  # nothing written
        assert (got[4] == -1).all()
