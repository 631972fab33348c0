"""GPU parity of candidate token selection: the HIP kernel against the CPU
oracle on the same seeded pools, bit-exact (pool indices, re-indexed parents,
tokens, depths, sizes, and the untouched rows past V)."""
import json

import numpy as np
import pytest

import gpu_util as U
import oracle
import paper_2603_01639_amd as ltd
import test_oracle_select as TS
import workloads as W

pytestmark = pytest.mark.gpu


def _gpu_select(sb, *, optional=True, validate=False, status=None):
    import torch
    i32 = dict(dtype=torch.int32, device="cuda")
    outs = [torch.full((sb.B, sb.Nmax), -1, **i32) for _ in range(4)]
    nn = torch.full((sb.B,), -3, **i32)
    ltd.select_candidates(U.to_dev(sb.scores), U.to_dev(sb.pool_parents), U.to_dev(sb.pool_tokens),
                          U.to_dev(sb.pool_size), U.to_dev(sb.n_select), outs[1], outs[2], nn,
                          selected=outs[0] if optional else None,
                          depth=outs[3] if optional else None, validate=validate, status=status)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs] + [nn.cpu().numpy()]


def _parity(sb, optional=True):
    U.log(f"[select] {sb.label} B={sb.B} Vpool={sb.Vpool} Nmax={sb.Nmax} "
          f"pool={sb.pool_size.tolist()[:6]} V={sb.n_select.tolist()[:6]}")
    got = _gpu_select(sb, optional=optional)
    want = oracle.select_candidates(sb.scores, sb.pool_parents, sb.pool_tokens, sb.pool_size,
                                    sb.n_select, sb.Nmax)
    names = ("selected", "parents", "tokens", "depth")
    for k, name in enumerate(names):
        if not optional and name in ("selected", "depth"):
            assert (got[k] == -1).all(), name
            continue
        np.testing.assert_array_equal(got[k], want[k], err_msg=f"{sb.label}: {name}")
    np.testing.assert_array_equal(got[4], want[4], err_msg=f"{sb.label}: n_nodes")
    return want


def _batch(pars, scs, nsel, *, Vpool=None, Nmax=256, toks=None, label=""):
    S, P, T, sizes = TS._pack(pars, scs, toks, Vpool=Vpool)
    return W.SelectBatch(len(pars), S.shape[1], Nmax, S, P, T, sizes, np.array(nsel, np.int32),
                         label)


def _tied_pool(rng, n, signed_zero=False):
    par = W.tree_uniform_parent(rng, n)
    sc = np.zeros(n, np.float32)
    for i in range(1, n):
        sc[i] = sc[par[i]] - np.float32(rng.choice([0.0, 0.5, 1.0, np.inf], p=[0.3, 0.3, 0.35, 0.05]))
    if signed_zero:
        sc[1:] = np.where(sc[1:] == 0, np.float32(-0.0), sc[1:])
    return par, sc


@pytest.mark.parametrize("rep", range(3))
def test_paper_shaped_pools(rep):
    _parity(W.select_8b(rep))
    _parity(W.select_batch16(rep))
    if rep < 2:
        _parity(W.select_deep(rep))


def test_worked_examples():
    g = json.load(open(TS.GOLDEN))
    par = np.array(g["pool"]["parents"], np.int32)
    sc = np.array([float(x) for x in g["pool"]["scores"]], np.float32)
    tok = np.array(g["pool"]["tokens"], np.int32)
    nsel = [ex["n_select"] for ex in g["examples"]]
    sb = _batch([par] * len(nsel), [sc] * len(nsel), nsel, Nmax=16, toks=[tok] * len(nsel),
                label="worked examples")
    got = _gpu_select(sb)
    for b, ex in enumerate(g["examples"]):
        V = len(ex["selected"])
        assert got[4][b] == V, ex["name"]
        assert got[0][b, :V].tolist() == ex["selected"], ex["name"]
        assert got[1][b, :V].tolist() == ex["parents"], ex["name"]
        assert got[2][b, :V].tolist() == ex["tokens"], ex["name"]
        assert got[3][b, :V].tolist() == ex["depth"], ex["name"]
        assert (got[0][b, V:] == -1).all()
    _parity(sb)


@pytest.mark.parametrize("Vpool", [1, 2, 63, 64, 65, 127, 129, 500, 1023, 1024])
def test_ragged_pool_widths_with_heavy_ties(Vpool):
    rng = np.random.default_rng(Vpool)
    pars, scs, nsel = [], [], []
    for k in range(6):
        n = int(rng.integers(1, Vpool + 1)) if k else Vpool
        par, sc = _tied_pool(rng, n, signed_zero=bool(k % 2))
        pars.append(par)
        scs.append(sc)
        nsel.append(int(rng.integers(1, 257)))
    _parity(_batch(pars, scs, nsel, Vpool=Vpool, label=f"ties Vpool={Vpool}"))


def test_extreme_shapes():
    """A 1024-link chain (depth 1023, the longest pointer-jumping run), a
    1024-leaf star, a pool whose scores are all equal (depth and index decide
    everything), V = 1, and V above the pool size."""
    n = W.MAX_POOL
    chain = W.tree_chain(n)
    star = W.tree_star(n)
    rng = np.random.default_rng(9)
    flat_par = W.tree_uniform_parent(rng, n)
    pars = [chain, star, flat_par, flat_par, chain[:5]]
    scs = [-np.arange(n, dtype=np.float32) / 7, np.concatenate([[0], -rng.random(n - 1)]).astype(
        np.float32), np.zeros(n, np.float32), np.zeros(n, np.float32), np.zeros(5, np.float32)]
    _parity(_batch(pars, scs, [256, 256, 256, 1, 200], Vpool=n, label="chain/star/equal/V=1/V>pool"))


def test_optional_outputs_may_be_null():
    _parity(W.select_batch16(1), optional=False)


def test_validation_reports_the_oracles_code_and_writes_nothing():
    import torch
    rng = np.random.default_rng(4)
    good = [_tied_pool(rng, n) for n in (40, 300, 7)]
    base = _batch([g[0] for g in good], [g[1] for g in good], [20, 60, 7], Vpool=320, Nmax=64,
                  label="validation")
    cases = []
    sb = W.SelectBatch(**vars(base)); sb.pool_size = sb.pool_size.copy(); sb.pool_size[2] = 0
    cases.append(("pool_size 0", sb))
    sb = W.SelectBatch(**vars(base)); sb.pool_size = sb.pool_size.copy(); sb.pool_size[1] = 321
    cases.append(("pool_size > Vpool", sb))
    sb = W.SelectBatch(**vars(base)); sb.n_select = sb.n_select.copy(); sb.n_select[0] = 65
    cases.append(("n_select > Nmax", sb))
    sb = W.SelectBatch(**vars(base)); sb.pool_parents = sb.pool_parents.copy()
    sb.pool_parents[1, 17] = 17
    cases.append(("parent not below", sb))
    sb = W.SelectBatch(**vars(base)); sb.pool_parents = sb.pool_parents.copy()
    sb.pool_parents[2, 0] = 0
    cases.append(("root with a parent", sb))
    sb = W.SelectBatch(**vars(base)); sb.scores = sb.scores.copy(); sb.scores[1, 200] = np.nan
    cases.append(("NaN score", sb))
    sb = W.SelectBatch(**vars(base)); sb.scores = sb.scores.copy()
    c = 30
    sb.scores[0, c] = sb.scores[0, base.pool_parents[0, c]] + 1.0
    cases.append(("child above parent", sb))
    sb = W.SelectBatch(**vars(base)); sb.scores = sb.scores.copy(); sb.scores[0, 38] = np.nan
    sb.pool_parents = sb.pool_parents.copy(); sb.pool_parents[2, 3] = -4
    cases.append(("lowest sequence wins", sb))
    for name, sb in cases:
        U.log(f"[select] validation: {name}")
        try:
            oracle.select_candidates(sb.scores, sb.pool_parents, sb.pool_tokens, sb.pool_size,
                                     sb.n_select, sb.Nmax)
            want = 0
        except oracle.OracleError as e:
            want = e.code
        assert want != 0, name
        st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        got = _gpu_select(sb, validate=True, status=st)
        assert int(st.item()) == want, name
        assert all((g == -1).all() for g in got[:4]) and (got[4] == -3).all(), name
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    got = _gpu_select(base, validate=True, status=st)
    assert int(st.item()) == 0
    _parity(base)


def test_selected_tree_feeds_verification():
    """Selection writes the tree straight into the verification inputs on the
    device; attention, acceptance and compaction over it match the oracle run
    on the oracle's own selection of the same pools."""
    import torch
    rng = W.rng_for(77)
    pools = [W.draft_pool(rng, D, 10, 5000) for D in (6, 4, 8, 2)]
    nsel = [60, 100, 140, 20]
    sb = W.make_select_batch(pools, nsel, Nmax=160, label="select->verify")
    sel = oracle.select_candidates(sb.scores, sb.pool_parents, sb.pool_tokens, sb.pool_size,
                                   sb.n_select, sb.Nmax)
    trees = [sel[1][b, :sel[4][b]] for b in range(sb.B)]
    toks = [sel[2][b, :sel[4][b]] for b in range(sb.B)]
    batch = W.make_batch(rng, dtype=W.DTYPE_BF16, Hq=8, Hkv=2, d=128, prefix=[300, 0, 1000, 65],
                         trees=trees, tokens=toks, Voc=5000, p_match=0.7, Nmax=sb.Nmax,
                         label="select->verify")
    U.log(f"[select] {batch.label} n_nodes={batch.n_nodes.tolist()}")
    dev = U.upload(batch)
    dev.parents.fill_(-1)
    dev.tokens.fill_(0)
    dev.n_nodes.fill_(0)
    ltd.select_candidates(U.to_dev(sb.scores), U.to_dev(sb.pool_parents), U.to_dev(sb.pool_tokens),
                          U.to_dev(sb.pool_size), U.to_dev(sb.n_select), dev.parents, dev.tokens,
                          dev.n_nodes)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(U.to_host(dev.parents), batch.parents)
    np.testing.assert_array_equal(U.to_host(dev.tokens), batch.draft_tokens)
    got = U.gpu_attention(batch, dev)
    U.compare_attention(batch, got, U.oracle_attention(batch))
    pred, acc, toks_out, nacc = U.gpu_accept(batch, dev)
    U.check_accept(batch, (pred, acc, toks_out, nacc))
    U.check_compact(batch, dev, acc, nacc)
