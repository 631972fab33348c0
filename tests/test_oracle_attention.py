"""Pins for the oracle's tree attention (CPU only).

The oracle is checked against what the paper fixes, never against itself:
* brute force: every node equals causal attention over prefix + its root path
  (the tree attention mask of section 3.2), exhaustively over all trees with
  N <= 6 and on random trees up to N = 32;
* a library routine: torch's scaled_dot_product_attention in fp64 with the
  ancestor mask built as a transitive closure;
* special cases: a chain tree is causal decoding of N new tokens, N = 1 is
  single-token decode, a star tree sees prefix + root + itself;
* invariants: prefix row permutation, a common shift of all keys, and
  relabelling the tree in another topological order.
"""
import numpy as np
import pytest
import torch

import oracle
from brute import all_parent_arrays, ancestor_mask_closure, attention_by_root_path
import workloads as W

F32 = oracle.DTYPE_F32
BF16 = oracle.DTYPE_BF16


def _case(rng, parents, P, Hq=4, Hkv=2, d=8, dtype=F32, slack=3):
    """One-sequence inputs; returns (q, kc, vc, logical k rows, logical v rows)."""
    N = len(parents)
    cap = P + N + slack
    q = rng.standard_normal((1, N, Hq, d), dtype=np.float32)
    kc = rng.standard_normal((1, Hkv, cap, d), dtype=np.float32)
    vc = rng.standard_normal((1, Hkv, cap, d), dtype=np.float32)
    if dtype == BF16:
        q, kc, vc = (W.f32_to_bf16_bits(a) for a in (q, kc, vc))
        qf, kf, vf = (W.bf16_bits_to_f32(a) for a in (q, kc, vc))
    else:
        qf, kf, vf = q, kc, vc
    return q, kc, vc, qf, kf, vf


def _run_oracle(q, kc, vc, P, parents, Hkv, dtype=F32, scale=None):
    N = len(parents)
    return oracle.tree_verify_attn(q, kc, vc, np.array([P], np.int32), np.array([parents], np.int32),
                                   np.array([N], np.int32), Hkv=Hkv, dtype=dtype, scale=scale)[0]


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 6])
def test_every_tree_up_to_6_nodes_matches_root_path_attention(n):
    rng = np.random.default_rng(100 + n)
    for parents in all_parent_arrays(n):
        P = int(rng.integers(0, 6))
        q, kc, vc, qf, kf, vf = _case(rng, parents, P)
        got = _run_oracle(q, kc, vc, P, parents, Hkv=2)
        want = attention_by_root_path(qf[0], kf[0], vf[0], P, parents, 1 / np.sqrt(8))
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_random_trees_up_to_32_nodes(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(7, 33))
    parents = W.tree_uniform_parent(rng, N)
    P = int(rng.integers(0, 40))
    Hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 4]))
    d = int(rng.choice([8, 16, 64]))
    dtype = [F32, BF16][seed % 2]
    q, kc, vc, qf, kf, vf = _case(rng, parents, P, Hq=Hkv * G, Hkv=Hkv, d=d, dtype=dtype)
    got = _run_oracle(q, kc, vc, P, parents, Hkv=Hkv, dtype=dtype)
    want = attention_by_root_path(qf[0], kf[0], vf[0], P, parents, 1 / np.sqrt(d))
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def _sdpa(qf, kf, vf, P, mask_tree, Hkv, scale):
    """torch SDPA (fp64, CPU) with mask [N][P+N] = [all prefix | tree mask]."""
    N, Hq, d = qf.shape
    G = Hq // Hkv
    rows = P + N
    mask = torch.zeros((N, rows), dtype=torch.bool)
    mask[:, :P] = True
    mask[:, P:] = torch.from_numpy(mask_tree)
    qt = torch.from_numpy(qf.astype(np.float64)).permute(1, 0, 2)  # [Hq][N][d]
    kt = torch.from_numpy(kf[:, :rows].astype(np.float64)).repeat_interleave(G, 0).contiguous()
    vt = torch.from_numpy(vf[:, :rows].astype(np.float64)).repeat_interleave(G, 0).contiguous()
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("seed", range(4))
def test_matches_library_sdpa_with_closure_mask(seed):
    rng = np.random.default_rng(50 + seed)
    N = [5, 17, 32, 60][seed]
    parents = W.tree_uniform_parent(rng, N)
    P = [0, 3, 33, 100][seed]
    q, kc, vc, qf, kf, vf = _case(rng, parents, P, Hq=8, Hkv=2, d=16)
    scale = 0.3 + 0.1 * seed
    got = _run_oracle(q, kc, vc, P, parents, Hkv=2, scale=scale)
    want = _sdpa(qf[0], kf[0], vf[0], P, ancestor_mask_closure(parents), 2, scale)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_chain_tree_is_causal_decoding():
    rng = np.random.default_rng(7)
    N, P = 12, 20
    parents = W.tree_chain(N)
    q, kc, vc, qf, kf, vf = _case(rng, parents, P, Hq=4, Hkv=4, d=16)
    got = _run_oracle(q, kc, vc, P, parents, Hkv=4)
    causal = np.tril(np.ones((N, N), dtype=bool))
    want = _sdpa(qf[0], kf[0], vf[0], P, causal, 4, 1 / 4.0)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_single_node_is_decode_attention():
    rng = np.random.default_rng(8)
    P = 37
    q, kc, vc, qf, kf, vf = _case(rng, [-1], P, Hq=8, Hkv=2, d=32)
    got = _run_oracle(q, kc, vc, P, [-1], Hkv=2)
    for h in range(8):
        k = kf[0, h // 4, :P + 1].astype(np.float64)
        v = vf[0, h // 4, :P + 1].astype(np.float64)
        s = k @ qf[0, 0, h].astype(np.float64) / np.sqrt(32)
        w = np.exp(s - s.max())
        np.testing.assert_allclose(got[0, h], (w @ v) / w.sum(), rtol=0, atol=1e-12)


def test_star_tree_sees_prefix_root_and_itself():
    rng = np.random.default_rng(9)
    N, P = 9, 10
    parents = W.tree_star(N)
    q, kc, vc, qf, kf, vf = _case(rng, parents, P, Hq=2, Hkv=1, d=8)
    got = _run_oracle(q, kc, vc, P, parents, Hkv=1)
    mask = np.zeros((N, N), bool)
    mask[:, 0] = True
    mask[np.arange(N), np.arange(N)] = True
    want = _sdpa(qf[0], kf[0], vf[0], P, mask, 1, 1 / np.sqrt(8))
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_invariant_prefix_row_permutation():
    rng = np.random.default_rng(10)
    parents = W.tree_uniform_parent(rng, 14)
    P = 25
    q, kc, vc, *_ = _case(rng, parents, P, Hq=4, Hkv=2, d=8)
    base = _run_oracle(q, kc, vc, P, parents, Hkv=2)
    perm = rng.permutation(P)
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[:, :, :P] = kc[:, :, perm]
    vc2[:, :, :P] = vc[:, :, perm]
    got = _run_oracle(q, kc2, vc2, P, parents, Hkv=2)
    np.testing.assert_allclose(got, base, rtol=0, atol=1e-12)


def test_invariant_common_key_shift():
    """Adding one vector c to every key adds <q, c> to every score of a query:
    softmax is unchanged."""
    rng = np.random.default_rng(11)
    parents = W.tree_uniform_parent(rng, 10)
    P = 8
    q, kc, vc, *_ = _case(rng, parents, P, Hq=2, Hkv=2, d=8)
    kc = np.round(kc * 1024) / 1024  # 2^-10 grid: the shifted keys stay exact in float32
    base = _run_oracle(q, kc, vc, P, parents, Hkv=2)
    c = (rng.integers(-4, 5, size=(1, 2, 1, 8)) * 0.25).astype(np.float32)
    got = _run_oracle(q, kc + c, vc, P, parents, Hkv=2)
    np.testing.assert_allclose(got, base, rtol=0, atol=1e-12)


def test_invariant_topological_relabelling():
    """Renumbering the tree by another topological order (moving each node's
    query and tree K/V row with it) permutes the output rows the same way."""
    rng = np.random.default_rng(12)
    N, P = 15, 6
    parents = W.tree_uniform_parent(rng, N)
    q, kc, vc, *_ = _case(rng, parents, P, Hq=4, Hkv=2, d=8, slack=0)
    base = _run_oracle(q, kc, vc, P, parents, Hkv=2)
    # random topological order: repeatedly pick a random node whose parent is placed
    placed, order = {0}, [0]
    while len(order) < N:
        ready = [i for i in range(N) if i not in placed and parents[i] in placed]
        pick = ready[rng.integers(0, len(ready))]
        placed.add(pick)
        order.append(pick)
    new_of = {old: new for new, old in enumerate(order)}
    par2 = np.array([-1] + [new_of[parents[old]] for old in order[1:]], np.int32)
    q2 = q[:, order]
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[:, :, P:P + N] = kc[:, :, P + np.array(order)]
    vc2[:, :, P:P + N] = vc[:, :, P + np.array(order)]
    got = _run_oracle(q2, kc2, vc2, P, par2, Hkv=2)
    np.testing.assert_allclose(got, base[order], rtol=0, atol=1e-12)


def test_paged_layout_equals_contiguous():
    """The same logical rows stored in shuffled 4-row blocks give the same result."""
    rng = np.random.default_rng(13)
    B, Hkv, d, bs = 3, 2, 8, 4
    prefix = [5, 0, 13]
    trees = [W.tree_uniform_parent(rng, n) for n in (7, 3, 11)]
    Nmax = 11
    cap = 24
    q = rng.standard_normal((B, Nmax, 4, d), dtype=np.float32)
    kc = rng.standard_normal((B, Hkv, cap, d), dtype=np.float32)
    vc = rng.standard_normal((B, Hkv, cap, d), dtype=np.float32)
    parents = np.full((B, Nmax), -1, np.int32)
    for b, t in enumerate(trees):
        parents[b, :len(t)] = t
    n_nodes = np.array([len(t) for t in trees], np.int32)
    pl = np.array(prefix, np.int32)
    base = oracle.tree_verify_attn(q, kc, vc, pl, parents, n_nodes, Hkv=Hkv, dtype=F32)
    nblk_per = cap // bs
    num_blocks = B * nblk_per + 5
    perm = rng.permutation(num_blocks)[:B * nblk_per].reshape(B, nblk_per).astype(np.int32)
    kp = rng.standard_normal((num_blocks, Hkv, bs, d), dtype=np.float32)
    vp = rng.standard_normal((num_blocks, Hkv, bs, d), dtype=np.float32)
    for b in range(B):
        for j in range(nblk_per):
            kp[perm[b, j]] = kc[b, :, j * bs:(j + 1) * bs]
            vp[perm[b, j]] = vc[b, :, j * bs:(j + 1) * bs]
    got = oracle.tree_verify_attn(q, kp, vp, pl, parents, n_nodes, Hkv=Hkv, block_table=perm,
                                  num_blocks=num_blocks, dtype=F32)
    np.testing.assert_array_equal(got, base)
    # padded rows (i >= n_nodes[b]) are left untouched (zeros)
    assert not got[1, 3:].any()


def test_bad_inputs_are_rejected():
    rng = np.random.default_rng(14)
    parents = np.array([-1, 0, 2], np.int32)  # parent of node 2 is itself
    q, kc, vc, *_ = _case(rng, [-1, 0, 1], 4)
    with pytest.raises(oracle.OracleError) as e:
        _run_oracle(q, kc, vc, 4, parents, Hkv=2)
    assert e.value.code == oracle.STATUS_BAD_PARENT
    with pytest.raises(oracle.OracleError) as e:
        _run_oracle(q, kc, vc, 8, [-1, 0, 1], Hkv=2)  # 8 + 3 > cap 10
    assert e.value.code == oracle.STATUS_BAD_PREFIX
