"""GPU parity: the HIP library against the CPU oracle on the same seeded
inputs.  Attention within max-abs 1e-5 (fp32) / 2e-2 (bf16); argmax, accepted
path, emitted tokens, count and the compacted cache bit-exact."""
import numpy as np
import pytest

import gpu_util as U
import paper_2603_01639_amd as ltd
import partition_cases as PC
import workloads as W

pytestmark = pytest.mark.gpu


def _full_step(b):
    """attention + acceptance + compaction on the GPU vs the oracle, every
    node and head of every sequence compared."""
    U.log(f"[parity] {b.label} B={b.B} Nmax={b.Nmax} P={b.prefix_len.tolist()[:4]}")
    dev = U.upload(b)
    got = U.gpu_attention(b, dev)
    want = U.oracle_attention(b)
    err = U.compare_attention(b, got, want)
    U.log(f"[parity] {b.label} attention max-abs {err:.3e}")
    if b.logits is not None:
        pred, acc, toks, nacc = U.gpu_accept(b, dev)
        U.check_accept(b, (pred, acc, toks, nacc))
        U.check_compact(b, dev, acc, nacc)
        U.log(f"[parity] {b.label} accept/compact exact, n_accepted={nacc.tolist()[:8]}")
    return err


@pytest.mark.parametrize("rep", range(5))
def test_config1_tiny_f32(rep):
    _full_step(W.config1_tiny_f32(rep))


@pytest.mark.parametrize("rep", range(5))
def test_config2_8b_bf16(rep):
    _full_step(W.config2_8b(rep))


@pytest.mark.parametrize("rep", range(5))
def test_config3_long_prefix(rep):
    _full_step(W.config3_long(rep))


def _c4_depths(n):
    """Depth 2, a middle depth and depth 10 (or the deepest tree N nodes
    allow), the span the depth policy moves over."""
    return sorted({2, min(6, n), min(10, n)})


@pytest.mark.parametrize("n,depth", [(n, d) for n in W.C4_SIZES for d in _c4_depths(n)])
def test_config4_sweep(n, depth):
    _full_step(W.config4_sweep(n, depth))


@pytest.mark.parametrize("rep", range(5))
def test_config5_paged_batch(rep):
    _full_step(W.config5_paged(rep))


@pytest.mark.parametrize("rep", range(3))
def test_config5_tp8_share(rep):
    """One GPU's share of c5 under 8-way tensor parallelism (one kv head, 8 q
    heads per sequence): every node and head against the oracle."""
    _full_step(W.config5_tp_share(rep, 8))


def test_config5_deterministic():
    """Two runs of the batched paged step give bit-identical outputs: the
    split merge order is fixed, whatever order the workgroups finish in."""
    b = W.config5_paged(1, with_logits=True)
    U.log(f"[parity] determinism {b.label}")
    dev = U.upload(b)
    a1 = U.gpu_attention(b, dev)
    a2 = U.gpu_attention(b, dev, fill=3.0)  # a different fill: every written row is rewritten
    for s in range(b.B):
        n = int(b.n_nodes[s])
        np.testing.assert_array_equal(a1[s, :n], a2[s, :n])
        assert (U.as_f64(a2[s, n:], b.dtype) == 3.0).all()
    r1 = U.gpu_accept(b, dev)
    r2 = U.gpu_accept(b, dev)
    for x, y in zip(r1, r2):
        np.testing.assert_array_equal(x, y)


# ----------------------------------------------------------------- edge cases

def _custom(trees, prefix, *, Hq=8, Hkv=2, d=128, dtype=W.DTYPE_BF16, Nmax=None, Voc=3000,
            block_size=0, seed=0, p_match=0.7, label="custom"):
    rng = W.rng_for(seed)
    toks = [W.distinct_sibling_tokens(rng, t, Voc) for t in trees]
    return W.make_batch(rng, dtype=dtype, Hq=Hq, Hkv=Hkv, d=d, prefix=prefix, trees=trees,
                        tokens=toks, Voc=Voc, p_match=p_match, Nmax=Nmax, block_size=block_size,
                        cap_slack=5, label=label)


@pytest.mark.parametrize("P", [0, 1, 5, 63, 64, 65, 1000, 2047, 2049])
def test_ragged_prefix_lengths(P):
    rng = np.random.default_rng(P)
    _full_step(_custom([W.tree_uniform_parent(rng, 37)], [P], seed=P, label=f"ragged P={P}"))


def test_single_node_tree_is_decode():
    _full_step(_custom([np.array([-1], np.int32)], [300], label="N=1"))


def test_max_nodes_chain_and_star():
    _full_step(_custom([W.tree_chain(256)], [129], Hq=8, Hkv=8, label="chain N=256"))
    _full_step(_custom([W.tree_star(256)], [77], Hq=16, Hkv=2, label="star N=256"))


def test_padded_rows_untouched_and_mixed_batch():
    rng = np.random.default_rng(3)
    trees = [W.tree_uniform_parent(rng, n) for n in (1, 20, 57, 3)]
    b = _custom(trees, [10, 0, 700, 129], Nmax=64, seed=3, label="mixed batch Nmax=64")
    dev = U.upload(b)
    got = U.gpu_attention(b, dev, fill=7.0)
    filled = U.as_f64(got, b.dtype)
    for s in range(b.B):
        assert (filled[s, b.n_nodes[s]:] == 7.0).all()
    _full_step(b)


@pytest.mark.parametrize("dtype,d,G", [(W.DTYPE_F32, 128, 4), (W.DTYPE_F32, 64, 1),
                                       (W.DTYPE_F32, 64, 8), (W.DTYPE_F32, 128, 6),
                                       (W.DTYPE_BF16, 64, 8), (W.DTYPE_BF16, 128, 1)])
def test_head_dims_dtypes_and_groups(dtype, d, G):
    rng = np.random.default_rng(d + G)
    trees = [W.tree_uniform_parent(rng, 45), W.tree_uniform_parent(rng, 12)]
    _full_step(_custom(trees, [333, 90], Hq=2 * G, Hkv=2, d=d, dtype=dtype, seed=d + G,
                       label=f"dtype={dtype} d={d} G={G}"))


def test_paged_small_blocks_fp32():
    rng = np.random.default_rng(11)
    trees = [W.tree_uniform_parent(rng, n) for n in (9, 30, 2)]
    _full_step(_custom(trees, [40, 100, 3], Hq=4, Hkv=4, d=64, dtype=W.DTYPE_F32, block_size=16,
                       seed=11, label="paged fp32"))


def test_deterministic():
    b = W.config2_8b(7)
    U.log(f"[parity] determinism {b.label}")
    dev = U.upload(b)
    a1 = U.gpu_attention(b, dev)
    a2 = U.gpu_attention(b, dev)
    np.testing.assert_array_equal(a1, a2)
    r1 = U.gpu_accept(b, dev)
    r2 = U.gpu_accept(b, dev)
    for x, y in zip(r1, r2):
        np.testing.assert_array_equal(x, y)


def test_argmax_ties_signed_zero_and_ragged_vocab():
    """Ties -> lowest index, -0.0 == +0.0, vocab not a multiple of 4 or of the
    argmax chunk."""
    for Voc in (5, 1000, 8193, 128257):
        rng = np.random.default_rng(Voc)
        n = 6
        par = W.tree_uniform_parent(rng, n)
        lg = rng.integers(-3, 3, size=(1, n, Voc)).astype(np.float32)
        lg[0, 0, :] = -1.0
        lg[0, 0, Voc // 2] = -0.0
        lg[0, 0, Voc - 1] = 0.0
        b = W.VerifyBatch(dtype=W.DTYPE_F32, B=1, Nmax=n, Hq=1, Hkv=1, d=64, Voc=Voc,
                          q=np.zeros((1, n, 1, 64), np.float32),
                          k_cache=np.zeros((1, 1, n, 64), np.float32),
                          v_cache=np.zeros((1, 1, n, 64), np.float32),
                          prefix_len=np.zeros(1, np.int32), parents=par[None].copy(),
                          n_nodes=np.array([n], np.int32),
                          draft_tokens=rng.integers(0, 3, size=(1, n)).astype(np.int32),
                          logits=lg, label=f"ties Voc={Voc}")
        U.log(f"[parity] {b.label}")
        dev = U.upload(b)
        got = U.gpu_accept(b, dev)
        want = U.check_accept(b, got)
        assert want[0][0, 0] == Voc // 2


@pytest.mark.parametrize("block_size", [0, 16])
@pytest.mark.parametrize("case", PC.CASES, ids=[c.label for c in PC.CASES])
def test_work_partition_cases(case, block_size):
    """Batches whose work partition holds a share that is a tree block alone,
    workgroups with nothing to do, units written whole and units cut into many
    pieces (the host test of the partition checks that these batches cover
    those cases), contiguous and paged."""
    rng = np.random.default_rng(len(case.prefix) * 1000 + case.Nmax + block_size)
    trees = [W.tree_uniform_parent(rng, n) for n in case.nodes]
    b = _custom(trees, list(case.prefix), Hq=case.Hq, Hkv=case.Hkv, Nmax=case.Nmax,
                block_size=block_size, seed=case.Nmax, label=f"{case.label} block={block_size}")
    assert ltd.attn_grid(b.B, b.Nmax, b.Hq, b.Hkv, b.d, b.max_prefix, b.dtype, b.kv_rows,
                         paged=b.paged) > 0
    _full_step(b)


def test_accept_workspace_reused_across_calls():
    """One acceptance workspace serves a sequence of calls with different B,
    Nmax and vocabularies, including a call that validation stops: no call
    depends on what an earlier one left in it."""
    import torch
    rng = np.random.default_rng(23)
    ws = torch.empty(max(ltd.accept_workspace_size(16, 128, 128256),
                         ltd.accept_workspace_size(3, 256, 9000)), dtype=torch.uint8, device="cuda")
    batches = [W.config5_paged(0)]
    for n_list, voc in (((256, 3, 77), 9000), ((60,), 128256), ((5, 200), 8192)):
        trees = [W.tree_uniform_parent(rng, n) for n in n_list]
        batches.append(_custom(trees, [0] * len(trees), Hq=2, Hkv=1, d=64, Voc=voc,
                               seed=len(n_list), label=f"reuse N={n_list} Voc={voc}"))
    batches.append(W.config2_8b(3))
    i32 = dict(dtype=torch.int32, device="cuda")
    for k, b in enumerate(batches):
        dev = U.upload(b)
        if k == 2:
            # validation stops this call: parents[0][5] = 5 is not below 5
            bad = dev.parents.clone()
            bad[0, 5] = 5
            st = torch.full((1,), -1, **i32)
            outs = [torch.full((b.B, b.Nmax), -1, **i32) for _ in range(3)]
            ltd.tree_accept(dev.logits, dev.tokens, bad, dev.n_nodes, *outs,
                            torch.zeros((b.B,), **i32), workspace=ws, validate=True, status=st)
            torch.cuda.synchronize()
            assert int(st.item()) == ltd.STATUS_BAD_PARENT and (outs[0] == -1).all()
        U.log(f"[parity] accept workspace reuse, call {k}: {b.label}")
        pred = torch.full((b.B, b.Nmax), -1, **i32)
        acc = torch.full((b.B, b.Nmax), -1, **i32)
        toks = torch.full((b.B, b.Nmax), -1, **i32)
        nacc = torch.zeros((b.B,), **i32)
        ltd.tree_accept(dev.logits, dev.tokens, dev.parents, dev.n_nodes, pred, acc, toks, nacc,
                        workspace=ws)
        torch.cuda.synchronize()
        U.check_accept(b, (pred.cpu().numpy(), acc.cpu().numpy(), toks.cpu().numpy(),
                           nacc.cpu().numpy()))


def test_batch_of_one_row_blocks_takes_the_split_plan():
    """A batch whose paged blocks are one row each: a stream share could span
    more block ids than the LDS table holds, so the batch runs on the split
    plan (its splits shortened to fit the table)."""
    rng = np.random.default_rng(4242)
    trees = [W.tree_uniform_parent(rng, n) for n in (37, 64)]
    b = _custom(trees, [47000, 30000], Hq=24, Hkv=3, block_size=1, seed=4242,
                label="one-row blocks B=2 P=47000")
    g = ltd.attn_grid(b.B, b.Nmax, b.Hq, b.Hkv, b.d, b.max_prefix, b.dtype, b.kv_rows, paged=True)
    assert g > 0 and g & (g - 1) != 0  # not the stream plan's power-of-two grid
    _full_step(b)


@pytest.mark.parametrize("block_size", [2, 3, 4, 8, 32, 64, 128, 256, 1024])
@pytest.mark.parametrize("B", [1, 3])
def test_paged_block_sizes(block_size, B):
    """Paged caches of many block sizes, one sequence (split plan) and a
    batch (stream plan): powers of two from 4 rows on take every full prefix
    tile's loads from one block per load instruction; 2 and 3 rows (and every
    tree tile or partial tile) address row by row."""
    rng = np.random.default_rng(100 * block_size + B)
    nodes = [41, 7, 130][:B]
    prefix = [1000 + 37 * block_size % 900, 2049, 64][:B]
    trees = [W.tree_uniform_parent(rng, n) for n in nodes]
    _full_step(_custom(trees, prefix, Hq=8, Hkv=2, block_size=block_size, seed=block_size + B,
                       label=f"paged block={block_size} B={B}"))


@pytest.mark.parametrize("rep", range(3))
def test_config2_head_dim_64(rep):
    """Config 2's shape with head_dim 64: the matrix-core kernels over the
    first 64 dims of their 128-dim LDS rows (split plan)."""
    _full_step(W.config2_d64(rep))


@pytest.mark.parametrize("block_size", [0, 3, 4, 16, 256])
def test_head_dim_64_batches(block_size):
    """bf16 head_dim 64 batches on the stream plan, contiguous and paged (row
    by row for 3-row blocks, one block per load instruction from 4 rows on),
    with ragged prefixes and trees, a grouped and an ungrouped head layout."""
    rng = np.random.default_rng(640 + block_size)
    trees = [W.tree_uniform_parent(rng, n) for n in (60, 1, 200, 33)]
    _full_step(_custom(trees, [2049, 5, 700, 64], Hq=16, Hkv=4, d=64, block_size=block_size,
                       seed=640 + block_size, label=f"d64 batch block={block_size}"))
    trees = [W.tree_uniform_parent(rng, n) for n in (17, 90)]
    _full_step(_custom(trees, [1000, 3000], Hq=4, Hkv=4, d=64, block_size=block_size,
                       seed=641 + block_size, label=f"d64 G=1 block={block_size}"))


def _rescaled(b, q_scale, k_fn, label):
    """b with Q multiplied by q_scale (q_scale 0: every element -40) and K
    replaced by k_fn(K), re-rounded to bf16: scores far from the usual range."""
    import dataclasses
    qf = W.bf16_bits_to_f32(b.q)
    qf = np.full_like(qf, np.float32(-40.0)) if q_scale == 0.0 else qf * np.float32(q_scale)
    q = W.f32_to_bf16_bits(qf)
    k = W.f32_to_bf16_bits(k_fn(W.bf16_bits_to_f32(b.k_cache)).astype(np.float32))
    return dataclasses.replace(b, q=q, k_cache=k, label=label)


@pytest.mark.parametrize("paged", [False, True])
def test_extreme_score_magnitudes(paged):
    """Scores near -2e5 (every key far below zero; the scaled scores stay
    within the 1e5 or so where an fp32 exponent argument keeps an absolute
    error under 1e-2) and of std ~ 300 (the reference max moves over many
    tiles): both work plans, against the fp64 oracle."""
    rng = np.random.default_rng(21)
    trees = [W.tree_uniform_parent(rng, n) for n in (40, 7, 64)]
    bs = 16 if paged else 0
    base = _custom(trees, [1500, 300, 2200], Hq=8, Hkv=2, block_size=bs, seed=21, label="extreme")
    one = _custom(trees[:1], [2900], Hq=8, Hkv=2, block_size=bs, seed=22, label="extreme B=1")
    for b in (base, one):
        # q = -40 elementwise, k in [0.5, 1.5] * 40: every score near -2e5
        _full_step(_rescaled(b, 0.0, lambda k: 40.0 * (1.0 + 0.5 * np.tanh(k)), b.label + " -2e5"))
        _full_step(_rescaled(b, 5.0, lambda k: 5.0 * k, b.label + " std 300"))


@pytest.mark.parametrize("paged", [False, True])
def test_long_prefix_65536(paged):
    """One sequence with a 65536-token prefix (the split plan at its longest
    splits and most pieces), contiguous and in 16-token blocks."""
    rng = np.random.default_rng(65536)
    trees = [W.tree_uniform_parent(rng, 48)]
    _full_step(_custom(trees, [65536], Hq=16, Hkv=2, block_size=16 if paged else 0, seed=65,
                       label=f"P=65536 paged={paged}"))


def test_many_sequences():
    """64 sequences of mixed prefixes and tree sizes (the stream plan with
    many short units), in 16-token blocks."""
    rng = np.random.default_rng(64)
    ns = [int(rng.integers(1, 40)) for _ in range(64)]
    ps = [int(rng.integers(0, 1500)) for _ in range(64)]
    trees = [W.tree_uniform_parent(rng, n) if n > 1 else np.array([-1], np.int32) for n in ns]
    _full_step(_custom(trees, ps, Hq=8, Hkv=2, block_size=16, seed=64, label="B=64"))


def test_fp32_unaligned_caches():
    """fp32 K/V caches whose base addresses are 4 but not 16 bytes aligned
    (the kernel's element-wise load path), against the oracle."""
    import torch
    rng = np.random.default_rng(44)
    trees = [W.tree_uniform_parent(rng, n) for n in (23, 5)]
    b = _custom(trees, [200, 77], Hq=8, Hkv=2, d=64, dtype=W.DTYPE_F32, seed=44, label="fp32 unaligned")
    dev = U.upload(b)
    for name in ("k", "v"):
        t = getattr(dev, name)
        buf = torch.empty(t.numel() + 1, dtype=t.dtype, device="cuda")
        view = buf[1:].view(t.shape)
        view.copy_(t)
        assert view.data_ptr() % 16 != 0
        setattr(dev, name, view)
    got = U.gpu_attention(b, dev)
    U.compare_attention(b, got, U.oracle_attention(b))
