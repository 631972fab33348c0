"""GPU parity on seeded random shapes: batch size, head counts, group size,
head size, dtype, prefix lengths, tree sizes and shapes, Nmax padding and the
paged block size all drawn per case, so that the work plans (stream and split),
the partition's cuts, the tree block's placement and the paged address paths
meet combinations the fixed workloads do not.  Every node, head and dim of
every sequence is compared with the fp64 oracle (attention), and the accepted
path, tokens and compacted cache bit for bit."""
import numpy as np
import pytest

import gpu_util as U
import workloads as W

pytestmark = pytest.mark.gpu

# the oracle's cost bound per case: query rows x visible keys
_BUDGET = 6_000_000


def _tree(rng, n):
    kind = rng.integers(0, 4)
    if n == 1:
        return np.array([-1], np.int32)
    if kind == 0:
        return W.tree_chain(n)
    if kind == 1:
        return W.tree_star(n)
    return W.tree_uniform_parent(rng, n)


def _case(seed):
    rng = np.random.default_rng(7000 + seed)
    dtype = W.DTYPE_F32 if rng.random() < 0.15 else W.DTYPE_BF16
    d = int(rng.choice([64, 128]))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 4, 8]))
    B = int(rng.integers(1, 7))
    block = int(rng.choice([0, 0, 1, 2, 4, 16, 64, 256]))
    while True:
        ns = [int(rng.choice([1, int(rng.integers(2, 64)), int(rng.integers(64, 257))])) for _ in range(B)]
        ps = [int(rng.choice([0, int(rng.integers(1, 300)), int(rng.integers(300, 6000))])) for _ in range(B)]
        if sum(n * Hkv * G * (p + n) for n, p in zip(ns, ps)) <= _BUDGET:
            break
        B = max(1, B - 1)
    trees = [_tree(rng, n) for n in ns]
    Nmax = min(256, max(ns) + int(rng.integers(0, 3)))  # the ABI takes at most 256 nodes
    Voc = int(rng.choice([257, 3000]))
    toks = [W.distinct_sibling_tokens(rng, t, Voc) for t in trees]
    label = (f"random seed={seed} dtype={dtype} d={d} Hkv={Hkv} G={G} B={B} block={block} "
             f"N={ns} P={ps}")
    return W.make_batch(rng, dtype=dtype, Hq=Hkv * G, Hkv=Hkv, d=d, prefix=ps, trees=trees,
                        tokens=toks, Voc=Voc, p_match=0.7, Nmax=Nmax, block_size=block,
                        cap_slack=int(rng.integers(0, 9)), label=label)


@pytest.mark.parametrize("seed", range(64))
def test_random_shape(seed):
    b = _case(seed)
    U.log(f"[random] {b.label}")
    dev = U.upload(b)
    got = U.gpu_attention(b, dev)
    want = U.oracle_attention(b)
    err = U.compare_attention(b, got, want)
    pred, acc, toks, nacc = U.gpu_accept(b, dev)
    U.check_accept(b, (pred, acc, toks, nacc))
    U.check_compact(b, dev, acc, nacc)
    U.log(f"[random] seed={seed} attention max-abs {err:.3e}")
