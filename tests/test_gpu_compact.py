"""GPU parity of KV compaction over several layers (the candidates after the
first mismatch are discarded, section 3.2, "Draft Tree Verification").

Each case stacks num_layers copies of the single-layer cache layout
layer_stride_elems elements apart, with a gap between layers that no layer's
rows reach (spare sequences in the contiguous layout, spare blocks no block
table names in the paged one).  The GPU result must equal the oracle's on every
byte of the buffer: the moved rows of every layer, the rows left alone and the
gaps between layers."""
import numpy as np
import pytest

import gpu_util as U
import oracle
import paper_2603_01639_amd as ltd
import workloads as W

pytestmark = pytest.mark.gpu


def _root_path(parents, leaf):
    path = []
    j = leaf
    while j >= 0:
        path.append(int(j))
        j = int(parents[j])
    return path[::-1]


def _case(rng, *, B, Hkv, d, dtype, layers, block_size, hazard=False):
    ns = [int(rng.integers(2, 60)) for _ in range(B)]
    prefix = [int(rng.integers(0, 300)) for _ in range(B)]
    trees = [W.tree_uniform_parent(rng, n) for n in ns]
    Nmax = max(ns)
    acc = np.full((B, Nmax), -1, np.int32)
    nacc = np.zeros(B, np.int32)
    for b in range(B):
        path = _root_path(trees[b], int(rng.integers(0, ns[b])))
        if hazard and b == 0 and ns[0] >= 7:
            path = [0, 1, 3, 6]  # row P+3 is read for j = 2 and written for j = 3
        acc[b, :len(path)] = path
        nacc[b] = len(path)
    np_dt = np.float32 if dtype == W.DTYPE_F32 else np.uint16

    def fill(shape):
        if dtype == W.DTYPE_F32:
            return rng.standard_normal(size=shape, dtype=np.float32)
        return rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)

    if block_size:
        per = [-(-(prefix[b] + ns[b]) // block_size) for b in range(B)]
        used = sum(per)
        spare = 3  # blocks no table names: the gap after each layer
        nblk = used + spare
        perm = rng.permutation(used).astype(np.int32)
        table = np.zeros((B, max(per)), np.int32)
        pos = 0
        for b in range(B):
            table[b, :per[b]] = perm[pos:pos + per[b]]
            pos += per[b]
        shape = (layers, nblk, Hkv, block_size, d)
        num_blocks = used
    else:
        cap = max(prefix[b] + ns[b] for b in range(B)) + 4
        shape = (layers, B + 2, Hkv, cap, d)  # two spare sequences per layer: the gap
        table, num_blocks = None, 0
    k, v = fill(shape).astype(np_dt), fill(shape).astype(np_dt)
    stride = int(np.prod(shape[1:]))
    return dict(k=k, v=v, prefix=np.array(prefix, np.int32), acc=acc, nacc=nacc, table=table,
                num_blocks=num_blocks, Hkv=Hkv, layers=layers, stride=stride, B=B)


@pytest.mark.parametrize("layers", [2, 4])
@pytest.mark.parametrize("block_size", [0, 16])
@pytest.mark.parametrize("dtype", [W.DTYPE_BF16, W.DTYPE_F32])
def test_multilayer_compaction_bit_exact(layers, block_size, dtype):
    import torch
    rng = np.random.default_rng(1000 * layers + 10 * block_size + dtype)
    c = _case(rng, B=5, Hkv=8, d=128 if dtype == W.DTYPE_BF16 else 64, dtype=dtype,
              layers=layers, block_size=block_size, hazard=True)
    U.log(f"[compact] layers={layers} block={block_size} dtype={dtype} paths={c['nacc'].tolist()}")
    B = c["B"]
    # the device views: [layers][...][Hkv][rows][d] in the library's layout
    dk, dv = U.to_dev(c["k"]), U.to_dev(c["v"])
    new_len = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    ltd.kv_compact(dk, dv, U.to_dev(c["prefix"]), new_len, U.to_dev(c["acc"]), U.to_dev(c["nacc"]),
                   block_table=U.to_dev(c["table"]), num_blocks=c["num_blocks"],
                   num_layers=layers, layer_stride_elems=c["stride"])
    torch.cuda.synchronize()
    k, v = c["k"].copy(), c["v"].copy()
    want_len = oracle.kv_compact(k, v, c["prefix"], c["acc"], c["nacc"], Hkv=c["Hkv"],
                                 block_table=c["table"], num_blocks=c["num_blocks"],
                                 num_layers=layers, layer_stride_elems=c["stride"])
    np.testing.assert_array_equal(new_len.cpu().numpy(), want_len)
    assert not np.array_equal(k, c["k"])  # something moved
    np.testing.assert_array_equal(U.to_host(dk), k)
    np.testing.assert_array_equal(U.to_host(dv), v)


def test_multilayer_compaction_validation_stops_every_layer():
    """A bad path stops the whole call: no layer is touched."""
    import torch
    rng = np.random.default_rng(77)
    c = _case(rng, B=3, Hkv=2, d=64, dtype=W.DTYPE_F32, layers=3, block_size=16)
    c["acc"][1, 1] = 0  # not strictly increasing
    c["nacc"][1] = max(2, int(c["nacc"][1]))
    dk, dv = U.to_dev(c["k"]), U.to_dev(c["v"])
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    new_len = torch.full((c["B"],), -7, dtype=torch.int32, device="cuda")
    ltd.kv_compact(dk, dv, U.to_dev(c["prefix"]), new_len, U.to_dev(c["acc"]), U.to_dev(c["nacc"]),
                   block_table=U.to_dev(c["table"]), num_blocks=c["num_blocks"], num_layers=3,
                   layer_stride_elems=c["stride"], validate=True, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == ltd.STATUS_BAD_PATH
    assert (new_len.cpu().numpy() == -7).all()
    np.testing.assert_array_equal(U.to_host(dk), c["k"])
    np.testing.assert_array_equal(U.to_host(dv), c["v"])
