"""Error handling of the C ABI.  Malformed calls return LTD_E* codes from the
host; malformed data is reported in the device status word when validation is
on, and then nothing is written.  Every bad input here is caught by a check
before any kernel could read out of bounds."""
import numpy as np
import pytest

import gpu_util as U
import paper_2603_01639_amd as ltd
import workloads as W

pytestmark = pytest.mark.gpu


def _batch(paged=False):
    rng = W.rng_for(77)
    trees = [W.tree_uniform_parent(rng, 9), W.tree_uniform_parent(rng, 5)]
    toks = [W.distinct_sibling_tokens(rng, t, 500) for t in trees]
    return W.make_batch(rng, dtype=W.DTYPE_BF16, Hq=4, Hkv=2, d=64, prefix=[30, 12], trees=trees,
                        tokens=toks, Voc=500, p_match=0.5, block_size=16 if paged else 0,
                        cap_slack=4, label="errors")


def _status():
    import torch
    return torch.full((1,), -99, dtype=torch.int32, device="cuda")


def _attn_status(b, dev):
    st = _status()
    got = U.gpu_attention(b, dev, fill=3.0, validate=True, status=st)
    return int(st.item()), got


def test_valid_data_reports_ok():
    b = _batch()
    U.log("[errors] valid data")
    dev = U.upload(b)
    code, got = _attn_status(b, dev)
    assert code == ltd.STATUS_OK
    U.compare_attention(b, got, U.oracle_attention(b))


def test_bad_parent_reported_and_nothing_written():
    b = _batch()
    b.parents[1, 3] = 3  # a node that is its own parent
    U.log("[errors] bad parent")
    dev = U.upload(b)
    code, got = _attn_status(b, dev)
    assert code == ltd.STATUS_BAD_PARENT
    assert (U.as_f64(got, b.dtype) == 3.0).all()
    st = _status()
    pred, acc, toks, nacc = U.gpu_accept(b, dev, validate=True, status=st)
    assert int(st.item()) == ltd.STATUS_BAD_PARENT and (pred == -1).all() and (nacc == 0).all()


def test_bad_node_count_and_prefix():
    b = _batch()
    b.n_nodes[0] = 0
    dev = U.upload(b)
    U.log("[errors] n_nodes = 0")
    assert _attn_status(b, dev)[0] == ltd.STATUS_BAD_NNODES
    b = _batch()
    b.prefix_len[1] = b.k_cache.shape[2]  # prefix + tree past the capacity
    dev = U.upload(b)
    U.log("[errors] prefix past capacity")
    import torch
    st = _status()
    out = torch.full(tuple(b.q.shape), 3.0, dtype=dev.q.dtype, device="cuda")
    ltd.tree_verify_attn(dev.q, dev.k, dev.v, dev.prefix_len, dev.parents, dev.n_nodes, out,
                         max_prefix=int(b.prefix_len.max()), validate=True, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == ltd.STATUS_BAD_PREFIX
    assert (out.float() == 3.0).all()


def test_prefix_above_declared_max():
    b = _batch()
    dev = U.upload(b)
    import torch
    st = _status()
    out = torch.zeros(tuple(b.q.shape), dtype=dev.q.dtype, device="cuda")
    U.log("[errors] prefix above max_prefix")
    ltd.tree_verify_attn(dev.q, dev.k, dev.v, dev.prefix_len, dev.parents, dev.n_nodes, out,
                         max_prefix=int(b.prefix_len.max()) - 1, validate=True, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == ltd.STATUS_BAD_PREFIX


def test_bad_block_id():
    b = _batch(paged=True)
    b.block_table[1, 0] = b.num_blocks  # one past the pool
    dev = U.upload(b)
    U.log("[errors] bad block id")
    assert _attn_status(b, dev)[0] == ltd.STATUS_BAD_BLOCK


def test_bad_path_leaves_cache_untouched():
    b = _batch()
    dev = U.upload(b)
    acc = np.full((b.B, b.Nmax), -1, np.int32)
    acc[0, :3] = [0, 4, 2]  # not increasing
    acc[1, :1] = [0]
    nacc = np.array([3, 1], np.int32)
    st = _status()
    U.log("[errors] bad path")
    new_len = U.gpu_compact(b, dev, acc, nacc, validate=True, status=st)
    assert int(st.item()) == ltd.STATUS_BAD_PATH
    assert (new_len == -7).all()
    np.testing.assert_array_equal(U.to_host(dev.k), b.k_cache)


def test_host_side_argument_errors():
    import torch
    b = _batch()
    dev = U.upload(b)
    out = torch.zeros(tuple(b.q.shape), dtype=dev.q.dtype, device="cuda")
    U.log("[errors] host-side argument checks")
    with pytest.raises(ltd.LtdError) as e:  # head dim the kernels do not implement
        ltd.tree_verify_attn(dev.q[..., :48].contiguous(), dev.k[..., :48].contiguous(),
                             dev.v[..., :48].contiguous(), dev.prefix_len, dev.parents,
                             dev.n_nodes, out[..., :48].contiguous(), max_prefix=30)
    assert e.value.code == ltd.LTD_EUNSUPPORTED
    with pytest.raises(ltd.LtdError) as e:  # aliasing prefix_len / new_prefix_len
        ltd.kv_compact(dev.k, dev.v, dev.prefix_len, dev.prefix_len,
                       U.to_dev(np.zeros((2, b.Nmax), np.int32)), U.to_dev(np.ones(2, np.int32)))
    assert e.value.code == ltd.LTD_EINVAL
    with pytest.raises(ltd.LtdError) as e:  # workspace too small
        ltd.tree_accept(dev.logits, dev.tokens, dev.parents, dev.n_nodes,
                        *[torch.zeros((2, b.Nmax), dtype=torch.int32, device="cuda")] * 3,
                        torch.zeros(2, dtype=torch.int32, device="cuda"),
                        workspace=torch.zeros(8, dtype=torch.uint8, device="cuda"))
    assert e.value.code == ltd.LTD_EWORKSPACE
