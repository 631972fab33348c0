"""Pins for the oracle's KV compaction (CPU only).

* explicit expected caches built by fancy indexing, including the in-place
  hazard path [0, 1, 3, 6] (destination P+3 is also the source of an earlier
  slot's neighbour: P+3 -> P+2 must be read before P+6 -> P+3 is written);
* after compaction, attention of a fresh query over rows [0, P + n) equals
  attention over the prefix plus the accepted path's rows of the old cache;
* paged and multi-layer layouts move exactly the same logical rows.
"""
import numpy as np
import pytest

import oracle
from brute import softmax_attention_1q


def _expected(kc, P, path):
    want = kc.copy()
    want[:, :, P:P + len(path)] = kc[:, :, [P + j for j in path]]
    return want


@pytest.mark.parametrize("path", [[0], [0, 1, 2], [0, 2, 5], [0, 1, 3, 6], [0, 4, 5, 9, 11]])
def test_contiguous_matches_explicit_gather(path):
    rng = np.random.default_rng(len(path))
    B, Hkv, cap, d, P, Nmax = 1, 3, 40, 8, 17, 12
    kc = rng.standard_normal((B, Hkv, cap, d), dtype=np.float32)
    vc = rng.standard_normal((B, Hkv, cap, d), dtype=np.float32)
    want_k, want_v = _expected(kc, P, path), _expected(vc, P, path)
    acc = np.full((B, Nmax), -1, np.int32)
    acc[0, :len(path)] = path
    new_len = oracle.kv_compact(kc, vc, np.array([P], np.int32), acc, np.array([len(path)], np.int32),
                                Hkv=Hkv)
    assert new_len.tolist() == [P + len(path)]
    np.testing.assert_array_equal(kc, want_k)
    np.testing.assert_array_equal(vc, want_v)


def test_attention_after_compaction_equals_attention_over_path():
    rng = np.random.default_rng(5)
    Hkv, cap, d, P = 2, 64, 16, 30
    path = [0, 1, 4, 9, 10]
    kc = rng.standard_normal((1, Hkv, cap, d), dtype=np.float32)
    vc = rng.standard_normal((1, Hkv, cap, d), dtype=np.float32)
    old_k, old_v = kc.copy(), vc.copy()
    acc = np.array([path + [-1] * 7], np.int32)
    new_len = oracle.kv_compact(kc, vc, np.array([P], np.int32), acc, np.array([5], np.int32), Hkv=Hkv)
    L = int(new_len[0])
    rows = list(range(P)) + [P + j for j in path]
    for g in range(Hkv):
        qv = rng.standard_normal(d)
        a = softmax_attention_1q(qv, kc[0, g, :L], vc[0, g, :L], 0.25)
        b = softmax_attention_1q(qv, old_k[0, g, rows], old_v[0, g, rows], 0.25)
        np.testing.assert_array_equal(a, b)


def test_paged_multilayer_bf16_moves_the_same_rows():
    rng = np.random.default_rng(6)
    B, Hkv, d, bs, layers = 2, 2, 8, 4, 3
    prefix = [6, 9]
    paths = [[0, 2, 3, 7], [0, 1]]
    nblk = 6
    num_blocks = B * nblk + 3
    table = rng.permutation(num_blocks)[:B * nblk].reshape(B, nblk).astype(np.int32)
    per_layer = num_blocks * Hkv * bs * d
    kp = rng.integers(0, 65535, size=(layers, num_blocks, Hkv, bs, d)).astype(np.uint16)
    vp = rng.integers(0, 65535, size=(layers, num_blocks, Hkv, bs, d)).astype(np.uint16)

    def logical(cache, layer, b):  # [Hkv][nblk*bs][d]
        return np.concatenate([cache[layer, table[b, j]] for j in range(nblk)], axis=1)

    want = [[_expected(logical(c, L, b)[None], prefix[b], paths[b])[0] for b in range(B)
             for L in range(layers)] for c in (kp, vp)]
    acc = np.full((B, 8), -1, np.int32)
    for b, p in enumerate(paths):
        acc[b, :len(p)] = p
    new_len = oracle.kv_compact(kp, vp, np.array(prefix, np.int32), acc,
                                np.array([len(p) for p in paths], np.int32), Hkv=Hkv,
                                block_table=table, num_blocks=num_blocks, num_layers=layers,
                                layer_stride_elems=per_layer)
    assert new_len.tolist() == [prefix[b] + len(paths[b]) for b in range(B)]
    for ci, c in enumerate((kp, vp)):
        got = [logical(c, L, b) for b in range(B) for L in range(layers)]
        for g, w in zip(got, want[ci]):
            np.testing.assert_array_equal(g, w)


def test_bad_paths_rejected():
    kc = np.zeros((1, 1, 16, 4), np.float32)
    vc = np.zeros_like(kc)
    for path, n in (([1, 2], 2), ([0, 3, 3], 3), ([0, 2, 1], 3), ([0], 0)):
        acc = np.array([path + [-1] * (4 - len(path))], np.int32)
        with pytest.raises(oracle.OracleError) as e:
            oracle.kv_compact(kc, vc, np.array([4], np.int32), acc, np.array([n], np.int32), Hkv=1)
        assert e.value.code == oracle.STATUS_BAD_PATH
    acc = np.array([[0, 1, 13, -1]], np.int32)  # P + 13 = 17 > capacity 16
    with pytest.raises(oracle.OracleError) as e:
        oracle.kv_compact(kc, vc, np.array([4], np.int32), acc, np.array([3], np.int32), Hkv=1)
    assert e.value.code == oracle.STATUS_BAD_PREFIX
