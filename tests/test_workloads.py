"""The seeded generators produce the shapes and structure the workloads state."""
import numpy as np
import pytest

from brute import root_path
import workloads as W


def _levels(par):
    return np.array([len(root_path(par, i)) - 1 for i in range(len(par))])


def _topological(par):
    return par[0] == -1 and all(0 <= par[i] < i for i in range(1, len(par)))


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -2.5, 0.0, -0.0, 3.0e38], np.float32)
    b = W.f32_to_bf16_bits(x)
    back = W.bf16_bits_to_f32(b)
    assert back[0] == 1.0
    assert back[1] == 1.0  # exact tie -> even mantissa
    assert back[2] == np.float32(1.0 + 2 ** -7)  # 1.5 ulp -> rounds up to 2 ulp
    assert back[3] == -2.5 and back[4] == 0.0 and np.signbit(back[5])
    r = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    assert np.all(np.abs(W.bf16_bits_to_f32(W.f32_to_bf16_bits(r)) - r) <= np.abs(r) * 2 ** -8)


def test_eagle_tree_shape_and_order():
    rng = W.rng_for(1)
    t = W.tree_eagle(rng, 60, 6, 10, 128256)
    assert len(t.parents) == 60 and _topological(t.parents)
    lv = _levels(t.parents)
    assert lv.max() <= 5 and np.all(np.diff(lv) >= 0)  # re-indexed by level
    # scores decrease along every edge, so the kept set is ancestor-closed
    for i in range(1, 60):
        assert t.scores[i] < t.scores[t.parents[i]]
    # sibling tokens are distinct
    for p in range(60):
        kids = t.tokens[t.parents == p]
        assert len(set(kids.tolist())) == len(kids)


def test_eagle_pool_size_formula():
    """The pool holds 1 + W + (D-2) W^2 candidates (section 3.2)."""
    for D, W_ in ((2, 3), (3, 4), (6, 10)):
        pool = 1 + W_ + (D - 2) * W_ * W_
        W.tree_eagle(W.rng_for(2), pool, D, W_, 1000)
        with pytest.raises(ValueError):
            W.tree_eagle(W.rng_for(2), pool + 1, D, W_, 1000)


def test_draft_pool_levels_scores_and_selection_batches():
    """The pool is listed level by level, its levels are true depths, scores
    strictly decrease along every root path (also after float32 rounding they
    never increase), and the selection batches pad with junk past each pool."""
    for D in (1, 2, 6, 12):
        p = W.draft_pool(W.rng_for(D), D, 10, 1000)
        assert len(p.parents) == W.pool_size(D, 10)
        assert _topological(p.parents)
        assert (_levels(p.parents) == p.level).all() and (np.diff(p.level) >= 0).all()
        assert (p.scores[1:] < p.scores[p.parents[1:]]).all()
        s32 = p.scores.astype(np.float32)
        assert (s32[1:] <= s32[p.parents[1:]]).all()
    sb = W.select_batch16()
    assert sb.Vpool == W.MAX_POOL and sb.pool_size.max() <= W.pool_size(12, 10) == 1011
    assert set(sb.n_select.tolist()) <= {W.select_size_action(a) for a in range(12)}
    for b in range(sb.B):
        n = sb.pool_size[b]
        assert (sb.pool_parents[b, n:] >= sb.Vpool).all() and (sb.pool_tokens[b, n:] < 0).all()


@pytest.mark.parametrize("n,depth", [(8, 2), (8, 8), (64, 5), (256, 10)])
def test_exact_depth_trees(n, depth):
    par = W.tree_random_exact_depth(W.rng_for(3), n, depth)
    assert _topological(par) and _levels(par).max() == depth - 1


def test_planted_logits_match_rate():
    rng = W.rng_for(4)
    trees = [W.tree_eagle(rng, 60, 6, 10, 5000) for _ in range(30)]
    hits = internal = 0
    for t in trees:
        lg = rng.standard_normal((60, 5000), dtype=np.float32)
        W.plant_logits(rng, lg, t.parents, t.tokens, 0.7)
        top = lg.argmax(1)
        for u in range(60):
            kids = np.nonzero(t.parents == u)[0]
            srt = np.sort(lg[u])
            assert srt[-1] - srt[-2] >= 1.0 - 1e-6  # planted max is unique
            if len(kids):
                internal += 1
                hits += int(top[u] in set(t.tokens[kids].tolist()))
            else:
                assert top[u] not in set(t.tokens[kids].tolist())
    assert 0.6 < hits / internal < 0.8


def test_paged_batch_block_table_is_a_permutation():
    b = W.config5_paged(with_logits=False, B=4)
    used = []
    for i in range(b.B):
        nb = -(-(int(b.prefix_len[i]) + int(b.n_nodes[i])) // 16)
        used.extend(b.block_table[i, :nb].tolist())
    assert sorted(used) == list(range(b.num_blocks))
    assert b.k_cache.shape == (b.num_blocks, 8, 16, 128)
    assert all(1024 <= p <= 8192 for p in b.prefix_len) and all(16 <= n <= 128 for n in b.n_nodes)


def test_configs_are_deterministic():
    a = W.config1_tiny_f32()
    b = W.config1_tiny_f32()
    for x, y in ((a.q, b.q), (a.k_cache, b.k_cache), (a.parents, b.parents), (a.logits, b.logits)):
        np.testing.assert_array_equal(x, y)
    assert a.q.shape == (1, 16, 8, 64) and a.k_cache.shape == (1, 8, 144, 64)
