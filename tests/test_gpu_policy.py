"""GPU parity of draft-policy inference against the float64 oracle.

Logits: float32 accumulation of K-term dot products errs by at most about
K * 2^-24 times the sum of |w x| terms; chaining the layers, the error of every
logit is bounded by (K1 + K2 + K3) * 2^-24 times the same network run on |s|,
|W| and |b| (oracle.policy.policy_mlp_abs), which the test uses as its
tolerance.  Actions: if every logit of a state is within e of the oracle's and
the oracle's two largest differ by more than 2e, the argmax is the same; so
the action must equal the oracle's wherever its margin exceeds twice the
measured error, and otherwise be one whose logit is within 2e of the best."""
import numpy as np
import pytest

import gpu_util as U
from oracle import policy as OP
import paper_2603_01639_amd as ltd
import workloads as W

pytestmark = pytest.mark.gpu


def _run(pb, pad=W.STATE_PAD):
    import torch
    layers = [(U.to_dev(w), U.to_dev(b)) for w, b in pb.layers]
    logits = torch.full((pb.B, pb.dims[-1]), float("nan"), dtype=torch.float32, device="cuda")
    action = torch.full((pb.B,), -7, dtype=torch.int32, device="cuda")
    ltd.policy_forward(pb.layout, U.to_dev(pb.scores), U.to_dev(pb.pool_size), U.to_dev(pb.depth),
                       U.to_dev(pb.ctx_len), layers, logits, action, pad=pad,
                       action_offset=pb.action_offset, action_scale=pb.action_scale)
    torch.cuda.synchronize()
    return logits.cpu().numpy(), action.cpu().numpy()


def _check(pb, pad=W.STATE_PAD):
    U.log(f"[policy] {pb.label} B={pb.B}")
    got_l, got_a = _run(pb, pad)
    state = OP.policy_state(pb.layout, pb.scores, pb.pool_size, pb.depth, pb.ctx_len,
                            pb.dims[0] - 2, pad)
    want_l, want_a = OP.policy_mlp(state, pb.layers, pb.action_offset, pb.action_scale)
    bound = sum(pb.dims[:-1]) * 2.0 ** -24 * OP.policy_mlp_abs(state, pb.layers) + 1e-30
    err = np.abs(got_l - want_l)
    assert np.isfinite(got_l).all() and (err <= bound).all(), f"{pb.label}: {(err / bound).max()}"
    _check_actions(pb, got_l, got_a, want_l, want_a)
    U.log(f"[policy] {pb.label} max err/bound {(err / bound).max():.3f}")
    return got_l, got_a


def _check_actions(pb, got_l, got_a, want_l, want_a):
    for b in range(pb.B):
        e = np.abs(got_l[b] - want_l[b]).max()
        srt = np.sort(want_l[b])[::-1]
        margin = srt[0] - srt[1] if len(srt) > 1 else np.inf
        if margin > 2 * e:
            assert got_a[b] == want_a[b], (pb.label, b)
        else:  # a near-tie: a logit within 2e of the best
            idx = (got_a[b] - pb.action_offset) // pb.action_scale
            assert want_l[b, idx] >= srt[0] - 2 * e, (pb.label, b)


@pytest.mark.parametrize("B", [1, 3, 8, 9, 16])
def test_size_policy(B):
    _check(W.policy_batch(W.LAYOUT_SIZE, B))


@pytest.mark.parametrize("B", [1, 7, 16])
def test_depth_policy(B):
    _check(W.policy_batch(W.LAYOUT_DEPTH, B))


@pytest.mark.parametrize("dims", [(3, 1, 1), (7, 5, 3), (50, 64, 33, 64), (1024, 1024, 1024, 2),
                                  (130, 100, 7)])
def test_other_shapes_and_limits(dims):
    """Tiny and maximal widths, a single output, widths that are not multiples
    of the wave or of four units per workgroup."""
    base = W.policy_batch(W.LAYOUT_SIZE, 11, rep=len(dims))
    rng = np.random.default_rng(sum(dims))
    pb = W.PolicyBatch(W.LAYOUT_SIZE if dims[0] % 2 else W.LAYOUT_DEPTH, dims,
                       W.policy_layers(rng, dims), base.scores, base.pool_size, base.depth,
                       base.ctx_len, 3, 5, label=f"dims {dims}")
    _check(pb, pad=-7.5)


def test_deterministic():
    pb = W.policy_batch(W.LAYOUT_SIZE, 16, rep=3)
    a = _run(pb)
    b = _run(pb)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_size_action_feeds_selection():
    """The size policy writes V = 20 + 20 a into the selection's n_select on
    the device; the selection then matches the oracle run with the oracle's
    action."""
    import torch
    import oracle
    pb = W.policy_batch(W.LAYOUT_SIZE, 16, rep=5)
    layers = [(U.to_dev(w), U.to_dev(b)) for w, b in pb.layers]
    scores = U.to_dev(pb.scores)
    pool_size = U.to_dev(pb.pool_size)
    n_select = torch.zeros((pb.B,), dtype=torch.int32, device="cuda")
    logits = torch.empty((pb.B, 12), dtype=torch.float32, device="cuda")
    ltd.policy_forward(pb.layout, scores, pool_size, U.to_dev(pb.depth), U.to_dev(pb.ctx_len),
                       layers, logits, n_select, pad=W.STATE_PAD, action_offset=20,
                       action_scale=20)
    i32 = dict(dtype=torch.int32, device="cuda")
    parents_pool, tokens_pool = pb.pool_parents, pb.pool_tokens
    outs = [torch.full((pb.B, 256), -1, **i32) for _ in range(2)]
    nn = torch.zeros((pb.B,), **i32)
    ltd.select_candidates(scores, U.to_dev(parents_pool), U.to_dev(tokens_pool), pool_size,
                          n_select, outs[0], outs[1], nn)
    torch.cuda.synchronize()
    state = OP.policy_state(pb.layout, pb.scores, pb.pool_size, pb.depth, pb.ctx_len,
                            pb.dims[0] - 2, W.STATE_PAD)
    want_l, want_v = OP.policy_mlp(state, pb.layers, 20, 20)
    got_l, got_v = logits.cpu().numpy(), n_select.cpu().numpy()
    srt = np.sort(want_l, axis=1)
    err = np.abs(got_l - want_l).max(axis=1)
    assert (srt[:, -1] - srt[:, -2] > 2 * err).all()  # no near-tie: the actions must agree
    np.testing.assert_array_equal(got_v, want_v)
    want = oracle.select_candidates(pb.scores, parents_pool, tokens_pool, pb.pool_size,
                                    want_v.astype(np.int32), 256)
    np.testing.assert_array_equal(outs[0].cpu().numpy(), want[1])
    np.testing.assert_array_equal(outs[1].cpu().numpy(), want[2])
    np.testing.assert_array_equal(nn.cpu().numpy(), want[4])

