"""The allocation-free acceptance entry point (ltd_tree_accept_noalloc)
against the workspace entry point (ltd_tree_accept), bit for bit, on two
calls in a row whose second is smaller than the first (the shared scratch
keeps the first call's contents), plus the oracle on both, and the size limit
reported before anything is launched."""
import numpy as np
import pytest

import gpu_util as U
import paper_2603_01639_amd as ltd
import workloads as W

pytestmark = pytest.mark.gpu


def _outs(torch, B, Nmax):
    i32 = dict(dtype=torch.int32, device="cuda")
    return ([torch.full((B, Nmax), -1, **i32) for _ in range(3)] + [torch.zeros((B,), **i32)])


def _batch(seed, ns, Voc, p_match=0.7):
    rng = W.rng_for(seed)
    trees = [W.tree_uniform_parent(rng, n) for n in ns]
    toks = [W.distinct_sibling_tokens(rng, t, Voc) for t in trees]
    return W.make_batch(rng, dtype=W.DTYPE_F32, Hq=1, Hkv=1, d=64, prefix=[0] * len(ns),
                        trees=trees, tokens=toks, Voc=Voc, p_match=p_match,
                        label=f"noalloc N={ns} Voc={Voc}")


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    import torch
    first = _batch(501, (256, 60, 128, 9, 200, 33, 77, 150), 128256)
    second = _batch(502, (40, 7, 18), 32000)
    assert ltd.accept_workspace_size(first.B, first.Nmax, first.Voc) <= ltd.accept_noalloc_max_bytes()
    for b in (first, second):
        U.log(f"[noalloc] {b.label}")
        dev = U.upload(b)
        a = _outs(torch, b.B, b.Nmax)
        ltd.tree_accept_noalloc(dev.logits, dev.tokens, dev.parents, dev.n_nodes, *a)
        w = _outs(torch, b.B, b.Nmax)
        ltd.tree_accept(dev.logits, dev.tokens, dev.parents, dev.n_nodes, *w)
        torch.cuda.synchronize()
        for x, y in zip(a, w):
            np.testing.assert_array_equal(x.cpu().numpy(), y.cpu().numpy())
        U.check_accept(b, tuple(x.cpu().numpy() for x in a))


def test_noalloc_validation_and_limit():
    import torch
    b = _batch(503, (12, 30), 5000)
    dev = U.upload(b)
    bad = dev.parents.clone()
    bad[1, 4] = 9  # not below 4
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    outs = _outs(torch, b.B, b.Nmax)
    ltd.tree_accept_noalloc(dev.logits, dev.tokens, bad, dev.n_nodes, *outs, validate=True,
                            status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == ltd.STATUS_BAD_PARENT
    assert all((o.cpu().numpy() == -1).all() for o in outs[:3])
    # a size past the scratch array is refused on the host, before any launch
    huge_B = ltd.accept_noalloc_max_bytes() // (256 * 8) + 1
    rc = ltd.lib().ltd_tree_accept_noalloc(1, 1, 1, 1, huge_B, 256, 8192, 1, 1, 1, 1, 0, None, None)
    assert rc == ltd.LTD_EWORKSPACE
