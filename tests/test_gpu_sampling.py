"""GPU parity of acceptance by recursive rejection sampling (T > 0) against
the oracle, plus the losslessness property measured on the GPU itself.

The kernel's accept tests use float32 element arithmetic with double sums, so
a decision can differ from the oracle's only where a uniform lies within about
1e-6 (relative) of its threshold: the accepted paths must match exactly for
every sequence whose smallest accept-test margin (reported by the oracle)
exceeds 1e-4.  The bonus token is an inverse-CDF sample over up to 262144
tokens whose steps can be far finer than that rounding, so it must be a valid
sample of the oracle's final distribution: its cumulative mass brackets the
target r * total within 1e-5 of the total (and it equals the oracle's token
wherever the target is that far from a step)."""
import numpy as np
import pytest

import gpu_util as U
import oracle
import paper_2603_01639_amd as ltd
import workloads as W
import test_oracle_sampling as TS

pytestmark = pytest.mark.gpu


def _gpu(sb):
    import torch
    i32 = dict(dtype=torch.int32, device="cuda")
    acc = torch.full((sb.B, sb.logits.shape[1]), -1, **i32)
    toks = torch.full((sb.B, sb.logits.shape[1]), -1, **i32)
    n = torch.zeros((sb.B,), **i32)
    ltd.tree_accept_sampling(U.to_dev(sb.logits), U.to_dev(sb.draft_probs),
                             U.to_dev(sb.draft_tokens), U.to_dev(sb.parents), U.to_dev(sb.n_nodes),
                             U.to_dev(sb.uniforms), acc, toks, n, temperature=sb.temperature)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), toks.cpu().numpy(), n.cpu().numpy()


def _check(sb):
    U.log(f"[sampling] {sb.label} B={sb.B} Voc={sb.logits.shape[2]} T={sb.temperature}")
    acc, toks, n = _gpu(sb)
    wacc, wtoks, wn, margin, final = oracle.tree_accept_sampling(
        sb.logits, sb.draft_probs, sb.draft_tokens, sb.parents, sb.n_nodes, sb.uniforms,
        temperature=sb.temperature, want_final=True)
    checked = exact_bonus = 0
    for b in range(sb.B):
        if margin[b] <= 1e-4:
            continue  # a uniform within rounding of its threshold
        checked += 1
        k = int(wn[b])
        assert n[b] == k, (sb.label, b, n[b], k)
        np.testing.assert_array_equal(acc[b, :k], wacc[b, :k])
        np.testing.assert_array_equal(toks[b, :k - 1], wtoks[b, :k - 1])
        assert (acc[b, k:] == -1).all() and (toks[b, k:] == -1).all()
        # the bonus: a valid inverse-CDF sample of the oracle's final distribution
        cdf = np.cumsum(final[b])
        total = cdf[-1]
        u = int(wacc[b, k - 1])
        target = float(sb.uniforms[b, u, 1]) * total
        v = int(toks[b, k - 1])
        below = cdf[v - 1] if v > 0 else 0.0
        tol = 1e-5 * total
        assert final[b, v] > 0 and below <= target + tol and cdf[v] >= target - tol, (sb.label, b)
        exact_bonus += int(v == wtoks[b, k - 1])
    assert checked >= max(1, sb.B // 2)
    U.log(f"[sampling] {sb.label}: {checked} sequences checked, {exact_bonus} bonus tokens equal")
    return acc, toks, n


@pytest.mark.parametrize("rep", range(3))
def test_8b_shaped_tree(rep):
    _check(W.sampling_8b(rep))


@pytest.mark.parametrize("T,noise,Voc", [(1.0, 1.0, 4096), (0.7, 2.0, 5000), (1.5, 0.5, 152064),
                                         (1.0, 4.0, 333), (1.0, 0.0, 1000)])
def test_batches_of_trees(T, noise, Voc):
    rng = W.rng_for(int(T * 10) + int(noise * 100) + Voc)
    trees = [W.tree_uniform_parent(rng, n) for n in (1, 7, 40, 120, 256, 3)]
    trees.append(W.tree_chain(30))
    trees.append(W.tree_star(50))
    sb = W.make_sampling_batch(rng, trees, Voc, temperature=T, draft_noise=noise,
                               label=f"batch T={T} noise={noise}")
    acc, toks, n = _check(sb)
    if noise == 0.0:  # the draft is the target: every first child is accepted
        for b, tr in enumerate(trees):
            depth_path = []
            u = 0
            while True:
                kids = [c for c in range(u + 1, len(tr)) if tr[c] == u]
                if not kids:
                    break
                u = kids[0]
                depth_path.append(u)
            assert acc[b, 1:n[b]].tolist() == depth_path


def test_rejections_that_exhaust_the_draft_mass():
    """Peaked drafts (noise 8) at T = 0.3 over stars of 120 to 256 children:
    after a few rejections the rejected drafts hold all but a sliver of the
    draft mass, and after a few more all but less than double rounding of 1.
    The remaining mass must be summed over the tokens left; taken as 1 minus
    the rejected mass it loses every digit, and the walk then accepted
    children the rule rejects."""
    for seed in range(2):
        rng = W.rng_for(4242 + seed)
        trees = [W.tree_star(n) for n in (200, 150, 120, 256)]
        _check(W.make_sampling_batch(rng, trees, 4097, temperature=0.3, draft_noise=8.0,
                                     label=f"exhausted draft mass {seed}"))


def test_losslessness_on_the_gpu():
    """The property the rule exists for, measured on the kernel alone: 40000
    toy verifications; the first emitted token follows the root's target and
    the second the target given the first (every |z| < 5)."""
    rng = np.random.default_rng(11)
    tb = TS.toy_batch(rng, 40000)
    sb = W.SamplingBatch(tb["logits"], tb["q"], tb["tok"], tb["par"], tb["n"], tb["uni"], tb["T"],
                         "toy")
    U.log("[sampling] toy losslessness, 40000 trials")
    acc, toks, n = _gpu(sb)
    V = tb["P0"].size
    TS._z_ok(np.bincount(toks[:, 0], minlength=V), tb["P0"], "gpu first token")
    two = n >= 2
    for y in range(V):
        sel = two & (toks[:, 0] == y)
        if sel.sum() > 2000:
            TS._z_ok(np.bincount(toks[sel, 1], minlength=V), tb["P1"][y], f"gpu second after {y}")


def test_validation_stops_a_bad_tree():
    import torch
    sb = W.make_sampling_batch(W.rng_for(5), [W.tree_uniform_parent(W.rng_for(6), 9)], 100)
    par = sb.parents.copy()
    par[0, 4] = 4
    i32 = dict(dtype=torch.int32, device="cuda")
    acc = torch.full((1, 9), -1, **i32)
    toks = torch.full((1, 9), -1, **i32)
    n = torch.full((1,), -3, **i32)
    st = torch.full((1,), -1, **i32)
    ltd.tree_accept_sampling(U.to_dev(sb.logits), U.to_dev(sb.draft_probs),
                             U.to_dev(sb.draft_tokens), U.to_dev(par), U.to_dev(sb.n_nodes),
                             U.to_dev(sb.uniforms), acc, toks, n, validate=True, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == ltd.STATUS_BAD_PARENT
    assert (acc == -1).all() and int(n.item()) == -3
