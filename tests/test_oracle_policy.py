"""Pins for the policy-inference oracle (CPU only).

* hand-derived forward passes (tests/golden/policy_examples.json): a ReLU that
  clips, a tie between logits, the size policy's action-to-V mapping;
* a different library: torch.nn Linear/ReLU stacks in float64 with the same
  weights, at the paper's shapes (size policy 1013 -> 1024 -> 256 -> 12, depth
  policy 102 -> 1024 -> 2);
* special cases: zero weights give the bias, and every action in 0..11 maps
  to V = 20, 40, ..., 240;
* the state layouts, against vectors built by hand.
"""
import json
import os

import numpy as np
import pytest

from oracle import policy as OP

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "policy_examples.json")


def _layers(spec):
    return [(np.array(l["w"], np.float64), np.array(l["b"], np.float64)) for l in spec]


def random_layers(rng, dims):
    """Uniform(+-1/sqrt(fan_in)) weights and biases (torch's Linear default)."""
    out = []
    for i, o in zip(dims[:-1], dims[1:]):
        k = 1.0 / np.sqrt(i)
        out.append((rng.uniform(-k, k, size=(o, i)).astype(np.float32),
                    rng.uniform(-k, k, size=o).astype(np.float32)))
    return out


def test_worked_examples():
    for ex in json.load(open(GOLDEN))["examples"]:
        layers = _layers(ex["layers"])
        x = np.array([ex["x"]], np.float64)
        logits, a = OP.policy_mlp(x, layers)
        assert logits[0].tolist() == ex["logits"], ex["name"]
        assert a[0] == ex["argmax"], ex["name"]
        _, a2 = OP.policy_mlp(x, layers, ex["action_offset"], ex["action_scale"])
        assert a2[0] == ex["action"], ex["name"]
        # the hidden activations, one layer at a time
        h = x
        for k, want in enumerate(ex["hidden"]):
            h, _ = OP.policy_mlp(h, layers[k:k + 1] + [(np.eye(len(want)), np.zeros(len(want)))])
            assert h[0].tolist() == want, (ex["name"], k)


@pytest.mark.parametrize("dims", [(1013, 1024, 256, 12), (102, 1024, 2), (7, 5, 3)])
def test_matches_torch_linear_relu_stack(dims):
    import torch
    rng = np.random.default_rng(len(dims) * 100 + dims[-1])
    layers = random_layers(rng, list(dims))
    x = rng.normal(size=(9, dims[0])) * 3
    mods = []
    for k, (w, b) in enumerate(layers):
        lin = torch.nn.Linear(w.shape[1], w.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(w.astype(np.float64)))
            lin.bias.copy_(torch.from_numpy(b.astype(np.float64)))
        mods.append(lin)
        if k + 1 < len(layers):
            mods.append(torch.nn.ReLU())
    with torch.no_grad():
        want = torch.nn.Sequential(*mods)(torch.from_numpy(x)).numpy()
    got, a = OP.policy_mlp(x, layers)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    assert (a == want.argmax(axis=1)).all()


def test_zero_weights_give_the_bias_and_the_action_map():
    x = np.ones((3, 4))
    bias = np.array([0.0, 3.0, -1.0, 3.0, 2.0, 0.5, 0, 0, 0, 0, 0, 0])
    layers = [(np.zeros((6, 4)), np.zeros(6)), (np.zeros((12, 6)), bias)]
    logits, a = OP.policy_mlp(x, layers, 20, 20)
    assert (logits == bias).all() and (a == 20 + 20 * 1).all()  # tie 1 vs 3 -> 1
    for act in range(12):
        b = np.full(12, -1.0)
        b[act] = 1.0
        _, v = OP.policy_mlp(np.zeros((1, 2)), [(np.zeros((12, 2)), b)], 20, 20)
        assert v[0] == 20 + 20 * act
    assert [20 + 20 * a for a in (0, 11)] == [20, 240]


def test_state_layouts():
    scores = np.array([[0.0, -1.0, -2.0, -3.0, -4.0, 9.0], [0.0, -0.5, 7.0, 7.0, 7.0, 7.0]])
    size = [5, 2]
    D = [4, 2]
    L = [2048, 77]
    s = OP.policy_state(OP.LAYOUT_SIZE, scores, size, D, L, 4, -50.0)
    assert s.tolist() == [[4, 2048, 0, -1, -2, -3], [2, 77, 0, -0.5, -50, -50]]
    s = OP.policy_state(OP.LAYOUT_DEPTH, scores, size, D, L, 3, -50.0)
    assert s.tolist() == [[-2, -3, -4, 4, 2048], [-50, 0, -0.5, 2, 77]]


# ------------------------------------------------- the rounding-bound network
# policy_mlp_abs feeds the GPU test's tolerance: sum(in widths) * 2^-24 * the
# network evaluated on |x|, |W|, |b| without clipping (the first-order bound on
# the rounding error of float32 dot products accumulated in any order).

def test_abs_network_worked_example():
    """By hand: |x| = [1, 2]; layer 1 gives [1*1 + 1*2 + 1, 3*1 + 2*2 + 0.5] =
    [4, 7.5]; layer 2 gives 2*4 + 1*7.5 + 4 = 19.5."""
    layers = [(np.array([[1.0, -1.0], [-3.0, 2.0]]), np.array([-1.0, 0.5])),
              (np.array([[2.0, -1.0]]), np.array([-4.0]))]
    got = OP.policy_mlp_abs(np.array([[1.0, -2.0]]), layers)
    assert got.tolist() == [[19.5]]


def test_abs_network_bounds_every_partial_sum_and_is_tight():
    rng = np.random.default_rng(5)
    dims = [13, 17, 11, 5]
    layers = random_layers(rng, dims)
    x = rng.normal(size=(6, dims[0])) * 4
    for k in range(len(layers)):
        bound = OP.policy_mlp_abs(x, layers[:k + 1])
        # the input of layer k, exactly
        h = x if k == 0 else OP.policy_mlp(x, layers[:k] + [(np.eye(dims[k]), np.zeros(dims[k]))])[0]
        w, b = (np.asarray(a, np.float64) for a in layers[k])
        partial = np.cumsum(h[:, None, :] * w[None, :, :], axis=2) + b[None, :, None]
        assert (np.abs(partial) <= bound[:, :, None] * (1 + 1e-12)).all(), k
    # nonnegative inputs, weights and biases: no ReLU clips, the bound is the output
    pos = [(np.abs(np.asarray(w, np.float64)), np.abs(np.asarray(b, np.float64))) for w, b in layers]
    xp = np.abs(x)
    np.testing.assert_allclose(OP.policy_mlp_abs(xp, pos), OP.policy_mlp(xp, pos)[0], rtol=1e-12)


def _forward_f32(x, layers, order):
    """Float32 forward pass with each dot product accumulated one term at a
    time in the given order of the input index (the bias added last)."""
    h = np.asarray(x, np.float32)
    for k, (w, b) in enumerate(layers):
        w = np.asarray(w, np.float32)
        acc = np.zeros((h.shape[0], w.shape[0]), np.float32)
        for j in order(w.shape[1]):
            acc = (acc + h[:, j:j + 1] * w[None, :, j][0]).astype(np.float32)
        acc = (acc + np.asarray(b, np.float32)).astype(np.float32)
        h = np.maximum(acc, np.float32(0)) if k + 1 < len(layers) else acc
    return h.astype(np.float64)


@pytest.mark.parametrize("order", ["forward", "reverse", "strided"])
def test_float32_forward_within_the_derived_tolerance(order):
    """The tolerance the GPU test applies holds for float32 passes that sum in
    different orders, and it is not vacuous: a pass that drops one input term
    of every dot product (a loop bound off by one) breaks it."""
    orders = {"forward": lambda n: range(n), "reverse": lambda n: range(n - 1, -1, -1),
              "strided": lambda n: [j for r in range(8) for j in range(r, n, 8)],
              "drop_last": lambda n: range(n - 1)}
    rng = np.random.default_rng(11)
    dims = [102, 256, 64, 12]
    layers = random_layers(rng, dims)
    x = rng.normal(size=(4, dims[0])) * 5
    x32 = x.astype(np.float32).astype(np.float64)
    exact = OP.policy_mlp(x32, layers)[0]
    tol = sum(dims[:-1]) * 2.0 ** -24 * OP.policy_mlp_abs(x32, layers)
    got = _forward_f32(x32, layers, orders[order])
    assert (np.abs(got - exact) <= tol).all()
    bad = _forward_f32(x32, layers, orders["drop_last"])
    assert (np.abs(bad - exact) > tol).any()
