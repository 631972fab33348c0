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
