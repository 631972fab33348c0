"""CPU oracle for the draft policies' inference (arXiv 2603.01639).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  Plain numpy in float64; it shares no code with the HIP library.

What it follows:

* the state (section 4, equation of the state vector): the draft depth D,
  the context length L and the candidates' scores.  The size policy sees every
  candidate of the draft tree (appendix A.2, "Size Policy": the scores of all
  1 + W + (D-2) W^2 candidates, padded to a fixed size), laid out
  [D, L, P_1 .. P_n, pad ..]; the depth policy sees only the scores of the
  newest expansion, W^2 of them, followed by the two scalars (appendix A.2,
  "Depth Policy"), laid out [P_1 .. P_{W^2}, D, L];
* the networks (appendix A.2 and the training details): fully connected
  layers with ReLU, hidden widths [1024, 256] for the size policy and [1024]
  for the depth policy, 12 and 2 output logits; the action is the most likely
  one (lowest index on ties), and the size policy's 12 actions map linearly
  onto V in [20, 240].
"""
import numpy as np

LAYOUT_SIZE = 0
LAYOUT_DEPTH = 1


def policy_state(layout, scores, pool_size, depth, ctx_len, n_feat, pad):
    """States ``[B][n_feat + 2]`` (float64) from pool scores ``[B][Vpool]``.

    LAYOUT_SIZE: ``[D, L, scores[0:n], pad ...]`` with n = min(pool_size,
    n_feat).  LAYOUT_DEPTH: ``[scores[n - n_feat : n], D, L]`` with n =
    pool_size, i.e. the last ``n_feat`` candidates of the pool (padded in front
    when the pool is shorter)."""
    scores = np.asarray(scores, np.float64)
    B = scores.shape[0]
    out = np.full((B, n_feat + 2), float(pad))
    for b in range(B):
        n = int(pool_size[b])
        if layout == LAYOUT_SIZE:
            out[b, 0] = depth[b]
            out[b, 1] = ctx_len[b]
            k = min(n, n_feat)
            out[b, 2:2 + k] = scores[b, :k]
        else:
            k = min(n, n_feat)
            out[b, n_feat - k:n_feat] = scores[b, n - k:n]
            out[b, n_feat] = depth[b]
            out[b, n_feat + 1] = ctx_len[b]
    return out


def policy_mlp(x, layers, action_offset=0, action_scale=1):
    """Forward pass.  ``layers`` is a list of (W [out][in], b [out]); ReLU
    after every layer but the last.  Returns (logits [B][A], action [B]) with
    action = action_offset + action_scale * argmax(logits)."""
    h = np.asarray(x, np.float64)
    for k, (w, bias) in enumerate(layers):
        h = h @ np.asarray(w, np.float64).T + np.asarray(bias, np.float64)
        if k + 1 < len(layers):
            h = np.maximum(h, 0.0)
    action = action_offset + action_scale * np.argmax(h, axis=1)
    return h, action.astype(np.int64)


def policy_mlp_abs(x, layers):
    """The same network on |x| and |W|, |b| with no ReLU clipping: a bound on
    the magnitude of every partial sum, used to derive rounding tolerances."""
    h = np.abs(np.asarray(x, np.float64))
    for w, bias in layers:
        h = h @ np.abs(np.asarray(w, np.float64)).T + np.abs(np.asarray(bias, np.float64))
    return h
