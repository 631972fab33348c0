"""Independent references that pin the CPU oracle (test code only).

None of this shares code with ``oracle/`` or with the HIP library.  Each
function restates what the paper fixes in a *different* form from the oracle:

* ``attention_by_root_path``: a tree node's verification output is ordinary
  causal attention for the last token of the sequence "prefix + the node's root
  path" (the tree attention mask of section 3.2 shows a candidate exactly its
  ancestors).  Here the sequence is materialised explicitly and textbook
  single-query softmax attention is run over it.
* ``ancestor_mask_closure``: the same visibility relation computed as the
  reflexive-transitive closure of the child->parent adjacency matrix (boolean
  matrix products), for use with a library attention routine.
* ``accept_by_enumeration``: greedy acceptance (section 3.2, "Draft Tree
  Verification") restated as "among all root paths whose every draft token
  equals the target prediction at its parent, take the longest (smallest leaf
  index on ties)", by listing every root path.
* ``ToyLM``: a one-layer attention language model for the greedy-equivalence
  pin: verifying a draft tree must emit exactly the tokens that token-by-token
  greedy decoding emits.
"""
from __future__ import annotations

import itertools
from typing import List, Sequence, Tuple

import numpy as np


def all_parent_arrays(n: int):
    """Every topologically ordered tree with n nodes: parent[i] in [0, i)."""
    if n == 1:
        yield np.array([-1], np.int32)
        return
    for choice in itertools.product(*[range(i) for i in range(1, n)]):
        yield np.array((-1,) + choice, np.int32)


def root_path(parents: Sequence[int], i: int) -> List[int]:
    path = []
    j = i
    while j != -1:
        path.append(j)
        j = int(parents[j])
    return path[::-1]


def softmax_attention_1q(q: np.ndarray, keys: np.ndarray, vals: np.ndarray, scale: float) -> np.ndarray:
    """Textbook single-query attention in float64."""
    s = (keys.astype(np.float64) @ q.astype(np.float64)) * scale
    w = np.exp(s - s.max())
    return (w[:, None] * vals.astype(np.float64)).sum(0) / w.sum()


def attention_by_root_path(q, k_rows, v_rows, prefix_len: int, parents, scale: float):
    """Per-node causal attention over the explicit sequence prefix + root path.

    q: [N][Hq][d]; k_rows/v_rows: [Hkv][P+N][d] logical rows (prefix, then tree
    nodes in index order).  Returns [N][Hq][d] float64.
    """
    N, Hq, d = q.shape
    Hkv = k_rows.shape[0]
    G = Hq // Hkv
    out = np.zeros((N, Hq, d))
    for i in range(N):
        rows = list(range(prefix_len)) + [prefix_len + j for j in root_path(parents, i)]
        for h in range(Hq):
            g = h // G
            out[i, h] = softmax_attention_1q(q[i, h], k_rows[g, rows], v_rows[g, rows], scale)
    return out


def ancestor_mask_closure(parents) -> np.ndarray:
    """[N][N] bool: m[i][j] = node j is node i or one of its ancestors.

    Reflexive-transitive closure of the adjacency A[i][parent(i)] = 1 by
    repeated squaring of boolean matrices."""
    n = len(parents)
    reach = np.eye(n, dtype=bool)
    for i in range(1, n):
        reach[i, parents[i]] = True
    while True:
        nxt = (reach.astype(np.int64) @ reach.astype(np.int64)) > 0
        if (nxt == reach).all():
            return reach
        reach = nxt


def accept_by_enumeration(pred, tokens, parents) -> Tuple[List[int], List[int]]:
    """Longest fully-matching root path; ties -> smallest leaf index.

    Returns (path, emitted tokens) where the emitted tokens are the accepted
    drafts after the root followed by pred[leaf]."""
    n = len(parents)
    best = [0]
    for leaf in range(n):
        path = root_path(parents, leaf)
        if all(int(tokens[path[k]]) == int(pred[path[k - 1]]) for k in range(1, len(path))):
            if len(path) > len(best):
                best = path
    emitted = [int(tokens[j]) for j in best[1:]] + [int(pred[best[-1]])]
    return best, emitted


class ToyLM:
    """One attention layer + LM head over a small vocabulary, float64 math on
    float32-rounded projections (so the oracle, which sees float32 K/V/Q, and
    the greedy decoder below work on identical values)."""

    def __init__(self, seed: int, vocab: int = 40, width: int = 32, Hq: int = 4, Hkv: int = 2,
                 d: int = 8, max_pos: int = 128):
        r = np.random.Generator(np.random.PCG64(seed))
        self.vocab, self.Hq, self.Hkv, self.d = vocab, Hq, Hkv, d
        self.emb = r.standard_normal((vocab, width))
        self.pos = r.standard_normal((max_pos, width)) * 0.5
        self.wq = r.standard_normal((width, Hq * d)) / np.sqrt(width)
        self.wk = r.standard_normal((width, Hkv * d)) / np.sqrt(width)
        self.wv = r.standard_normal((width, Hkv * d)) / np.sqrt(width)
        self.wo = r.standard_normal((Hq * d, width)) / np.sqrt(Hq * d)
        self.head = r.standard_normal((width, vocab)) * 2.0
        self.scale = 1.0 / np.sqrt(d)

    def hidden(self, tok: int, pos: int) -> np.ndarray:
        return self.emb[tok] + self.pos[pos]

    def qkv(self, tok: int, pos: int):
        x = self.hidden(tok, pos)
        f32 = lambda a: a.astype(np.float32)  # noqa: E731
        return (f32(x @ self.wq).reshape(self.Hq, self.d), f32(x @ self.wk).reshape(self.Hkv, self.d),
                f32(x @ self.wv).reshape(self.Hkv, self.d))

    def logits_from_attention(self, tok: int, pos: int, attn: np.ndarray) -> np.ndarray:
        """attn: [Hq][d] attention output of this position."""
        x = self.hidden(tok, pos)
        h = x + attn.reshape(-1) @ self.wo
        return (h @ self.head).astype(np.float32)

    def greedy(self, prompt: Sequence[int], steps: int) -> Tuple[List[int], float]:
        """Token-by-token greedy continuation with a plain KV cache.  Returns
        the tokens and the smallest top-1/top-2 logit margin seen."""
        seq = list(prompt)
        ks, vs = [], []
        for p, t in enumerate(seq[:-1]):
            _, k, v = self.qkv(t, p)
            ks.append(k)
            vs.append(v)
        out, margin = [], np.inf
        G = self.Hq // self.Hkv
        for _ in range(steps):
            p = len(seq) - 1
            q, k, v = self.qkv(seq[-1], p)
            K = np.stack(ks + [k], 1)  # [Hkv][T][d]
            V = np.stack(vs + [v], 1)
            attn = np.stack([softmax_attention_1q(q[h], K[h // G], V[h // G], self.scale)
                             for h in range(self.Hq)])
            lg = self.logits_from_attention(seq[-1], p, attn)
            srt = np.sort(lg.astype(np.float64))
            margin = min(margin, srt[-1] - srt[-2])
            nxt = int(np.argmax(lg))
            ks.append(k)
            vs.append(v)
            seq.append(nxt)
            out.append(nxt)
        return out, margin
