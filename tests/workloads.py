"""Seeded synthetic inputs shaped like the paper's verification workloads.

Test infrastructure: the GPU parity tests, the oracle's pins, the smoke check
and the benchmark draw their inputs here; nothing in the HIP library or the
oracle imports it.  It computes none of the verification step itself (no
attention, argmax, acceptance walk or compaction).  It does hold two pieces of
the draft side of the method, written independently in numpy, because
realistic trees need them: ``draft_pool`` runs the beam of section 3.2 ("Draft
Tree Generation") on random draft distributions, and ``tree_eagle`` cuts a
pool to its top-N candidates ("Candidate Token Selection").  The kernels only
ever see their outputs (parents, tokens, scores); the oracle's selection and
expansion are also checked against these two functions as independent
implementations.

Shapes follow the paper's setting (arXiv 2603.01639): Eagle-style beam trees of
width W and depth D (section 3.2, "Draft Tree Generation"), a verification size
V taken as the top-V candidates by cumulative probability (section 3.2,
"Candidate Token Selection"; the size policy moves V over [20, 240], appendix
A.2), and Llama-3-8B / Qwen3-32B / 70B-like attention shapes.  The paper's
datasets and weights are not used: every tensor is synthetic.

Conventions:
* RNG: ``numpy.random.Generator(PCG64(seed))``; the standard seed of config c,
  repetition r is ``1639 + 100 * c + r``.
* bf16 tensors are returned as uint16 bit patterns, rounded to nearest even
  from the float32 draw.
* Trees are parent arrays in topological order: ``parents[0] = -1`` and
  ``0 <= parents[i] < i``.  N counts the root.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

DTYPE_F32 = 0
DTYPE_BF16 = 1


def rng_for(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def config_seed(config: int, rep: int = 0) -> int:
    return 1639 + 100 * config + rep


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); return uint16 bits.

    In 32-bit integer arithmetic, in place on a copy: adding 0x7FFF plus the
    kept part's lowest bit cannot wrap for any finite or infinite input (the
    largest pattern, -inf = 0xFF800000, stays far below 2^32 - 0x8000)."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    t = u >> 16
    t &= 1
    t += 0x7FFF
    u += t
    u >>= 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------- trees

def tree_uniform_parent(rng: np.random.Generator, n: int) -> np.ndarray:
    """Node i's parent uniform in [0, i-1]; node 0 is the root."""
    par = np.empty(n, np.int32)
    par[0] = -1
    for i in range(1, n):
        par[i] = rng.integers(0, i)
    return par


def tree_chain(n: int) -> np.ndarray:
    par = np.arange(-1, n - 1, dtype=np.int32)
    return par


def tree_star(n: int) -> np.ndarray:
    par = np.zeros(n, np.int32)
    par[0] = -1
    return par


def tree_random_exact_depth(rng: np.random.Generator, n: int, depth: int) -> np.ndarray:
    """A chain 0 -> ... -> depth-1 (so the tree has exactly ``depth`` levels),
    then every further node picks a uniform parent among nodes whose level is
    below depth-1."""
    if not (1 <= depth <= n):
        raise ValueError("need 1 <= depth <= n")
    par = np.empty(n, np.int32)
    par[0] = -1
    level = np.zeros(n, np.int32)
    for i in range(1, depth):
        par[i] = i - 1
        level[i] = i
    eligible = [i for i in range(depth) if level[i] < depth - 1]
    for i in range(depth, n):
        p = eligible[rng.integers(0, len(eligible))]
        par[i] = p
        level[i] = level[p] + 1
        if level[i] < depth - 1:
            eligible.append(i)
    return par


@dataclasses.dataclass
class DraftTree:
    parents: np.ndarray  # int32 [N]
    tokens: np.ndarray  # int32 [N]; tokens[0] is the root token
    scores: np.ndarray  # float64 [N] cumulative log-probability (root = 0)


@dataclasses.dataclass
class DraftPool:
    """Every candidate a beam-like drafter produced, in the order it produced
    them (the root, then level after level), before any selection."""
    parents: np.ndarray  # int32 [n]; parents[0] = -1, 0 <= parents[i] < i
    tokens: np.ndarray  # int32 [n]
    scores: np.ndarray  # float64 [n] cumulative log-probability (root = 0)
    level: np.ndarray  # int32 [n] depth below the root
    # every expansion, in order: (node, the W + 1 Dirichlet components sorted
    # descending, the W child tokens); rounds of expansions are separated by
    # the beam selection of the next leaves
    draws: Optional[list] = None


def _children_of(parents: np.ndarray) -> List[List[int]]:
    ch: List[List[int]] = [[] for _ in range(len(parents))]
    for i in range(1, len(parents)):
        ch[parents[i]].append(i)
    return ch


def pool_size(depth: int, width: int) -> int:
    """Candidates in a depth-``depth`` pool: 1 + W + (D-2) W^2 for D >= 2
    (section 3.2, "Draft Tree Generation"), the root alone for D = 1."""
    return 1 if depth <= 1 else 1 + width + (depth - 2) * width * width


def draft_pool(rng: np.random.Generator, depth: int, width: int, vocab: int) -> DraftPool:
    """Beam-like draft pool (section 3.2, "Draft Tree Generation").

    ``depth`` counts levels including the root: level 1 is the root's top-W
    children, then depth-2 rounds each add the W*W children of the current W
    leaves and keep the top-W of them (by cumulative score) as the next leaves,
    so the pool has 1 + W + (depth-2) * W^2 nodes.  Conditional log-probs of a
    node's W children are the logs of the sorted top-W components of a
    Dirichlet(0.5 * 1_{W+1}) draw; sibling tokens are distinct.  Scores
    strictly decrease along every root path.
    """
    pool_par = [-1]
    pool_lvl = [0]
    pool_score = [0.0]
    pool_tok = [int(rng.integers(0, vocab))]

    draws = []

    def expand(node: int) -> List[int]:
        full = np.sort(rng.dirichlet(np.full(width + 1, 0.5)))[::-1]
        p = np.maximum(full[:width], 1e-300)
        toks = rng.choice(vocab, size=width, replace=False)
        draws.append((node, full.copy(), toks.copy()))
        out = []
        for c in range(width):
            pool_par.append(node)
            pool_lvl.append(pool_lvl[node] + 1)
            pool_score.append(pool_score[node] + float(np.log(p[c])))
            pool_tok.append(int(toks[c]))
            out.append(len(pool_par) - 1)
        return out

    if depth >= 2:
        leaves = expand(0)
        for _ in range(depth - 2):
            cand: List[int] = []
            for leaf in leaves:
                cand.extend(expand(leaf))
            cand.sort(key=lambda j: -pool_score[j])
            leaves = cand[:width]
    return DraftPool(np.array(pool_par, np.int32), np.array(pool_tok, np.int32),
                     np.array(pool_score, np.float64), np.array(pool_lvl, np.int32), draws)


def tree_eagle(rng: np.random.Generator, n: int, depth: int, width: int, vocab: int) -> DraftTree:
    """A ``draft_pool`` cut down to its top-``n`` candidates by cumulative
    score (section 3.2, "Candidate Token Selection") and re-indexed by (level,
    score rank).  The top-n set is ancestor-closed because scores strictly
    decrease along a path.  (This is the generator's own short selection, used
    to shape verification inputs; the selection step itself is a separate
    kernel with its own oracle.)
    """
    pool = draft_pool(rng, depth, width, vocab)
    total = len(pool.parents)
    if n > total:
        raise ValueError(f"tree pool has {total} nodes, asked for {n}")
    order = sorted(range(total), key=lambda j: -pool.scores[j])[:n]
    keep = set(order)
    for j in order:  # ancestor closure (guaranteed by strictly decreasing scores)
        assert pool.parents[j] == -1 or pool.parents[j] in keep
    order.sort(key=lambda j: (pool.level[j], -pool.scores[j]))
    new_id = {old: new for new, old in enumerate(order)}
    parents = np.array([-1 if pool.parents[j] == -1 else new_id[pool.parents[j]] for j in order],
                       np.int32)
    return DraftTree(parents, pool.tokens[order].astype(np.int32), pool.scores[order].copy())


def distinct_sibling_tokens(rng: np.random.Generator, parents: np.ndarray, vocab: int) -> np.ndarray:
    """Uniform tokens with siblings distinct; the root token is uniform too."""
    n = len(parents)
    tok = np.empty(n, np.int32)
    tok[0] = rng.integers(0, vocab)
    for p, kids in enumerate(_children_of(parents)):
        if kids:
            tok[kids] = rng.choice(vocab, size=len(kids), replace=False)
    return tok


def plant_logits(rng: np.random.Generator, logits: np.ndarray, parents: np.ndarray,
                 tokens: np.ndarray, p_match: float) -> None:
    """In place: logits[u] ~ N(0,1) gets one entry raised to max(row) + 1.

    For a node with children, with probability ``p_match`` the raised entry is
    a uniformly chosen child's token (that child is then the target's
    prediction); otherwise, and for leaves, it is a token no child of u uses.
    """
    n, vocab = logits.shape[0], logits.shape[1]
    kids = _children_of(parents)
    for u in range(len(parents)):
        row = logits[u]
        ch = kids[u]
        if ch and rng.random() < p_match:
            t = int(tokens[ch[rng.integers(0, len(ch))]])
        else:
            used = set(int(tokens[c]) for c in ch)
            while True:
                t = int(rng.integers(0, vocab))
                if t not in used:
                    break
        row[t] = row.max() + np.float32(1.0)
    del n


# --------------------------------------------------------------------------- batches

@dataclasses.dataclass
class VerifyBatch:
    """One verification step's inputs (host arrays)."""
    dtype: int
    B: int
    Nmax: int
    Hq: int
    Hkv: int
    d: int
    Voc: int
    q: np.ndarray  # [B][Nmax][Hq][d]   f32 or bf16 bits
    k_cache: np.ndarray  # contiguous [B][Hkv][cap][d] or paged [nblk][Hkv][bs][d]
    v_cache: np.ndarray
    prefix_len: np.ndarray  # int32 [B]
    parents: np.ndarray  # int32 [B][Nmax]
    n_nodes: np.ndarray  # int32 [B]
    draft_tokens: np.ndarray  # int32 [B][Nmax]
    logits: Optional[np.ndarray]  # float32 [B][Nmax][Voc]
    block_table: Optional[np.ndarray] = None  # int32 [B][max_blocks]
    block_size: int = 0
    num_blocks: int = 0
    label: str = ""

    @property
    def paged(self) -> bool:
        return self.block_table is not None

    @property
    def kv_rows(self) -> int:
        return self.block_size if self.paged else self.k_cache.shape[2]

    @property
    def max_blocks(self) -> int:
        return 0 if self.block_table is None else self.block_table.shape[1]

    @property
    def max_prefix(self) -> int:
        return int(self.prefix_len.max()) if self.B else 0


def _normal(rng, shape, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    return x if dtype == DTYPE_F32 else f32_to_bf16_bits(x)


def make_batch(rng: np.random.Generator, *, dtype: int, Hq: int, Hkv: int, d: int,
               prefix: List[int], trees: List[np.ndarray], tokens: List[np.ndarray], Voc: int,
               p_match: Optional[float], Nmax: Optional[int] = None, block_size: int = 0,
               cap_slack: int = 0, with_logits: bool = True, label: str = "") -> VerifyBatch:
    """Assemble a batch.  ``p_match=None`` leaves the logits unplanted N(0,1).

    With ``block_size > 0`` the cache is paged: every sequence gets
    ceil((P_b + N_b) / block_size) blocks whose physical ids are a seeded
    permutation of the pool; unused block-table entries hold 0.
    """
    B = len(prefix)
    ns = [len(t) for t in trees]
    Nmax = max(ns) if Nmax is None else Nmax
    parents = np.full((B, Nmax), -1, np.int32)
    toks = np.zeros((B, Nmax), np.int32)
    for b in range(B):
        parents[b, :ns[b]] = trees[b]
        toks[b, :ns[b]] = tokens[b]
    prefix_len = np.array(prefix, np.int32)
    n_nodes = np.array(ns, np.int32)
    q = _normal(rng, (B, Nmax, Hq, d), dtype)
    if block_size > 0:
        blocks_per = [-(-(prefix[b] + ns[b]) // block_size) for b in range(B)]
        num_blocks = int(sum(blocks_per))
        max_blocks = max(blocks_per)
        perm = rng.permutation(num_blocks).astype(np.int32)
        table = np.zeros((B, max_blocks), np.int32)
        pos = 0
        for b in range(B):
            table[b, :blocks_per[b]] = perm[pos:pos + blocks_per[b]]
            pos += blocks_per[b]
        k = _normal(rng, (num_blocks, Hkv, block_size, d), dtype)
        v = _normal(rng, (num_blocks, Hkv, block_size, d), dtype)
    else:
        table = None
        num_blocks = 0
        cap = max(prefix[b] + ns[b] for b in range(B)) + cap_slack
        k = _normal(rng, (B, Hkv, cap, d), dtype)
        v = _normal(rng, (B, Hkv, cap, d), dtype)
    logits = None
    if with_logits:
        logits = rng.standard_normal(size=(B, Nmax, Voc), dtype=np.float32)
        if p_match is not None:
            for b in range(B):
                plant_logits(rng, logits[b], trees[b], tokens[b], p_match)
    return VerifyBatch(dtype=dtype, B=B, Nmax=Nmax, Hq=Hq, Hkv=Hkv, d=d, Voc=Voc, q=q, k_cache=k,
                       v_cache=v, prefix_len=prefix_len, parents=parents, n_nodes=n_nodes,
                       draft_tokens=toks, logits=logits, block_table=table, block_size=block_size,
                       num_blocks=num_blocks, label=label)


# --------------------------------------------------------------------------- the five workloads

def config1_tiny_f32(rep: int = 0) -> VerifyBatch:
    """Tiny fp32: B=1, 8/8 heads, d=64, prefix 128, 16-node uniform-parent
    tree, vocab 1000, unplanted N(0,1) logits and uniform draft tokens."""
    rng = rng_for(config_seed(1, rep))
    par = tree_uniform_parent(rng, 16)
    tok = rng.integers(0, 1000, size=16).astype(np.int32)
    return make_batch(rng, dtype=DTYPE_F32, Hq=8, Hkv=8, d=64, prefix=[128], trees=[par],
                      tokens=[tok], Voc=1000, p_match=None, label="tiny-f32 P128 N16")


def config2_8b(rep: int = 0, with_logits: bool = True) -> VerifyBatch:
    """Llama-3-8B-shaped bf16: 32/8 heads, d=128, prefix 2048, Eagle tree of
    depth 6 with top-10 expansion reranked to 60 nodes, vocab 128256, p=0.7."""
    rng = rng_for(config_seed(2, rep))
    t = tree_eagle(rng, 60, 6, 10, 128256)
    return make_batch(rng, dtype=DTYPE_BF16, Hq=32, Hkv=8, d=128, prefix=[2048], trees=[t.parents],
                      tokens=[t.tokens], Voc=128256, p_match=0.7, with_logits=with_logits,
                      label="8B bf16 P2048 N60")


def config2_d64(rep: int = 0, with_logits: bool = True) -> VerifyBatch:
    """Config 2's shape with head_dim 64 (32/8 heads, prefix 2048, the same
    Eagle tree, vocab 128256): the bf16 head size the MFMA kernel does not
    take, which runs on the row-wise kernel."""
    rng = rng_for(config_seed(2, rep) + 500)
    t = tree_eagle(rng, 60, 6, 10, 128256)
    return make_batch(rng, dtype=DTYPE_BF16, Hq=32, Hkv=8, d=64, prefix=[2048], trees=[t.parents],
                      tokens=[t.tokens], Voc=128256, p_match=0.7, with_logits=with_logits,
                      label="8B-shaped bf16 d64 P2048 N60")


def config3_long(rep: int = 0, with_logits: bool = True) -> VerifyBatch:
    """As config 2 with prefix 16384 and p=0.8 (long-reasoning context)."""
    rng = rng_for(config_seed(3, rep))
    t = tree_eagle(rng, 60, 6, 10, 128256)
    return make_batch(rng, dtype=DTYPE_BF16, Hq=32, Hkv=8, d=128, prefix=[16384],
                      trees=[t.parents], tokens=[t.tokens], Voc=128256, p_match=0.8,
                      with_logits=with_logits, label="8B bf16 P16384 N60")


C4_SIZES = (8, 16, 32, 64, 128, 256)


def config4_sweep(n: int, depth: int, rep: int = 0, with_logits: bool = True) -> VerifyBatch:
    """32B-shaped bf16: 64/8 heads, d=128, prefix 4096, random tree with N
    nodes and exactly ``depth`` levels, vocab 152064, p=0.6."""
    rng = rng_for(config_seed(4, rep) * 1000 + n * 16 + depth)
    par = tree_random_exact_depth(rng, n, depth)
    tok = distinct_sibling_tokens(rng, par, 152064)
    return make_batch(rng, dtype=DTYPE_BF16, Hq=64, Hkv=8, d=128, prefix=[4096], trees=[par],
                      tokens=[tok], Voc=152064, p_match=0.6, with_logits=with_logits,
                      label=f"32B bf16 P4096 N{n} D{depth}")


def config5_paged(rep: int = 0, with_logits: bool = True, B: int = 16) -> VerifyBatch:
    """Batched paged verify: B=16, 70B-shaped 64/8 heads, d=128, prefix
    uniform in [1024, 8192], 16-token blocks with a shuffled block table, tree
    size uniform in [16, 128] (Eagle depth-6 trees reranked), vocab 128256,
    p=0.7."""
    rng = rng_for(config_seed(5, rep))
    prefix = [int(rng.integers(1024, 8193)) for _ in range(B)]
    ns = [int(rng.integers(16, 129)) for _ in range(B)]
    trees, toks = [], []
    for b in range(B):
        t = tree_eagle(rng, ns[b], 6, 10, 128256)
        trees.append(t.parents)
        toks.append(t.tokens)
    return make_batch(rng, dtype=DTYPE_BF16, Hq=64, Hkv=8, d=128, prefix=prefix, trees=trees,
                      tokens=toks, Voc=128256, p_match=0.7, Nmax=max(ns), block_size=16,
                      with_logits=with_logits, label="70B bf16 paged B16")


def config5_tp_share(rep: int = 0, tp: int = 8) -> VerifyBatch:
    """One GPU's share of the c5 batch under tp-way tensor parallelism over
    the kv heads: the same sequences, prefixes, trees and 16-token paged
    layout as config5_paged, with 64/tp query and 8/tp kv heads.  Attention
    only: acceptance needs the whole vocabulary, which a vocabulary-sharded LM
    head gathers first."""
    rng = rng_for(config_seed(5, rep))
    B = 16
    prefix = [int(rng.integers(1024, 8193)) for _ in range(B)]
    ns = [int(rng.integers(16, 129)) for _ in range(B)]
    trees, toks = [], []
    for b in range(B):
        t = tree_eagle(rng, ns[b], 6, 10, 128256)
        trees.append(t.parents)
        toks.append(t.tokens)
    return make_batch(rng, dtype=DTYPE_BF16, Hq=64 // tp, Hkv=8 // tp, d=128, prefix=prefix,
                      trees=trees, tokens=toks, Voc=128256, p_match=0.7, Nmax=max(ns),
                      block_size=16, with_logits=False, label=f"70B bf16 paged B16, TP{tp} share")


# ------------------------------------------------------ candidate selection

MAX_POOL = 1024  # candidate pools up to 1 + W + (D-2) W^2 = 1011 (W = 10, D = 12)


@dataclasses.dataclass
class SelectBatch:
    """Inputs of candidate selection for B sequences: draft pools padded to
    Vpool columns, and the verification size V each sequence asks for."""
    B: int
    Vpool: int
    Nmax: int
    scores: np.ndarray  # float32 [B, Vpool] cumulative log-probability
    pool_parents: np.ndarray  # int32 [B, Vpool]
    pool_tokens: np.ndarray  # int32 [B, Vpool]
    pool_size: np.ndarray  # int32 [B]
    n_select: np.ndarray  # int32 [B]
    label: str = ""


def make_select_batch(pools: List[DraftPool], n_select: List[int], *, Vpool: Optional[int] = None, Nmax: Optional[int] = None,
                      label: str = "") -> SelectBatch:
    """Pack pools into [B, Vpool] arrays.  Columns past a pool's size hold
    junk that a correct consumer never reads (scores above the root's, parent
    indices out of range, negative tokens)."""
    B = len(pools)
    sizes = [len(p.parents) for p in pools]
    Vpool = Vpool or max(sizes)
    Nmax = Nmax or max(n_select)
    scores = np.full((B, Vpool), 1e30, np.float32)
    par = np.full((B, Vpool), Vpool + 7, np.int32)
    tok = np.full((B, Vpool), -5, np.int32)
    for b, p in enumerate(pools):
        n = sizes[b]
        # float32 rounding is monotone, so a child never scores above its parent
        scores[b, :n] = p.scores.astype(np.float32)
        par[b, :n] = p.parents
        tok[b, :n] = p.tokens
    return SelectBatch(B, Vpool, Nmax, scores, par, tok, np.array(sizes, np.int32),
                       np.array(n_select, np.int32), label)


def select_size_action(a: int) -> int:
    """Verification size of size-policy action a in 0..11: 12 actions mapped
    linearly onto [20, 240] (appendix A.2, "Size Policy")."""
    return 20 + 20 * a


def select_8b(rep: int = 0) -> SelectBatch:
    """The 8B-shaped step's selection: one depth-6, width-10 pool (411
    candidates) cut to V = 60."""
    rng = rng_for(config_seed(6, rep))
    pool = draft_pool(rng, 6, 10, 128256)
    return make_select_batch([pool], [60], label="select D6 W10 pool411 V60")


def select_deep(rep: int = 0) -> SelectBatch:
    """The largest pool: depth 12, width 10 (1011 candidates) cut to V = 240."""
    rng = rng_for(config_seed(7, rep))
    pool = draft_pool(rng, 12, 10, 128256)
    return make_select_batch([pool], [240], Nmax=256, label="select D12 W10 pool1011 V240")


def select_batch16(rep: int = 0) -> SelectBatch:
    """16 sequences with depth uniform in [1, 12] (the depth range the size
    policy is trained over, section 4, "Initial Policy Training") and V from a uniform size-policy action, padded to 1024
    pool columns and 256 output rows."""
    rng = rng_for(config_seed(8, rep))
    depths = [int(rng.integers(1, 13)) for _ in range(16)]
    vs = [select_size_action(int(rng.integers(0, 12))) for _ in range(16)]
    pools = [draft_pool(rng, D, 10, 128256) for D in depths]
    return make_select_batch(pools, vs, Vpool=MAX_POOL, Nmax=256,
                             label="select B16 D1-12 W10 V20-240")


# ------------------------------------------------------------ draft policies

LAYOUT_SIZE = 0  # state [D, L, scores of every pool candidate, pad]
LAYOUT_DEPTH = 1  # state [scores of the newest W^2 candidates, D, L]
SIZE_POLICY_DIMS = (2 + 1011, 1024, 256, 12)  # appendix A.2: hidden [1024, 256], 12 actions
DEPTH_POLICY_DIMS = (2 + 100, 1024, 2)  # hidden [1024], CONTINUE / STOP
STATE_PAD = -100.0  # the score written past a pool's end


def policy_layers(rng: np.random.Generator, dims) -> List[tuple]:
    """Random weights of a ReLU network (trained weights are not available):
    per layer W [out][in] and b [out], uniform in +-1/sqrt(in) (the usual
    default initialisation of a fully connected layer), float32."""
    out = []
    for i, o in zip(dims[:-1], dims[1:]):
        k = 1.0 / np.sqrt(i)
        out.append((rng.uniform(-k, k, size=(o, i)).astype(np.float32),
                    rng.uniform(-k, k, size=o).astype(np.float32)))
    return out


@dataclasses.dataclass
class PolicyBatch:
    """Pool scores of B sequences plus their draft depth and context length,
    and a random-weight network of the paper's shape."""
    layout: int
    dims: tuple
    layers: List[tuple]
    scores: np.ndarray  # float32 [B][Vpool]
    pool_size: np.ndarray  # int32 [B]
    depth: np.ndarray  # int32 [B]
    ctx_len: np.ndarray  # int32 [B]
    action_offset: int
    action_scale: int
    label: str = ""
    pool_parents: Optional[np.ndarray] = None  # int32 [B][Vpool] (the pools behind the scores)
    pool_tokens: Optional[np.ndarray] = None  # int32 [B][Vpool]

    @property
    def B(self) -> int:
        return self.scores.shape[0]


def policy_batch(layout: int, B: int, rep: int = 0) -> PolicyBatch:
    """B sequences, each with a depth-D, width-10 draft pool (D uniform in
    [2, 12]) and a context length uniform in [128, 16384]; the size policy's
    actions map to V = 20 + 20 a."""
    rng = rng_for(config_seed(9 + layout, rep) * 100 + B)
    dims = SIZE_POLICY_DIMS if layout == LAYOUT_SIZE else DEPTH_POLICY_DIMS
    layers = policy_layers(rng, dims)
    depths = [int(rng.integers(2, 13)) for _ in range(B)]
    pools = [draft_pool(rng, D, 10, 128256) for D in depths]
    sb = make_select_batch(pools, [1] * B, Vpool=MAX_POOL)
    ctx = rng.integers(128, 16385, size=B).astype(np.int32)
    off, scale = (20, 20) if layout == LAYOUT_SIZE else (0, 1)
    name = "size" if layout == LAYOUT_SIZE else "depth"
    return PolicyBatch(layout, dims, layers, sb.scores, sb.pool_size, np.array(depths, np.int32),
                       ctx, off, scale, label=f"{name} policy B{B} dims {dims}",
                       pool_parents=sb.pool_parents, pool_tokens=sb.pool_tokens)


# ------------------------------------------------------ sampling acceptance

@dataclasses.dataclass
class SamplingBatch:
    """Inputs of acceptance at temperature T: the target logits at every
    node, the draft distribution at every node with children (zeros
    elsewhere), child tokens drawn from it without replacement in ascending
    node order, and the uniforms of every decision."""
    logits: np.ndarray  # float32 [B][Nmax][Voc]
    draft_probs: np.ndarray  # float32 [B][Nmax][Voc]
    draft_tokens: np.ndarray  # int32 [B][Nmax]
    parents: np.ndarray  # int32 [B][Nmax]
    n_nodes: np.ndarray  # int32 [B]
    uniforms: np.ndarray  # float32 [B][Nmax][2] in [0, 1)
    temperature: float
    label: str = ""

    @property
    def B(self) -> int:
        return self.logits.shape[0]


def _softmax_rows(x: np.ndarray) -> np.ndarray:
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def make_sampling_batch(rng: np.random.Generator, trees: List[np.ndarray], Voc: int, *,
                        temperature: float = 1.0, logit_scale: float = 3.0,
                        draft_noise: float = 1.0, Nmax: Optional[int] = None,
                        label: str = "") -> SamplingBatch:
    """Target logits N(0, logit_scale^2); the draft distribution at a node is
    softmax((logits + N(0, draft_noise^2)) / T) (draft_noise = 0: the draft
    equals the target); a node's children take tokens drawn without
    replacement from it (Gumbel top-k), in ascending node order."""
    B = len(trees)
    Nmax = Nmax or max(len(t) for t in trees)
    logits = (rng.standard_normal((B, Nmax, Voc)) * logit_scale).astype(np.float32)
    q = np.zeros((B, Nmax, Voc), np.float32)
    toks = np.zeros((B, Nmax), np.int32)
    par = np.full((B, Nmax), -1, np.int32)
    for b, tr in enumerate(trees):
        n = len(tr)
        par[b, :n] = tr
        for u in range(n):
            kids = [c for c in range(u + 1, n) if tr[c] == u]
            if not kids:
                continue
            noisy = logits[b, u].astype(np.float64)
            if draft_noise > 0:
                noisy = noisy + rng.standard_normal(Voc) * draft_noise
            qu = _softmax_rows(noisy / temperature)
            q[b, u] = qu.astype(np.float32)
            g = np.log(np.maximum(qu, 1e-300)) - np.log(-np.log(rng.random(Voc)))
            order = np.argsort(-g, kind="stable")[:len(kids)]
            toks[b, kids] = order.astype(np.int32)
    uni = np.minimum(rng.random((B, Nmax, 2)), 1.0 - 2.0 ** -24).astype(np.float32)
    return SamplingBatch(logits, q, toks, par, np.array([len(t) for t in trees], np.int32), uni,
                         float(temperature), label)


def sampling_8b(rep: int = 0) -> SamplingBatch:
    """The 8B-shaped step at T = 1: one 60-node Eagle tree (depth 6, top-10)
    over a 128256-token vocabulary."""
    rng = rng_for(config_seed(12, rep))
    t = tree_eagle(rng, 60, 6, 10, 128256)
    return make_sampling_batch(rng, [t.parents], 128256, label="sampling 8B T=1 N60")
