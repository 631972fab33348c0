"""CPU oracle for the tree-verification step (arXiv 2603.01639, section 3.2).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It wraps the plain
fp64 C library ``libltdoracle.so`` (``ltd_oracle.c``) with numpy-array calls.
It shares no code with the HIP library, and the HIP library never reaches it.

Every function takes host numpy arrays in the same layouts as the GPU contract:

* ``q``: ``[B][Nmax][Hq][d]``, float32 or bf16 bit patterns (uint16);
* ``k_cache``/``v_cache``: contiguous ``[B][Hkv][cap][d]`` or paged
  ``[num_blocks][Hkv][block_size][d]`` with ``block_table`` ``[B][max_blocks]``;
* ``parents``: ``[B][Nmax]`` int32 with ``parents[b][0] == -1``.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libltdoracle.so")

DTYPE_F32 = 0
DTYPE_BF16 = 1

STATUS_BAD_NNODES = 1
STATUS_BAD_PARENT = 2
STATUS_BAD_PREFIX = 3
STATUS_BAD_BLOCK = 4
STATUS_BAD_PATH = 5
STATUS_BAD_SCORE = 6


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle returned {code}")
        self.code = code


_lib = None


def load_library(path: str) -> ctypes.CDLL:
    """Open an oracle build at ``path`` and declare its signatures."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32 = ctypes.c_int
    lib.ltd_oracle_tree_verify_attn.argtypes = [P, P, P, P, P, P, P, P, P, i32, i32, i32, i32,
                                                i32, i32, i32, i32, ctypes.c_double, i32]
    lib.ltd_oracle_tree_verify_attn.restype = i32
    lib.ltd_oracle_tree_accept.argtypes = [P, P, P, P, i32, i32, i32, P, P, P, P]
    lib.ltd_oracle_tree_accept.restype = i32
    lib.ltd_oracle_kv_compact.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, i32, i32, i32,
                                          i32, i32, ctypes.c_int64, i32]
    lib.ltd_oracle_kv_compact.restype = i32
    lib.ltd_oracle_select_candidates.argtypes = [P, P, P, P, P, i32, i32, i32, P, P, P, P, P]
    lib.ltd_oracle_select_candidates.restype = i32
    lib.ltd_oracle_draft_expand.argtypes = [P, P, i32, i32, i32, i32, i32, P, P, P, P, i32, P]
    lib.ltd_oracle_draft_expand.restype = i32
    lib.ltd_oracle_tree_accept_sampling.argtypes = [P, P, P, P, P, P, i32, i32, i32, ctypes.c_double,
                                                     P, P, P, P, P]
    lib.ltd_oracle_tree_accept_sampling.restype = i32
    lib.ltd_oracle_num_threads.argtypes = []
    lib.ltd_oracle_num_threads.restype = i32
    lib.ltd_oracle_set_num_threads.argtypes = [i32]
    lib.ltd_oracle_set_num_threads.restype = None
    return lib


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("LTD_ORACLE_LIB") or LIB_PATH  # e.g. the sanitizer build
        if not os.path.exists(path):
            from . import build as _build
            _build.build()
        _lib = load_library(path)
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return int(_load().ltd_oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads for the oracle's OpenMP loops from now on (timing only)."""
    _load().ltd_oracle_set_num_threads(int(n))


def tree_verify_attn(q, k_cache, v_cache, prefix_len, parents, n_nodes, *, Hkv, block_table=None,
                     num_blocks=0, scale=None, dtype=DTYPE_BF16, out=None, node_mask=None):
    """fp64 tree attention.  Returns ``out`` ``[B][Nmax][Hq][d]`` float64.

    Rows ``i >= n_nodes[b]`` (and rows outside ``node_mask`` when it is given)
    are left as they were in ``out`` (zeros if not given).
    """
    lib = _load()
    elem = np.float32 if dtype == DTYPE_F32 else np.uint16
    q = _c(q, elem)
    k_cache = _c(k_cache, elem)
    v_cache = _c(v_cache, elem)
    B, Nmax, Hq, d = q.shape
    prefix_len = _c(prefix_len, np.int32)
    parents = _c(parents, np.int32)
    n_nodes = _c(n_nodes, np.int32)
    block_table = _c(block_table, np.int32)
    if block_table is None:
        kv_rows = k_cache.shape[2]
        max_blocks = 0
    else:
        kv_rows = k_cache.shape[2]
        max_blocks = block_table.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    node_mask = _c(node_mask, np.uint8)
    if out is None:
        out = np.zeros((B, Nmax, Hq, d), dtype=np.float64)
    rc = lib.ltd_oracle_tree_verify_attn(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                         _ptr(prefix_len), _ptr(parents), _ptr(n_nodes),
                                         _ptr(node_mask), _ptr(out),
                                         B, Nmax, Hq, Hkv, d, kv_rows, max_blocks, num_blocks,
                                         float(scale), dtype)
    if rc != 0:
        raise OracleError(rc)
    return out


def tree_accept(logits, draft_tokens, parents, n_nodes):
    """Greedy acceptance.  Returns ``(pred, accepted_nodes, out_tokens, n_accepted)``.

    Entries past ``n_nodes[b]`` (pred) or past ``n_accepted[b]`` (path, tokens)
    are -1.
    """
    lib = _load()
    logits = _c(logits, np.float32)
    B, Nmax, Voc = logits.shape
    draft_tokens = _c(draft_tokens, np.int32)
    parents = _c(parents, np.int32)
    n_nodes = _c(n_nodes, np.int32)
    pred = np.full((B, Nmax), -1, np.int32)
    acc = np.full((B, Nmax), -1, np.int32)
    toks = np.full((B, Nmax), -1, np.int32)
    n_acc = np.zeros((B,), np.int32)
    rc = lib.ltd_oracle_tree_accept(_ptr(logits), _ptr(draft_tokens), _ptr(parents), _ptr(n_nodes),
                                    B, Nmax, Voc, _ptr(pred), _ptr(acc), _ptr(toks), _ptr(n_acc))
    if rc != 0:
        raise OracleError(rc)
    return pred, acc, toks, n_acc


def kv_compact(k_cache, v_cache, prefix_len, accepted_nodes, n_accepted, *, Hkv, block_table=None,
               num_blocks=0, num_layers=1, layer_stride_elems=0):
    """In-place compaction of ``k_cache``/``v_cache`` (numpy, modified).

    ``k_cache``/``v_cache`` hold ``num_layers`` layers ``layer_stride_elems``
    elements apart; each layer has the single-layer layout.  Returns the new
    prefix lengths.
    """
    lib = _load()
    assert k_cache.flags["C_CONTIGUOUS"] and v_cache.flags["C_CONTIGUOUS"]
    assert k_cache.dtype == v_cache.dtype and k_cache.dtype in (np.float32, np.uint16)
    elem_bytes = k_cache.dtype.itemsize
    prefix_len = _c(prefix_len, np.int32)
    accepted_nodes = _c(accepted_nodes, np.int32)
    n_accepted = _c(n_accepted, np.int32)
    block_table = _c(block_table, np.int32)
    B, Nmax = accepted_nodes.shape
    d = k_cache.shape[-1]
    kv_rows = k_cache.shape[-2]
    max_blocks = 0 if block_table is None else block_table.shape[1]
    new_len = np.zeros((B,), np.int32)
    rc = lib.ltd_oracle_kv_compact(_ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(prefix_len),
                                   _ptr(new_len), _ptr(accepted_nodes), _ptr(n_accepted), B, Nmax,
                                   Hkv, d, kv_rows, max_blocks, num_blocks, num_layers,
                                   int(layer_stride_elems), elem_bytes)
    if rc != 0:
        raise OracleError(rc)
    return new_len


def select_candidates(scores, pool_parents, pool_tokens, pool_size, n_select, Nmax):
    """Candidate token selection (section 3.2): the V = min(n_select, pool
    size) candidates of highest cumulative score (equal scores: lower pool
    index first), flattened in pool order.  Returns (selected, parents,
    tokens, depth, n_nodes); entries past V hold -1."""
    scores = np.ascontiguousarray(scores, np.float32)
    B, Vpool = scores.shape
    pool_parents = np.ascontiguousarray(pool_parents, np.int32)
    pool_tokens = np.ascontiguousarray(pool_tokens, np.int32)
    pool_size = np.ascontiguousarray(pool_size, np.int32)
    n_select = np.ascontiguousarray(n_select, np.int32)
    outs = [np.full((B, Nmax), -1, np.int32) for _ in range(4)]
    n_nodes = np.zeros(B, np.int32)
    rc = _load().ltd_oracle_select_candidates(
        _ptr(scores), _ptr(pool_parents), _ptr(pool_tokens), _ptr(pool_size), _ptr(n_select),
        B, Vpool, Nmax, *[_ptr(o) for o in outs], _ptr(n_nodes))
    if rc != 0:
        raise OracleError(rc)
    return (*outs, n_nodes)


def draft_expand(logits, frontier, scores, pool_parents, pool_tokens, pool_size, *, W, W_next):
    """One round of draft tree expansion (section 3.2, "Draft Tree
    Generation"), in place on copies of the pool arrays.  Returns (scores,
    pool_parents, pool_tokens, pool_size, new_frontier)."""
    logits = np.ascontiguousarray(logits, np.float32)
    B, F, Voc = logits.shape
    frontier = np.ascontiguousarray(frontier, np.int32)
    scores = np.array(scores, np.float32, copy=True)
    pool_parents = np.array(pool_parents, np.int32, copy=True)
    pool_tokens = np.array(pool_tokens, np.int32, copy=True)
    pool_size = np.array(pool_size, np.int32, copy=True)
    Vpool = scores.shape[1]
    new_frontier = np.full((B, W_next), -1, np.int32)
    rc = _load().ltd_oracle_draft_expand(
        _ptr(logits), _ptr(frontier), B, F, Voc, W, W_next, _ptr(scores), _ptr(pool_parents),
        _ptr(pool_tokens), _ptr(pool_size), Vpool, _ptr(new_frontier))
    if rc != 0:
        raise OracleError(rc)
    return scores, pool_parents, pool_tokens, pool_size, new_frontier


def tree_accept_sampling(logits, draft_probs, draft_tokens, parents, n_nodes, uniforms, *,
                         temperature=1.0, want_final=False):
    """Acceptance by recursive rejection sampling at temperature T > 0.
    Returns (accepted_nodes, out_tokens, n_accepted, min_margin) and, with
    want_final, the distribution each bonus token was drawn from."""
    logits = np.ascontiguousarray(logits, np.float32)
    B, Nmax, Voc = logits.shape
    draft_probs = np.ascontiguousarray(draft_probs, np.float32)
    draft_tokens = np.ascontiguousarray(draft_tokens, np.int32)
    parents = np.ascontiguousarray(parents, np.int32)
    n_nodes = np.ascontiguousarray(n_nodes, np.int32)
    uniforms = np.ascontiguousarray(uniforms, np.float32)
    acc = np.full((B, Nmax), -1, np.int32)
    toks = np.full((B, Nmax), -1, np.int32)
    n_acc = np.zeros(B, np.int32)
    margin = np.zeros(B, np.float64)
    final = np.zeros((B, Voc), np.float64) if want_final else None
    rc = _load().ltd_oracle_tree_accept_sampling(
        _ptr(logits), _ptr(draft_probs), _ptr(draft_tokens), _ptr(parents), _ptr(n_nodes),
        _ptr(uniforms), B, Nmax, Voc, float(temperature), _ptr(acc), _ptr(toks), _ptr(n_acc),
        _ptr(final), _ptr(margin))
    if rc != 0:
        raise OracleError(rc)
    return (acc, toks, n_acc, margin, final) if want_final else (acc, toks, n_acc, margin)
