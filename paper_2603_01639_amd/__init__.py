"""ltd_verify: the tree-verification step of Learning-to-Draft speculative
decoding (arXiv 2603.01639, section 3.2) as hand-written HIP kernels for
MI355X (gfx950), behind the C ABI declared in ``include/ltd_verify.h``.

This module is the thin Python binding: it marshals torch device tensors to
raw pointers and calls ``libltdverify.so`` through ctypes.  Every step of the
path runs in the library's kernels; torch only provides device memory and the
current stream.  There is no fallback: if the library is missing, importing
the binding's calls raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libltdverify.so")

LTD_OK = 0
LTD_EINVAL = -1
LTD_EUNSUPPORTED = -2
LTD_EWORKSPACE = -3
LTD_EHIP = -4

DTYPE_F32 = 0
DTYPE_BF16 = 1

STATUS_OK = 0
STATUS_BAD_NNODES = 1
STATUS_BAD_PARENT = 2
STATUS_BAD_PREFIX = 3
STATUS_BAD_BLOCK = 4
STATUS_BAD_PATH = 5
STATUS_BAD_SCORE = 6

MAX_NODES = 256
MAX_POOL = 1024
POLICY_SIZE = 0
POLICY_DEPTH = 1

EXPORTED = (
    "ltd_tree_verify_attn_workspace_size",
    "ltd_tree_verify_attn",
    "ltd_tree_accept_workspace_size",
    "ltd_tree_accept",
    "ltd_kv_compact",
    "ltd_tree_verify_attn_grid",
    "ltd_version",
    "ltd_select_candidates",
    "ltd_policy_workspace_size",
    "ltd_policy_forward",
    "ltd_draft_expand_workspace_size",
    "ltd_draft_expand",
    "ltd_tree_accept_sampling_workspace_size",
    "ltd_tree_accept_sampling",
    "ltd_tree_accept_noalloc_max_bytes",
    "ltd_tree_accept_noalloc",
)


class LtdError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} returned {code}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded HIP library.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python paper_2603_01639_amd/build.py` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
        f32 = ctypes.c_float
        L.ltd_tree_verify_attn_workspace_size.argtypes = [i32] * 7
        L.ltd_tree_verify_attn_workspace_size.restype = sz
        L.ltd_tree_verify_attn.argtypes = [P] * 8 + [i32] * 9 + [f32, i32, P, sz, i32, P, P]
        L.ltd_tree_verify_attn.restype = i32
        L.ltd_tree_accept_workspace_size.argtypes = [i32] * 3
        L.ltd_tree_accept_workspace_size.restype = sz
        L.ltd_tree_accept.argtypes = [P] * 4 + [i32] * 3 + [P] * 5 + [sz, i32, P, P]
        L.ltd_tree_accept.restype = i32
        L.ltd_tree_accept_noalloc_max_bytes.argtypes = []
        L.ltd_tree_accept_noalloc_max_bytes.restype = sz
        L.ltd_tree_accept_noalloc.argtypes = [P] * 4 + [i32] * 3 + [P] * 4 + [i32, P, P]
        L.ltd_tree_accept_noalloc.restype = i32
        L.ltd_kv_compact.argtypes = [P] * 7 + [i32] * 8 + [i64, i32, i32, P, P]
        L.ltd_kv_compact.restype = i32
        L.ltd_tree_verify_attn_grid.argtypes = [i32] * 9
        L.ltd_tree_verify_attn_grid.restype = i32
        L.ltd_select_candidates.argtypes = [P] * 5 + [i32] * 3 + [P] * 5 + [i32, P, P]
        L.ltd_select_candidates.restype = i32
        L.ltd_policy_workspace_size.argtypes = [i32] * 3
        L.ltd_policy_workspace_size.restype = sz
        L.ltd_policy_forward.argtypes = ([i32, P, P, i32, P, P, f32, i32, i32, P, P, i32, P, P, i32,
                                          P, P, i32, i32, i32, P, P, P, sz, P])
        L.ltd_policy_forward.restype = i32
        L.ltd_draft_expand_workspace_size.argtypes = [i32] * 4
        L.ltd_draft_expand_workspace_size.restype = sz
        L.ltd_draft_expand.argtypes = [P, P] + [i32] * 5 + [P] * 4 + [i32, P, P, sz, i32, P, P]
        L.ltd_draft_expand.restype = i32
        L.ltd_tree_accept_sampling_workspace_size.argtypes = [i32] * 3
        L.ltd_tree_accept_sampling_workspace_size.restype = sz
        L.ltd_tree_accept_sampling.argtypes = [P] * 6 + [i32] * 3 + [f32] + [P] * 4 + [sz, i32, P,
                                                                                     P]
        L.ltd_tree_accept_sampling.restype = i32
        L.ltd_version.argtypes = []
        L.ltd_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _p(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return DTYPE_F32
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _check(fn, rc):
    if rc != LTD_OK:
        raise LtdError(fn, rc)


def version() -> str:
    return lib().ltd_version().decode()


def attn_workspace_size(B, Nmax, Hq, Hkv, d, max_prefix, dtype) -> int:
    return int(lib().ltd_tree_verify_attn_workspace_size(B, Nmax, Hq, Hkv, d, max_prefix, dtype))


def attn_grid(B, Nmax, Hq, Hkv, d, max_prefix, dtype, kv_rows, paged=False) -> int:
    """Workgroups of the attention launch; see ``ltd_tree_verify_attn_grid``."""
    return int(lib().ltd_tree_verify_attn_grid(B, Nmax, Hq, Hkv, d, max_prefix, dtype, kv_rows,
                                               int(bool(paged))))


def accept_workspace_size(B, Nmax, Voc) -> int:
    return int(lib().ltd_tree_accept_workspace_size(B, Nmax, Voc))


def _alloc_workspace(nbytes, device):
    import torch
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def tree_verify_attn(q, k_cache, v_cache, prefix_len, parents, n_nodes, out, *, max_prefix: int,
                     block_table=None, num_blocks: int = 0, scale: Optional[float] = None,
                     workspace=None, validate: bool = False, status=None, stream=None):
    """Tree attention; see ``ltd_tree_verify_attn`` in include/ltd_verify.h.

    Tensors are CUDA (HIP) tensors: q/out ``[B][Nmax][Hq][d]``, caches
    contiguous ``[B][Hkv][cap][d]`` or paged ``[num_blocks][Hkv][block][d]``.
    """
    B, Nmax, Hq, d = q.shape
    Hkv = k_cache.shape[1]
    kv_rows = k_cache.shape[2]
    max_blocks = 0 if block_table is None else block_table.shape[1]
    dtype = _dtype_code(q)
    if scale is None:
        scale = d ** -0.5
    if workspace is None:
        workspace = _alloc_workspace(attn_workspace_size(B, Nmax, Hq, Hkv, d, max_prefix, dtype),
                                     q.device)
    rc = lib().ltd_tree_verify_attn(
        _p(q), _p(k_cache), _p(v_cache), _p(block_table), _p(prefix_len), _p(parents), _p(n_nodes),
        _p(out), B, Nmax, Hq, Hkv, d, int(max_prefix), kv_rows, max_blocks, int(num_blocks),
        float(scale), dtype, _p(workspace), workspace.numel() * workspace.element_size(),
        int(validate), _p(status), _stream(stream))
    _check("ltd_tree_verify_attn", rc)
    return out


def tree_accept(logits, draft_tokens, parents, n_nodes, pred, accepted_nodes, out_tokens,
                n_accepted, *, workspace=None, validate: bool = False, status=None, stream=None):
    """Per-node argmax and greedy acceptance; see ``ltd_tree_accept``."""
    B, Nmax, Voc = logits.shape
    if workspace is None:
        workspace = _alloc_workspace(accept_workspace_size(B, Nmax, Voc), logits.device)
    rc = lib().ltd_tree_accept(
        _p(logits), _p(draft_tokens), _p(parents), _p(n_nodes), B, Nmax, Voc, _p(pred),
        _p(accepted_nodes), _p(out_tokens), _p(n_accepted), _p(workspace),
        workspace.numel() * workspace.element_size(), int(validate), _p(status), _stream(stream))
    _check("ltd_tree_accept", rc)


def accept_noalloc_max_bytes() -> int:
    return int(lib().ltd_tree_accept_noalloc_max_bytes())


def tree_accept_noalloc(logits, draft_tokens, parents, n_nodes, pred, accepted_nodes, out_tokens,
                        n_accepted, *, validate: bool = False, status=None, stream=None):
    """Greedy acceptance without a workspace; see ``ltd_tree_accept_noalloc``."""
    B, Nmax, Voc = logits.shape
    rc = lib().ltd_tree_accept_noalloc(
        _p(logits), _p(draft_tokens), _p(parents), _p(n_nodes), B, Nmax, Voc, _p(pred),
        _p(accepted_nodes), _p(out_tokens), _p(n_accepted), int(validate), _p(status),
        _stream(stream))
    _check("ltd_tree_accept_noalloc", rc)


def kv_compact(k_cache, v_cache, prefix_len, new_prefix_len, accepted_nodes, n_accepted, *,
               block_table=None, num_blocks: int = 0, num_layers: int = 1,
               layer_stride_elems: int = 0, validate: bool = False, status=None, stream=None):
    """In-place KV compaction; see ``ltd_kv_compact``.

    With ``num_layers > 1`` the caches hold the layers ``layer_stride_elems``
    elements apart and the last three dims are ``[Hkv][rows][d]``.
    """
    B, Nmax = accepted_nodes.shape
    Hkv, kv_rows, d = k_cache.shape[-3], k_cache.shape[-2], k_cache.shape[-1]
    max_blocks = 0 if block_table is None else block_table.shape[1]
    rc = lib().ltd_kv_compact(
        _p(k_cache), _p(v_cache), _p(block_table), _p(prefix_len), _p(new_prefix_len),
        _p(accepted_nodes), _p(n_accepted), B, Nmax, Hkv, d, kv_rows, max_blocks, int(num_blocks),
        int(num_layers), int(layer_stride_elems), _dtype_code(k_cache), int(validate), _p(status),
        _stream(stream))
    _check("ltd_kv_compact", rc)


def select_candidates(scores, pool_parents, pool_tokens, pool_size, n_select, parents, tokens,
                      n_nodes, *, selected=None, depth=None, validate: bool = False, status=None,
                      stream=None):
    """Candidate token selection; see ``ltd_select_candidates``.  Pools are
    ``[B][Vpool]``, outputs ``[B][Nmax]`` int32 CUDA (HIP) tensors."""
    B, Vpool = scores.shape
    Nmax = parents.shape[1]
    rc = lib().ltd_select_candidates(
        _p(scores), _p(pool_parents), _p(pool_tokens), _p(pool_size), _p(n_select), B, Vpool, Nmax,
        _p(selected), _p(parents), _p(tokens), _p(depth), _p(n_nodes), int(validate), _p(status),
        _stream(stream))
    _check("ltd_select_candidates", rc)


def policy_workspace_size(B, h1, h2) -> int:
    return int(lib().ltd_policy_workspace_size(B, h1, h2))


def policy_forward(layout, scores, pool_size, depth, ctx_len, layers, logits, action, *,
                   pad: float = -100.0, action_offset: int = 0, action_scale: int = 1,
                   workspace=None, stream=None):
    """Draft-policy inference; see ``ltd_policy_forward``.  ``layers`` is a
    list of (W [out][in], b [out]) float32 CUDA tensors: two or three layers
    (one or two hidden ReLU layers, then the output layer)."""
    if len(layers) not in (2, 3):
        raise ValueError("a policy has one or two hidden layers")
    B, Vpool = scores.shape
    (w1, b1), *mid, (wo, bo) = layers
    w2, b2 = mid[0] if mid else (None, None)
    h1 = w1.shape[0]
    h2 = 0 if w2 is None else w2.shape[0]
    if workspace is None:
        workspace = _alloc_workspace(policy_workspace_size(B, h1, h2), scores.device)
    rc = lib().ltd_policy_forward(
        int(layout), _p(scores), _p(pool_size), Vpool, _p(depth), _p(ctx_len), float(pad), B,
        w1.shape[1], _p(w1), _p(b1), h1, _p(w2), _p(b2), h2, _p(wo), _p(bo), wo.shape[0],
        int(action_offset), int(action_scale), _p(logits), _p(action), _p(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream))
    _check("ltd_policy_forward", rc)


def draft_expand_workspace_size(B, F, Voc, W) -> int:
    return int(lib().ltd_draft_expand_workspace_size(B, F, Voc, W))


def draft_expand(logits, frontier, scores, pool_parents, pool_tokens, pool_size, new_frontier, *,
                 W: int, workspace=None, validate: bool = False, status=None, stream=None):
    """One round of draft tree expansion; see ``ltd_draft_expand``.  logits
    ``[B][F][Voc]`` float32, pool arrays ``[B][Vpool]`` (updated in place),
    new_frontier ``[B][W_next]``."""
    B, F, Voc = logits.shape
    Vpool = scores.shape[1]
    if workspace is None:
        workspace = _alloc_workspace(draft_expand_workspace_size(B, F, Voc, W), logits.device)
    rc = lib().ltd_draft_expand(
        _p(logits), _p(frontier), B, F, Voc, int(W), new_frontier.shape[1], _p(scores),
        _p(pool_parents), _p(pool_tokens), _p(pool_size), Vpool, _p(new_frontier), _p(workspace),
        workspace.numel() * workspace.element_size(), int(validate), _p(status), _stream(stream))
    _check("ltd_draft_expand", rc)


def accept_sampling_workspace_size(B, Nmax, Voc) -> int:
    return int(lib().ltd_tree_accept_sampling_workspace_size(B, Nmax, Voc))


def tree_accept_sampling(logits, draft_probs, draft_tokens, parents, n_nodes, uniforms,
                         accepted_nodes, out_tokens, n_accepted, *, temperature: float = 1.0,
                         workspace=None, validate: bool = False, status=None, stream=None):
    """Acceptance by recursive rejection sampling at temperature T > 0; see
    ``ltd_tree_accept_sampling``."""
    B, Nmax, Voc = logits.shape
    if workspace is None:
        workspace = _alloc_workspace(accept_sampling_workspace_size(B, Nmax, Voc), logits.device)
    rc = lib().ltd_tree_accept_sampling(
        _p(logits), _p(draft_probs), _p(draft_tokens), _p(parents), _p(n_nodes), _p(uniforms), B,
        Nmax, Voc, float(temperature), _p(accepted_nodes), _p(out_tokens), _p(n_accepted),
        _p(workspace), workspace.numel() * workspace.element_size(), int(validate), _p(status),
        _stream(stream))
    _check("ltd_tree_accept_sampling", rc)
