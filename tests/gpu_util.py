"""Helpers for the GPU parity tests: move a generated batch to the device, run
the three library calls, run the oracle on the same host arrays, compare."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np

import oracle
import paper_2603_01639_amd as ltd
import workloads as W

ATOL = {W.DTYPE_F32: 1e-5, W.DTYPE_BF16: 2e-2}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _torch():
    import torch
    return torch


def to_dev(a, dtype=None):
    torch = _torch()
    if a is None:
        return None
    if a.dtype == np.uint16:  # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to("cuda").view(torch.bfloat16)
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to("cuda") if dtype is None else t.to("cuda", dtype)


def to_host(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def as_f64(a, dtype):
    return (W.bf16_bits_to_f32(a) if dtype == W.DTYPE_BF16 else a).astype(np.float64)


@dataclasses.dataclass
class DevBatch:
    q: object
    k: object
    v: object
    prefix_len: object
    parents: object
    n_nodes: object
    tokens: object
    logits: object
    block_table: object


def upload(b: W.VerifyBatch) -> DevBatch:
    return DevBatch(q=to_dev(b.q), k=to_dev(b.k_cache), v=to_dev(b.v_cache),
                    prefix_len=to_dev(b.prefix_len), parents=to_dev(b.parents),
                    n_nodes=to_dev(b.n_nodes), tokens=to_dev(b.draft_tokens),
                    logits=None if b.logits is None else to_dev(b.logits),
                    block_table=to_dev(b.block_table))


def gpu_attention(b: W.VerifyBatch, dev: DevBatch, fill=0.0, validate=False, status=None):
    torch = _torch()
    out = torch.full(tuple(b.q.shape), fill, dtype=dev.q.dtype, device="cuda")
    ltd.tree_verify_attn(dev.q, dev.k, dev.v, dev.prefix_len, dev.parents, dev.n_nodes, out,
                         max_prefix=b.max_prefix, block_table=dev.block_table,
                         num_blocks=b.num_blocks, validate=validate, status=status)
    torch.cuda.synchronize()
    return to_host(out)


def oracle_attention(b: W.VerifyBatch):
    return oracle.tree_verify_attn(b.q, b.k_cache, b.v_cache, b.prefix_len, b.parents, b.n_nodes,
                                   Hkv=b.Hkv, block_table=b.block_table, num_blocks=b.num_blocks,
                                   dtype=b.dtype)


def compare_attention(b: W.VerifyBatch, got, want):
    """Max-abs error over every written row (all nodes < n_nodes[b], every
    head, every dim); asserts within the tolerance."""
    g = as_f64(got, b.dtype)
    err = 0.0
    for s in range(b.B):
        n = int(b.n_nodes[s])
        e = np.abs(g[s, :n] - want[s, :n]).max()
        err = max(err, float(e))
    assert np.isfinite(err) and err <= ATOL[b.dtype], f"{b.label}: max abs err {err}"
    return err


def gpu_accept(b: W.VerifyBatch, dev: DevBatch, validate=False, status=None):
    torch = _torch()
    B, Nmax = b.B, b.Nmax
    pred = torch.full((B, Nmax), -1, dtype=torch.int32, device="cuda")
    acc = torch.full((B, Nmax), -1, dtype=torch.int32, device="cuda")
    toks = torch.full((B, Nmax), -1, dtype=torch.int32, device="cuda")
    nacc = torch.zeros((B,), dtype=torch.int32, device="cuda")
    ltd.tree_accept(dev.logits, dev.tokens, dev.parents, dev.n_nodes, pred, acc, toks, nacc,
                    validate=validate, status=status)
    torch.cuda.synchronize()
    return pred.cpu().numpy(), acc.cpu().numpy(), toks.cpu().numpy(), nacc.cpu().numpy()


def check_accept(b: W.VerifyBatch, got):
    want = oracle.tree_accept(b.logits, b.draft_tokens, b.parents, b.n_nodes)
    pred, acc, toks, nacc = got
    wpred, wacc, wtoks, wnacc = want
    np.testing.assert_array_equal(nacc, wnacc)
    for s in range(b.B):
        n, k = int(b.n_nodes[s]), int(wnacc[s])
        np.testing.assert_array_equal(pred[s, :n], wpred[s, :n])
        np.testing.assert_array_equal(acc[s, :k], wacc[s, :k])
        np.testing.assert_array_equal(toks[s, :k], wtoks[s, :k])
        assert (pred[s, n:] == -1).all() and (acc[s, k:] == -1).all() and (toks[s, k:] == -1).all()
    return want


def gpu_compact(b: W.VerifyBatch, dev: DevBatch, acc, nacc, validate=False, status=None):
    torch = _torch()
    new_len = torch.full((b.B,), -7, dtype=torch.int32, device="cuda")
    ltd.kv_compact(dev.k, dev.v, dev.prefix_len, new_len, to_dev(acc), to_dev(nacc),
                   block_table=dev.block_table, num_blocks=b.num_blocks, validate=validate,
                   status=status)
    torch.cuda.synchronize()
    return new_len.cpu().numpy()


def check_compact(b: W.VerifyBatch, dev: DevBatch, acc, nacc):
    new_len = gpu_compact(b, dev, acc, nacc)
    k, v = b.k_cache.copy(), b.v_cache.copy()
    want_len = oracle.kv_compact(k, v, b.prefix_len, acc, nacc, Hkv=b.Hkv,
                                 block_table=b.block_table, num_blocks=b.num_blocks)
    np.testing.assert_array_equal(new_len, want_len)
    np.testing.assert_array_equal(to_host(dev.k), k)
    np.testing.assert_array_equal(to_host(dev.v), v)
