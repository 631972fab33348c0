"""The C-ABI library loads on the CPU and exports every symbol its header
declares; host-only queries work without a GPU (no kernels are launched)."""
import os
import re

import pytest

import paper_2603_01639_amd as ltd

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "ltd_verify.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ltd_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_three_steps_and_the_selection():
    names = _declared()
    for fn in ("ltd_tree_verify_attn", "ltd_tree_accept", "ltd_kv_compact",
               "ltd_select_candidates"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    lib = ltd.lib()
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(ltd.EXPORTED)


def test_version_and_workspace_queries():
    assert "gfx950" in ltd.version()
    assert ltd.accept_workspace_size(1, 60, 128256) == 1 * 60 * 8 * 8
    assert ltd.accept_workspace_size(1, 300, 10) == 0  # Nmax above the node limit
    assert ltd.attn_workspace_size(1, 60, 32, 8, 96, 2048, ltd.DTYPE_BF16) == 0  # unsupported d
    assert ltd.attn_grid(1, 60, 32, 8, 128, 2048, ltd.DTYPE_BF16, 0) == -1  # kv_rows < 1
    assert ltd.attn_grid(1, 300, 32, 8, 128, 2048, ltd.DTYPE_BF16, 4096) == -1  # Nmax > 256


def test_library_links_only_hip_runtime():
    """The product library must not reach the oracle."""
    data = open(ltd.LIB_PATH, "rb").read()
    assert b"ltd_oracle" not in data


def _prototypes():
    """{name: number of parameters} from the header's declarations."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    out = {}
    for m in re.finditer(r"\b(ltd_[a-z_0-9]+)\s*\(([^)]*)\)\s*;", text):
        params = [p for p in m.group(2).split(",") if p.strip() and p.strip() != "void"]
        out[m.group(1)] = len(params)
    return out


def test_binding_signatures_match_header():
    lib = ltd.lib()
    protos = _prototypes()
    assert set(protos) == set(ltd.EXPORTED)
    for name, nparams in protos.items():
        assert len(getattr(lib, name).argtypes) == nparams, name


def test_bf16_head128_workloads_plan_the_mfma_grid():
    """bf16 head_dim 128 shapes run on the MFMA kernels.  A single sequence
    takes the split plan: grid (kv heads, row tiles, KV splits), e.g. the
    8B-shaped step at prefix 2048 cuts each kv head's prefix into 16 splits of
    two key tiles and gives the 60-node tree a split of its own (8 x 17
    workgroups).  A batch takes the stream plan: a power of two of at least 8
    workgroups (one eighth of the work per XCD), at most one per compute unit,
    two partial slots each.  bf16 head_dim 64 takes the same plans as 128;
    fp32 runs on the row-wise kernel (grid 0, no workspace)."""
    assert ltd.attn_grid(1, 60, 32, 8, 128, 2048, ltd.DTYPE_BF16, 2108) == 8 * 17
    for P, N, Hq in ((16384, 60, 32), (4096, 256, 64), (4096, 8, 64)):
        g = ltd.attn_grid(1, N, Hq, 8, 128, P, ltd.DTYPE_BF16, P + N)
        assert g > 8 and g % 8 == 0, (P, N, Hq, g)
        assert ltd.attn_workspace_size(1, N, Hq, 8, 128, P, ltd.DTYPE_BF16) > 0
    slot = 256 * (128 * 2 + 8)
    for B, Nmax, Hq, Hkv, P, W in ((16, 128, 64, 8, 8192, 256), (2, 60, 32, 8, 2048, 256),
                                   (2, 1, 8, 8, 0, 8)):
        g = ltd.attn_grid(B, Nmax, Hq, Hkv, 128, P, ltd.DTYPE_BF16, P + Nmax)
        assert g == W, (B, Nmax, Hq, Hkv, P, g)
        assert g == ltd.attn_grid(B, Nmax, Hq, Hkv, 128, P, ltd.DTYPE_BF16, 16, paged=True)
        assert ltd.attn_workspace_size(B, Nmax, Hq, Hkv, 128, P, ltd.DTYPE_BF16) >= 2 * g * slot
    # blocks so small that a stream share could span more block ids than the
    # LDS table holds: the split plan takes the batch (grid kv heads x row
    # tiles x splits, not a power of two)
    g = ltd.attn_grid(2, 64, 8, 8, 128, 400000, ltd.DTYPE_BF16, 1, paged=True)
    assert g > 0 and g % 16 == 0 and g & (g - 1) != 0
    assert ltd.attn_grid(2, 64, 8, 8, 128, 200000, ltd.DTYPE_BF16, 16, paged=True) == 256
    assert ltd.attn_grid(1, 16, 8, 8, 64, 128, ltd.DTYPE_F32, 144) == 0
    for B, P in ((1, 128), (1, 2048), (3, 2048)):
        g64 = ltd.attn_grid(B, 16, 8, 8, 64, P, ltd.DTYPE_BF16, P + 16)
        assert g64 > 0 and g64 == ltd.attn_grid(B, 16, 8, 8, 128, P, ltd.DTYPE_BF16, P + 16)
    assert ltd.attn_workspace_size(1, 16, 8, 8, 64, 128, ltd.DTYPE_F32) == 0


@pytest.mark.parametrize("scale", [0.0, -0.125, float("nan"), float("inf")])
def test_attention_rejects_a_scale_that_is_not_positive_and_finite(scale):
    """The softmax scale must be finite and > 0; anything else is refused on
    the host before any pointer is touched or kernel launched (the pointers
    here are dummies)."""
    P = 0x1000  # never dereferenced: the call returns before using them
    rc = ltd.lib().ltd_tree_verify_attn(P, P, P, None, P, P, P, P, 1, 4, 8, 2, 128, 64, 128, 0, 0,
                                        scale, ltd.DTYPE_BF16, None, 0, 0, None, None)
    assert rc == ltd.LTD_EINVAL


@pytest.mark.parametrize("B,Vpool,Nmax,validate,status", [
    (-1, 411, 60, 0, None), (1, 0, 60, 0, None), (1, ltd.MAX_POOL + 1, 60, 0, None),
    (1, 411, 0, 0, None), (1, 411, ltd.MAX_NODES + 1, 0, None), (1, 411, 60, 1, None)])
def test_selection_rejects_bad_scalar_arguments(B, Vpool, Nmax, validate, status):
    """Pool width, output rows, batch size and a missing status buffer are
    checked on the host before anything is launched (dummy pointers)."""
    P = 0x1000
    rc = ltd.lib().ltd_select_candidates(P, P, P, P, P, B, Vpool, Nmax, P, P, P, P, P, validate,
                                         status, None)
    assert rc == ltd.LTD_EINVAL


def test_selection_of_an_empty_batch_launches_nothing():
    assert ltd.lib().ltd_select_candidates(None, None, None, None, None, 0, 1024, 256, None, None,
                                           None, None, None, 0, None, None) == ltd.LTD_OK
    P = 0x1000  # a required output missing
    assert ltd.lib().ltd_select_candidates(P, P, P, P, P, 1, 16, 16, P, None, P, P, P, 0, None,
                                           None) == ltd.LTD_EINVAL


@pytest.mark.parametrize("args", [
    dict(layout=2), dict(B=-1), dict(Vpool=0), dict(in_dim=2), dict(in_dim=1025), dict(h1=0),
    dict(h1=1025), dict(h2=-1), dict(h2=1025), dict(n_out=0), dict(n_out=65)])
def test_policy_rejects_bad_scalar_arguments(args):
    P = 0x1000
    a = dict(layout=0, B=2, Vpool=1024, in_dim=1013, h1=1024, h2=256, n_out=12)
    a.update(args)
    rc = ltd.lib().ltd_policy_forward(a["layout"], P, P, a["Vpool"], P, P, -100.0, a["B"],
                                      a["in_dim"], P, P, a["h1"], P, P, a["h2"], P, P, a["n_out"],
                                      20, 20, P, P, P, 1 << 30, None)
    assert rc == ltd.LTD_EINVAL


def test_policy_workspace_and_missing_buffers():
    assert ltd.policy_workspace_size(16, 1024, 256) == 16 * (1024 + 256) * 4
    assert ltd.policy_workspace_size(1, 1024, 0) == 1024 * 4
    P = 0x1000
    # h2 > 0 needs w2/b2; too small a workspace is LTD_EWORKSPACE
    assert ltd.lib().ltd_policy_forward(0, P, P, 16, P, P, 0.0, 1, 10, P, P, 8, None, None, 4, P,
                                        P, 2, 0, 1, P, P, P, 1 << 20, None) == ltd.LTD_EINVAL
    assert ltd.lib().ltd_policy_forward(0, P, P, 16, P, P, 0.0, 1, 10, P, P, 8, P, P, 4, P, P, 2,
                                        0, 1, P, P, P, 4, None) == ltd.LTD_EWORKSPACE


@pytest.mark.parametrize("B,F,Voc,W,W_next", [
    (-1, 1, 100, 4, 4), (1, 0, 100, 4, 4), (1, 1, 100, 0, 1), (1, 1, 100, 17, 4), (1, 1, 3, 4, 4),
    (1, 1, 64 * 4096 + 1, 4, 4), (1, 17, 100, 16, 4), (1, 2, 100, 4, 9), (1, 2, 100, 4, 0)])
def test_draft_expand_rejects_bad_scalar_arguments(B, F, Voc, W, W_next):
    P = 0x1000
    rc = ltd.lib().ltd_draft_expand(P, P, B, F, Voc, W, W_next, P, P, P, P, 64, P, P, 1 << 30, 0,
                                    None, None)
    assert rc == ltd.LTD_EINVAL


def test_draft_expand_workspace():
    assert ltd.draft_expand_workspace_size(2, 10, 128256, 10) == 2 * 10 * 32 * (8 * 10 + 8)
    assert ltd.draft_expand_workspace_size(1, 1, 64 * 4096 + 1, 4) == 0


@pytest.mark.parametrize("args", [dict(B=-1), dict(Nmax=0), dict(Nmax=257), dict(Voc=0),
                                  dict(Voc=64 * 4096 + 1), dict(T=0.0), dict(T=-1.0),
                                  dict(T=float("inf")), dict(T=float("nan"))])
def test_sampling_rejects_bad_scalar_arguments(args):
    P = 0x1000
    a = dict(B=1, Nmax=60, Voc=128256, T=1.0)
    a.update(args)
    rc = ltd.lib().ltd_tree_accept_sampling(P, P, P, P, P, P, a["B"], a["Nmax"], a["Voc"], a["T"],
                                            P, P, P, P, 1 << 30, 0, None, None)
    assert rc == ltd.LTD_EINVAL


def test_sampling_workspace():
    # per node and 4096-token chunk: a softmax partial (16 bytes) and the
    # residual masses after the node's first three rejections (doubles)
    assert ltd.accept_sampling_workspace_size(1, 60, 128256) == 60 * 32 * (16 + 3 * 16)
