"""Host logic of bench.py (no GPU): the binding roof, the algorithmic byte
and FLOP counts of the workloads, the traffic lines and their source hashes."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import workloads as W  # noqa: E402


def test_binding_roof_hbm_and_mfma():
    # 9.6 MB and 2.0 GFLOP: 1.2 us at 8 TB/s against 0.8 us at 2.5 PFLOP/s -> HBM
    r = bench.binding_roof("tree_verify_attn", 9_600_000, 2.0e9, 12.0)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert r["frac"] == pytest.approx(1.2 / 12.0, abs=1e-4)
    assert r["achieved"] == pytest.approx(800.0, abs=0.1)
    # 360 MB and 199 GFLOP: 45 us against 79.6 us -> MFMA
    r = bench.binding_roof("tree_verify_attn", 360e6, 199e9, 446.0)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert r["frac"] == pytest.approx(79.6 / 446.0, abs=1e-3)
    assert r["achieved"] == pytest.approx(199e9 / 446e-6 / 1e12, abs=0.01)
    # no FLOPs (acceptance) is always HBM
    assert bench.binding_roof("tree_accept", 30.8e6, 0, 11.0)["bound"] == "hbm"


def test_algorithmic_bytes_of_the_8b_step():
    """The 8B-shaped step (bf16, prefix 2048, 60 nodes, 32/8 heads, d = 128,
    vocab 128256): 9.62 MB for attention (8.39 MB of prefix K/V, tree K/V, Q
    and O), 30.78 MB of logits for acceptance, 2.01 GFLOP for the prefix."""
    b = W.config2_8b(0, with_logits=False)
    attn, accept, flops = bench.algorithmic_bytes(b)
    assert attn == 8_388_608 + 245_760 + 2 * 491_520
    assert accept == 60 * 128_256 * 4
    assert flops == 4 * 32 * 60 * 2048 * 128


def test_traffic_lines_follow_the_sources(tmp_path):
    digest = bench.source_digest("tree_verify_attn")
    p = tmp_path / "t.txt"
    p.write_text(f"traffic c2 tree_verify_attn 123 {digest}\n"
                 f"traffic c3 tree_verify_attn 456 0000000000000000\n")
    assert bench.read_traffic(str(p), "c2", "tree_verify_attn") == 123
    assert bench.read_traffic(str(p), "c3", "tree_verify_attn") is None  # stale hash
    assert bench.read_traffic(str(p), "c5", "tree_verify_attn") is None  # no line
    assert bench.read_traffic(str(tmp_path / "missing.txt"), "c2", "tree_verify_attn") is None
