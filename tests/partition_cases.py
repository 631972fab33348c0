"""Batches (two or more sequences, the stream plan's domain) that exercise the
attention launch's work partition on the GPU:
between them they hold a share that is a tree block alone, workgroups with
nothing to do, units written whole and units cut into many pieces (checked on
the host by test_host_stream_plan.py, run through parity by
test_gpu_parity.py).  Plain data: shapes, prefix lengths and node counts."""
import dataclasses
from typing import List


@dataclasses.dataclass
class Case:
    label: str
    Hq: int
    Hkv: int
    Nmax: int
    prefix: List[int]
    nodes: List[int]


CASES = [
    # tiny sequences: fewer items than the smallest grid
    Case("tiny P=0 N=1 x2", 8, 8, 1, [0, 0], [1, 1]),
    Case("tiny P=5 N=3 x3", 8, 2, 3, [5, 0, 2], [3, 1, 2]),
    # sized for 256-node trees, given 1-node trees: most workgroups get nothing
    Case("Nmax 256, N=1 x2", 64, 8, 256, [0, 3], [1, 1]),
    # 8B-shaped, prefix around 2048: a few tiles per workgroup
    Case("8B P2048 N60 x2", 32, 8, 60, [2048, 2048], [60, 60]),
    Case("8B P1999 N128 + P2100 N9", 32, 8, 128, [1999, 2100], [128, 9]),
    # long prefixes cut into many pieces per unit
    Case("8B P16000 N70 x2", 32, 8, 70, [16000, 12000], [70, 3]),
    # ragged batch: empty prefixes, full and partial row tiles, big trees
    Case("ragged batch", 64, 8, 200, [0, 1, 63, 64, 65, 3000, 777, 128],
         [200, 1, 17, 64, 33, 150, 2, 99]),
    Case("many short", 16, 4, 40, [17 * i for i in range(24)], [1 + (7 * i) % 40 for i in range(24)]),
]
