"""The root-path walk the row-wise attention kernel uses to list a node's
tree keys (csrc/tree_walk.hpp), built for the host with g++ and run on
malformed parent arrays: it must end at the root within i + 1 entries and
stay inside the path buffer whatever the array holds, and follow the real
links on a well-formed tree."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_01639_amd", "csrc")

DRIVER = r"""
#include <cstdio>
#include <cstdlib>
#include "tree_walk.hpp"
// stdin: n, then n parent entries; stdout: the path of every node, one line each
int main() {
  int n;
  if (std::scanf("%d", &n) != 1) return 2;
  int32_t* par = new int32_t[n];
  for (int i = 0; i < n; ++i) if (std::scanf("%d", &par[i]) != 1) return 2;
  // one guard entry past the largest legal path, to catch overruns
  int* path = new int[n + 1];
  for (int i = 0; i < n; ++i) {
    path[i + 1] = -12345;
    const int len = ltd::root_path(par, i, path);
    if (path[i + 1] != -12345) return 3;
    std::printf("%d", len);
    for (int k = 0; k < len; ++k) std::printf(" %d", path[k]);
    std::printf("\n");
  }
  return 0;
}
"""


@pytest.fixture(scope="module")
def walker(tmp_path_factory):
    d = tmp_path_factory.mktemp("walk")
    src = d / "walk.cpp"
    src.write_text(DRIVER)
    exe = d / "walk"
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    return str(exe)


def _run(exe, par):
    inp = f"{len(par)} " + " ".join(str(int(x)) for x in par)
    r = subprocess.run([exe], input=inp, capture_output=True, text=True, timeout=20)
    assert r.returncode == 0, r.returncode
    out = []
    for line in r.stdout.splitlines():
        v = [int(x) for x in line.split()]
        assert v[0] == len(v) - 1
        out.append(v[1:])
    return out


def test_well_formed_trees_give_their_root_paths(walker):
    rng = np.random.default_rng(0)
    for n in (1, 2, 7, 60, 256):
        par = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, n)])
        paths = _run(walker, par)
        for i, p in enumerate(paths):
            want, j = [], i
            while j != -1:
                want.append(j)
                j = int(par[j])
            assert p == want


@pytest.mark.parametrize("name,par", [
    ("self parents", [-1, 1, 2, 3, 4]),
    ("two-cycle", [-1, 2, 1, 2, 3]),
    ("forward links", [-1, 4, 3, 4, 4]),
    ("large links", [-1, 10**6, 2**31 - 1, 77, 5]),
    ("negative links", [-1, -5, -2**31, -1, -7]),
    ("root with a parent", [3, 0, 1, 2, 0]),
])
def test_malformed_trees_end_at_the_root_in_bounds(walker, name, par):
    paths = _run(walker, par)
    for i, p in enumerate(paths):
        assert 1 <= len(p) <= i + 1, name
        assert p[0] == i and p[-1] == 0, name
        assert all(a > b for a, b in zip(p, p[1:])), name
