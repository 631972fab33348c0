"""The attention launch's work partition (csrc/stream_plan.hpp), built for the
host with g++ and checked on random and degenerate batches: every key tile
and every tree block of every (sequence, kv head, row tile) unit goes to
exactly one workgroup; a workgroup's shares are consecutive units; a share
is written as final output exactly when one workgroup owns the whole unit;
partial results never share a slot; and every cut unit is merged exactly once,
from exactly the slots its pieces wrote, in workgroup order."""
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_01639_amd", "csrc")

DRIVER = r"""
#include <cstdio>
#include <map>
#include <set>
#include <tuple>
#include <vector>
#include "stream_plan.hpp"
using namespace ltd::plan;
#define CHECK(c, msg) do { if (!(c)) { std::printf("FAIL %s (line %d)\n", msg, __LINE__); return 1; } } while (0)
// stdin: cases of "B G Hkv W" then B pairs "P n"; stdout: OK per case
int main() {
  int B, G, Hkv, W;
  while (std::scanf("%d %d %d %d", &B, &G, &Hkv, &W) == 4) {
    std::vector<int> P(B), N(B);
    for (int b = 0; b < B; ++b) if (std::scanf("%d %d", &P[b], &N[b]) != 2) return 2;
    std::vector<SeqCost> cost(B);
    std::vector<int64_t> pre(B + 1, 0);
    std::vector<int> ubase(B + 1, 0);
    for (int b = 0; b < B; ++b) {
      cost[b] = seq_cost(P[b], N[b], G);
      pre[b + 1] = pre[b] + Hkv * cost[b].per_head;
      ubase[b + 1] = ubase[b] + Hkv * cost[b].rt;
    }
    const int64_t C = pre[B];
    const Grid gr = make_grid(C, W);
    for (int w = 2; w <= 4; ++w)
      for (int64_t x = -3; x < 200000; x += (x < 5000 ? 1 : 7)) {
        const int cap = 1 << 30;
        const int64_t want = x <= 0 ? 0 : (x + w - 1) / w;
        CHECK(item_index(x, w, cap) == want, "item_index");
      }
    for (int s = 0; s <= W; ++s) {
      CHECK(range_lo(gr, s) == (int64_t(s) * C + W - 1) / W, "range_lo is ceil(s C / W)");
      if (s < W && range_lo(gr, s) < range_lo(gr, s + 1)) CHECK(owner(gr, range_lo(gr, s)) == s, "owner");
    }
    auto find = [&](int64_t p) {
      int b = 0;
      while (!(pre[b] <= p && p < pre[b + 1])) ++b;
      return SeqAt{b, P[b], N[b], pre[b], ubase[b], cost[b]};
    };
    // item key: (unit start U, item index j; j == t_pre for the tree block)
    std::map<std::pair<int64_t, int>, int> owner_of;
    std::map<int64_t, std::set<int>> unit_wgs;        // U -> workgroups with a share
    std::map<int64_t, bool> unit_whole;
    std::map<int64_t, std::vector<std::pair<int, int>>> unit_pieces;  // U -> (wg, slot) of partials
    std::set<int> slots;
    int64_t items = 0;
    for (int s = 0; s < W; ++s) {
      int64_t lastU = -1;
      int nshares = 0;
      bool bad = false;
      for_each_share(s, gr, find, [&](const SeqAt& q, const Unit& u, int64_t U, const Share& sh,
                                        bool whole, int slot) {
        if (U <= lastU) bad = true;           // consecutive, increasing units
        if (nshares > 0 && lastU >= 0 && U != lastU) {
          // a share after the first must start at its unit's first item
          if (sh.j0 != 0 && !(sh.j0 == q.c.t_pre && sh.j1 == q.c.t_pre)) bad = true;
        }
        lastU = U;
        ++nshares;
        const KeyRange kr = share_keys(sh, q.P);
        if (kr.begin < 0 || kr.count < 0 || kr.begin + kr.count > q.P) bad = true;
        if (sh.j1 > sh.j0 && (kr.begin != sh.j0 * 64 || kr.count <= 0)) bad = true;
        if (sh.tree && kr.begin + kr.count != q.P) bad = true;  // the tree follows the prefix
        for (int j = sh.j0; j < sh.j1; ++j) {
          if (owner_of.count({U, j})) bad = true;
          owner_of[{U, j}] = s;
          ++items;
        }
        if (sh.tree) {
          if (owner_of.count({U, q.c.t_pre})) bad = true;
          owner_of[{U, q.c.t_pre}] = s;
          ++items;
        }
        unit_wgs[U].insert(s);
        if (whole) unit_whole[U] = true;
        else {
          if (slot < 0 || slot >= 2 * W || slots.count(slot)) bad = true;
          slots.insert(slot);
          unit_pieces[U].push_back({s, slot});
        }
      });
      CHECK(!bad, "shares");
    }
    // every item of every unit owned once
    int64_t want_items = 0;
    for (int b = 0; b < B; ++b) want_items += int64_t(Hkv) * cost[b].rt * (cost[b].t_pre + 1);
    CHECK(items == want_items, "item count");
    CHECK((int64_t)owner_of.size() == want_items, "distinct items");
    for (auto& kv : unit_wgs) {
      const bool whole = unit_whole.count(kv.first) > 0;
      CHECK(whole == (kv.second.size() == 1), "whole iff one owner");
      if (whole) CHECK(unit_pieces[kv.first].empty(), "whole unit has no partials");
    }
    // merges: every unit's job is worked out once, by its tree block's owner;
    // a cut unit's job lists exactly its pieces' slots, in workgroup order
    std::map<int64_t, int> jobs;
    std::set<int> indices;
    for (int s = 0; s < W; ++s) {
      bool bad = false;
      for_each_share(s, gr, find, [&](const SeqAt& q, const Unit& u, int64_t U, const Share& sh,
                                      bool whole, int) {
        const int ui = unit_index(q, u);
        if (ui < 0 || ui >= ubase[B]) bad = true;
        if (!sh.tree) return;
        if (jobs.count(U) || indices.count(ui)) bad = true;
        jobs[U] = s;
        indices.insert(ui);
        const MergeJob j = unit_job(q, u, U, s, gr, find);
        if (j.active == whole) bad = true;
        std::vector<std::pair<int, int>> got;
        if (j.active)
          for (int k = 0; k <= s - j.sa; ++k) {
            const int slot = merge_piece_slot(j, k, gr);
            if (slot >= 0) got.push_back({j.sa + k, slot});
          }
        if (got != unit_pieces[U]) bad = true;
      });
      CHECK(!bad, "merge jobs");
    }
    CHECK((int)jobs.size() == (int)unit_wgs.size(), "one job per unit");
    CHECK((int)indices.size() == ubase[B] && *indices.begin() == 0 && *indices.rbegin() == ubase[B] - 1,
          "unit indices 0 .. units-1");
    // coverage of the partition's cases: shares holding only a tree block,
    // workgroups owning nothing, whole units, cut units, most pieces of one unit
    int tree_only = 0, empty_wgs = 0, whole = 0, cut = 0, max_pieces = 0;
    for (int s = 0; s < W; ++s) {
      int shares = 0;
      for_each_share(s, gr, find, [&](const SeqAt&, const Unit&, int64_t, const Share& sh,
                                        bool, int) {
        ++shares;
        if (sh.tree && sh.j0 == sh.j1) ++tree_only;
      });
      if (shares == 0) ++empty_wgs;
    }
    for (auto& kv : unit_wgs) {
      if (kv.second.size() == 1) ++whole;
      else ++cut;
      if ((int)kv.second.size() > max_pieces) max_pieces = (int)kv.second.size();
    }
    std::printf("OK %lld %lld %d %d %d %d %d\n", (long long)C, (long long)items, tree_only,
                empty_wgs, whole, cut, max_pieces);
  }
  return 0;
}
"""


@pytest.fixture(scope="module")
def planner(tmp_path_factory):
    d = tmp_path_factory.mktemp("plan")
    (d / "plan.cpp").write_text(DRIVER)
    exe = d / "plan"
    subprocess.run(["g++", "-std=c++17", "-O2", "-I", CSRC, str(d / "plan.cpp"), "-o", str(exe)],
                   check=True)
    return str(exe)


def _run(exe, cases):
    """Checks every case; returns per case (tree-only shares, workgroups with
    nothing, whole units, cut units, most pieces of a unit)."""
    text = []
    for B, G, Hkv, W, seqs in cases:
        text.append(f"{B} {G} {Hkv} {W} " + " ".join(f"{p} {n}" for p, n in seqs))
    r = subprocess.run([exe], input="\n".join(text), capture_output=True, text=True, timeout=300)
    lines = r.stdout.splitlines()
    assert r.returncode == 0 and len(lines) == len(cases) and all(l.startswith("OK") for l in lines), \
        (r.returncode, lines[-3:])
    return [tuple(int(x) for x in l.split()[3:]) for l in lines]


def test_gpu_partition_cases_cover_every_kind_of_share(planner):
    """The GPU parity test's partition batches (tests/partition_cases.py), on
    the grid the library plans for them on a 256-CU MI355X, hold between them
    every kind of share: a tree block alone, a workgroup with nothing, whole
    units and units cut into several pieces."""
    import partition_cases as PC
    import paper_2603_01639_amd as ltd
    cases = []
    for c in PC.CASES:
        W = ltd.attn_grid(len(c.prefix), c.Nmax, c.Hq, c.Hkv, 128, max(c.prefix), ltd.DTYPE_BF16,
                          max(c.prefix) + c.Nmax)
        assert W > 0
        cases.append((len(c.prefix), c.Hq // c.Hkv, c.Hkv, W, list(zip(c.prefix, c.nodes))))
    stats = np.array(_run(planner, cases))
    tree_only, empty, whole, cut, pieces = stats.T
    assert tree_only.max() > 0 and empty.max() > 0 and whole.max() > 0 and cut.max() > 0
    assert pieces.max() >= 8


def test_paper_shaped_batches(planner):
    rng = np.random.default_rng(7)
    cases = [
        (1, 4, 8, 128, [(2048, 60)]),
        (1, 4, 8, 256, [(16384, 60)]),
        (1, 8, 8, 256, [(4096, 256)]),
        (1, 8, 8, 256, [(4096, 8)]),
    ]
    seqs = [(int(rng.integers(1024, 8193)), int(rng.integers(16, 129))) for _ in range(16)]
    cases.append((16, 8, 8, 256, seqs))
    _run(planner, cases)


def test_random_and_degenerate_batches(planner):
    rng = np.random.default_rng(11)
    cases = []
    for _ in range(300):
        B = int(rng.integers(1, 70))
        G = int(rng.choice([1, 2, 4, 8]))
        Hkv = int(rng.choice([1, 2, 8]))
        W = int(rng.choice([8, 16, 64, 128, 256, 1024]))
        kind = rng.integers(0, 4)
        seqs = []
        for _ in range(B):
            if kind == 0:    # empty prefixes, tiny trees: fewer items than workgroups
                seqs.append((0, int(rng.integers(1, 4))))
            elif kind == 1:  # prefixes on and next to tile edges
                seqs.append((int(rng.choice([1, 63, 64, 65, 127, 128])), int(rng.integers(1, 257))))
            else:
                seqs.append((int(rng.integers(0, 9000)), int(rng.integers(1, 257))))
        cases.append((B, G, Hkv, W, seqs))
    _run(planner, cases)
