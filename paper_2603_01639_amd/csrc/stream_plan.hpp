// Work partition of the tree-attention launch: every workgroup of the grid
// takes an equal share of the whole call's key tiles.
//
// A unit is one (sequence b, kv head g, row tile rt): up to 256 stacked query
// rows that stream the sequence's keys.  Its work items, in order, are its
// prefix key tiles j = 0 .. T_pre - 1 (64 keys each) and then one tree block
// (the tree's ceil(n / 64) key tiles under the ancestor mask, never cut).
// Units are listed sequence by sequence, kv head by kv head, row tile by row
// tile, and laid end to end on one axis.  A unit that starts at U with
// per-tile weight wu first takes wu * kUnitOverhead for the fixed cost of a
// piece (its Q rows and first tiles in flight, the output written at the
// end); its items start at I = U + wu * kUnitOverhead, item j at I + wu * j,
// the tree block at I + wu * T_pre, and the unit ends at
// I + wu * (T_pre + kTreeCost * T_tree).  The weight prices a tile by the
// waves that compute on it: a row tile with few valid rows streams the same
// keys with fewer waves busy and costs less per tile.
//
// With C the axis length and W workgroups, workgroup s owns the items whose
// position p has floor(p * W / C) == s: a contiguous run of the unit list.
// Its first and last unit can be cut (shared with neighbours); the units
// between are whole.  A cut unit's pieces are the consecutive workgroups
// that own its items; each piece leaves a partial result in slot 2s (the
// piece is the first unit of workgroup s) or 2s + 1 (its last), and the merge
// combines them in workgroup order.
//
// Everything here is constexpr, so the same functions run in the kernels and
// in a plain host build (how the partition is tested without a GPU).
#pragma once

#include <stdint.h>

namespace ltd {
namespace plan {

constexpr int kKeyTile = 64;    // keys per tile
constexpr int kUnitRows = 256;  // stacked query rows per unit (8 waves x 32)
constexpr int kWaveRows = 32;

// Relative cost of one key tile for a row tile with v busy waves (measured
// with per-workgroup timestamps on a batch of 16 sequences: about 2.3 us per
// tile with 5-8 waves, 1.6 us with 1-4).
constexpr int tile_weight(int waves) { return waves >= 5 ? 3 : 2; }
// Axis extent of a tree key tile in prefix tiles (the ancestor masks are built
// and applied on them: about 6.5 us per tree tile with 5-8 waves), and of a
// piece's fixed cost (about 4.5 us before the first tile and 2 us after the
// last one).
constexpr int kTreeCost = 3;
constexpr int kUnitOverhead = 2;
// A unit's axis extent in units of its tile weight.
constexpr int64_t unit_extent(int t_pre, int t_tree) {
  return kUnitOverhead + static_cast<int64_t>(t_pre) + static_cast<int64_t>(kTreeCost) * t_tree;
}

struct SeqCost {
  int rt;      // row tiles (units per kv head)
  int w_full;  // weight of a full row tile
  int w_last;  // weight of the last row tile
  int t_pre;   // prefix key tiles
  int t_tree;  // tree key tiles (one block)
  int64_t per_head;  // axis length of one kv head's units
};

// Cost data of a sequence with prefix P and n tree nodes, G query heads per
// kv head.
constexpr SeqCost seq_cost(int P, int n, int G) {
  SeqCost c{};
  const int rows = G * n;
  c.rt = rows > 0 ? (rows + kUnitRows - 1) / kUnitRows : 0;
  c.w_full = tile_weight(kUnitRows / kWaveRows);
  const int last_rows = rows - (c.rt - 1) * kUnitRows;
  c.w_last = c.rt > 0 ? tile_weight((last_rows + kWaveRows - 1) / kWaveRows) : 0;
  c.t_pre = (P + kKeyTile - 1) / kKeyTile;
  c.t_tree = (n + kKeyTile - 1) / kKeyTile;
  const int64_t tiles = unit_extent(c.t_pre, c.t_tree);
  c.per_head = c.rt > 0 ? (static_cast<int64_t>(c.rt - 1) * c.w_full + c.w_last) * tiles : 0;
  return c;
}

// A unit located on the axis.
struct Unit {
  int g, rt;      // kv head and row tile within the sequence
  int64_t start;  // axis position of its first item (relative to the sequence's start)
  int w;          // per-tile weight
};

// The unit of sequence cost c that contains axis offset `off` (0 <= off <
// Hkv * c.per_head) from the sequence's start.  (Divisions are slow on the
// GPU; the kv head and row tile are found by stepping, at most Hkv and 8
// steps, and most calls take one or two.)
constexpr Unit locate(int64_t off, const SeqCost& c) {
  Unit u{};
  const int64_t tiles = unit_extent(c.t_pre, c.t_tree);
  const int64_t full = c.w_full * tiles;  // axis length of a full row tile
  int64_t in_head = off;
  u.g = 0;
  while (in_head >= c.per_head) {
    in_head -= c.per_head;
    ++u.g;
  }
  u.rt = 0;
  while (u.rt < c.rt - 1 && in_head >= full) {
    in_head -= full;
    ++u.rt;
  }
  u.start = off - in_head;
  u.w = u.rt < c.rt - 1 ? c.w_full : c.w_last;
  return u;
}

// The axis cut into W = 2^k ranges: C = q * W + r, and range s starts at
// ceil(s * C / W) = s * q + ceil(s * r / W), all shifts and multiplies.
struct Grid {
  int64_t C, q;
  int W, log2W, r;
};
constexpr Grid make_grid(int64_t C, int W) {
  int k = 0;
  while ((1 << k) < W) ++k;
  return Grid{C, C >> k, W, k, static_cast<int>(C & (W - 1))};
}
// First axis position owned by workgroup s (0 <= s <= W).
constexpr int64_t range_lo(const Grid& g, int s) {
  return static_cast<int64_t>(s) * g.q + ((static_cast<int64_t>(s) * g.r + g.W - 1) >> g.log2W);
}
// Workgroup owning axis position p (0 <= p < C): floor(p * W / C), from a
// float estimate corrected against the exact range starts.
constexpr int owner(const Grid& g, int64_t p) {
  int s = static_cast<int>(static_cast<float>(p) * static_cast<float>(g.W) / static_cast<float>(g.C));
  s = s < 0 ? 0 : (s > g.W - 1 ? g.W - 1 : s);
  while (s > 0 && range_lo(g, s) > p) --s;
  while (s < g.W - 1 && range_lo(g, s + 1) <= p) ++s;
  return s;
}

// Items of a unit (start U, weight w, t_pre prefix tiles) owned by the
// workgroup whose range is [lo, hi): prefix tiles [j0, j1) and whether the
// tree block is among them.
struct Share {
  int j0, j1;
  bool tree;
  constexpr bool empty() const { return j0 >= j1 && !tree; }
};
// ceil(max(x, 0) / w) for an item offset x and a tile weight w in {2, 3, 4},
// clamped to `cap` items (shifts, and a multiply by ceil(2^33 / 3) for w = 3).
// x counts from the unit's first item I.
constexpr int item_index(int64_t x, int w, int cap) {
  if (x <= 0) return 0;
  const int64_t lim = static_cast<int64_t>(cap) * w;
  const uint32_t xi = static_cast<uint32_t>((x < lim ? x : lim) + w - 1);
  if (w == 4) return static_cast<int>(xi >> 2);
  if (w == 2) return static_cast<int>(xi >> 1);
  return static_cast<int>((static_cast<uint64_t>(xi) * 0xAAAAAAABull) >> 33);
}
// Axis position of the first item of a unit that starts at U.
constexpr int64_t first_item(int64_t U, int w) { return U + static_cast<int64_t>(w) * kUnitOverhead; }
constexpr Share share_of(int64_t U, int w, int t_pre, int64_t lo, int64_t hi) {
  Share s{};
  const int64_t I = first_item(U, w);
  const int a = item_index(lo - I, w, t_pre + 1);  // first item index at or after lo
  const int b = item_index(hi - I, w, t_pre + 1);  // first item index at or after hi
  s.j0 = a < t_pre ? a : t_pre;
  s.j1 = b < t_pre ? b : t_pre;
  const int64_t tree_pos = I + static_cast<int64_t>(w) * t_pre;
  s.tree = lo <= tree_pos && tree_pos < hi;
  return s;
}

// The prefix keys [begin, begin + count) of a share of a sequence with prefix
// P (a share of the tree block alone starts at P with none).
struct KeyRange {
  int begin, count;
};
constexpr KeyRange share_keys(const Share& sh, int P) {
  const int b = sh.j0 * kKeyTile < P ? sh.j0 * kKeyTile : P;
  const int e = sh.j1 * kKeyTile < P ? sh.j1 * kKeyTile : P;
  return KeyRange{b, e - b};
}

// The partial-result slot of a piece: 2s when the unit is the first one
// workgroup s owns items of, else 2s + 1.
constexpr int piece_slot(int s, bool first_unit_of_wg) { return 2 * s + (first_unit_of_wg ? 0 : 1); }

// A sequence found on the axis: its index, first position, prefix length,
// node count and cost data.  `Find` callables map an axis position p
// (0 <= p < C) to the sequence whose units hold it.
struct SeqAt {
  int b, P, n;
  int64_t pre;
  int ubase;  // index of the sequence's first unit among all units of the call
  SeqCost c;
};

// Index of a unit among all units of the call (sequence by sequence, kv head
// by kv head, row tile by row tile).
constexpr int unit_index(const SeqAt& q, const Unit& u) { return q.ubase + u.g * q.c.rt + u.rt; }

constexpr int64_t unit_end(const SeqAt& q, const Unit& u) {
  return q.pre + u.start + static_cast<int64_t>(u.w) * unit_extent(q.c.t_pre, q.c.t_tree);
}
// Axis position of a unit's tree block (its last item).
constexpr int64_t tree_item(int64_t U, int w, int t_pre) {
  return first_item(U, w) + static_cast<int64_t>(w) * t_pre;
}

// Workgroup s's shares, in order, from axis position `pos` (its range start,
// or where an earlier call stopped): visit(seq, unit, U, share, whole, slot)
// for up to `limit` units it owns items of.  U is the unit's axis start,
// `whole` says the share is the entire unit (its output is final), `slot` is
// where a partial share leaves its result; `first` tracks whether a share was
// visited yet.  Returns the position to resume from, at or past the range's
// end once every share was visited.
template <class Find, class Visit>
constexpr int64_t walk_shares(int s, const Grid& gr, int64_t pos, bool& first, int limit, Find find,
                              Visit visit) {
  const int64_t lo = range_lo(gr, s);
  const int64_t hi = range_lo(gr, s + 1);
  int visited = 0;
  while (pos < hi && visited < limit) {
    const SeqAt q = find(pos);
    const Unit u = locate(pos - q.pre, q.c);
    const int64_t U = q.pre + u.start;
    const Share sh = share_of(U, u.w, q.c.t_pre, lo, hi);
    if (!sh.empty()) {
      visit(q, u, U, sh, first_item(U, u.w) >= lo && sh.j0 == 0 && sh.tree, piece_slot(s, first));
      first = false;
      ++visited;
    }
    pos = unit_end(q, u);
  }
  return pos;
}

template <class Find, class Visit>
constexpr void for_each_share(int s, const Grid& gr, Find find, Visit visit) {
  bool first = true;
  int64_t pos = range_lo(gr, s);
  const int64_t hi = range_lo(gr, s + 1);
  while (pos < hi) pos = walk_shares(s, gr, pos, first, 1 << 30, find, visit);
}

// The merge of a unit, worked out by the workgroup s that owns the unit's tree
// block (its last item, so every unit has exactly one such workgroup).  The
// unit is cut when its first item belongs to an earlier workgroup sa; its
// pieces are then workgroups sa .. s (a workgroup between them can own none
// of its items when its range falls between two of them).
struct MergeJob {
  bool active;  // the unit was cut
  SeqAt q;
  Unit u;
  int64_t U;
  int sa;
  bool sa_first;  // the unit is the first one workgroup sa owns items of
};

template <class Find>
constexpr MergeJob unit_job(const SeqAt& q, const Unit& u, int64_t U, int s, const Grid& gr,
                            Find find) {
  MergeJob j{};
  j.q = q;
  j.u = u;
  j.U = U;
  j.sa = owner(gr, first_item(U, u.w));
  j.active = j.sa != s;
  j.sa_first = false;
  if (!j.active) return j;
  // Is u the first unit workgroup sa owns items of?  Yes when sa's first
  // position is in u, or lies past the last item of the unit just before u.
  const int64_t lo_a = range_lo(gr, j.sa);
  const SeqAt qa = find(lo_a);
  const Unit ua = locate(lo_a - qa.pre, qa.c);
  const int64_t Ua = qa.pre + ua.start;
  j.sa_first = Ua == U || (lo_a > tree_item(Ua, ua.w, qa.c.t_pre) && unit_end(qa, ua) == U);
  return j;
}

// The slot of piece k (workgroup sa + k) of a merge job, or -1 when that
// workgroup owns no item of the unit (its range fell between two items).
constexpr int merge_piece_slot(const MergeJob& j, int k, const Grid& gr) {
  const int sp = j.sa + k;
  const Share sh = share_of(j.U, j.u.w, j.q.c.t_pre, range_lo(gr, sp), range_lo(gr, sp + 1));
  if (sh.empty()) return -1;
  return piece_slot(sp, k > 0 || j.sa_first);
}

}  // namespace plan
}  // namespace ltd
