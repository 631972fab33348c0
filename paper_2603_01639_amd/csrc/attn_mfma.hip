// Split-KV tree attention for bf16 on CDNA4 matrix cores (gfx950), head_dim 128 or 64.
//
// What is computed (arXiv 2603.01639, section 3.2): the N draft-tree
// candidates are verified in one pass, each seeing the KV prefix and its own
// ancestors (the tree attention mask).  For every (sequence b, kv head g) the
// G = Hq/Hkv query heads of the group and the N tree nodes are stacked into
// M = G*N query rows (row r = node*G + head-in-group) that share one K/V
// stream, so both contractions are dense MFMA tiles:
//
//   S^T[key][row] = K[key][:] . Q[row][:]        (v_mfma_f32_32x32x16_bf16)
//   O^T[dim][row] += V^T[dim][key] . P^T[key][row]
//
// Work split: a unit is one (sequence, kv head, row tile of up to 8*32
// stacked rows).  Its work is its prefix key tiles and then the tree's keys
// under the ancestor mask.  All units of the call are laid end to end and the
// grid's workgroups take equal shares of that sequence (stream_plan.hpp): a
// workgroup of 8 wavefronts (32 rows each) runs through its share unit by
// unit.  A unit it covers whole gets its final output written directly; a
// unit cut between workgroups gets a partial result (max, sum and normalised
// output) from each of them, which attn_stream_merge_kernel combines.  A
// single sequence instead cuts each unit into KV splits of equal length (the
// split plan: attn_split_kernel, attn_split_merge_kernel).
//
// K/V stream: 64-key tiles move from HBM straight into an LDS ring of
// kStages slots with global_load_lds_dwordx4 (no register staging); a lane
// picks the global 16-byte chunk whose LDS position is base + 16*lane, which
// is how the LDS swizzles are applied.  One barrier per tile.
//
// K in LDS: the 32 rows of each 32-key block are stored in the order the
// S^T operand reads them (row i holds key sigma(i)), with 16-byte chunk c of
// row i at c ^ (i & 15).  After the MFMA, accumulator register r of lane half
// h then holds key 16*h + r for the lane's query row, so the scores of one
// query row sit in one lane, the softmax state and the O^T accumulators are
// per-lane, and the score registers are directly the P^T operand.
//
// V in LDS keeps its natural [key][dim] layout (chunk c of key k at
// c ^ 4*(k & 3)); the V^T operand comes from ds_read_b64_tr_b16 transpose
// reads, two per MFMA.
//
// The ancestor sets of the tree split are built in LDS as N x 256-bit masks by
// pointer doubling over the parent links: anc(i) = anc(i) | anc(jump(i)),
// jump(i) = jump(jump(i)), ceil(log2(depth + 1)) <= 8 rounds for N <= 256.
//
// Head size: the LDS layouts are those of 128-dim rows (kD) for either size.
// With 64 dims a row's 8 chunks are fetched into both halves of its LDS row
// (the lane at chunk c takes global chunk c mod 8 of its swizzled position),
// and the contractions run over the first 64 dims only: 4 k-steps for S^T and
// 2 dim blocks for O^T, half the MFMAs of a tile.  Partial results keep the
// 128-dim row pitch in the workspace.
#include <algorithm>

#include "ltd_device.hpp"
#include "ltd_launch.hpp"
#include "stream_plan.hpp"

namespace ltd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void global_cvoid;

constexpr int kD = 128;                        // dims of an LDS row (the largest head size)
constexpr int kKT = 64;                        // keys per tile
constexpr int kWaves = 8;                      // waves per workgroup
constexpr int kThreads = kWaves * kWave;
constexpr int kAncWords = LTD_MAX_NODES / 32;  // 256 bits per node
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kKBytes = kKT * kD * 2;          // one K tile in LDS (16 KiB)
constexpr int kVBytes = kKT * kD * 2;          // one V tile in LDS (16 KiB)
constexpr int kTileBytes = kKBytes + kVBytes;
constexpr int kLoadsPerTile = 2 * (kKBytes / 16) / kThreads;  // 4 per lane
constexpr int kKLoads = kLoadsPerTile / 2;  // K (and V) chunks per lane per tile
// A running max is kept until a score exceeds it by 2^kLazyMax (log2 units):
// probabilities stay below 2^kLazyMax, exact in fp32 and well inside bf16
// range, and the O/l rescale runs only when the max really moves.
constexpr float kLazyMax = 8.f;
constexpr float kNoMax = -__FLT_MAX__;  // running max before any key (raw score units)
constexpr int kStages = 4;                // K/V tiles in the LDS ring
constexpr int kMaxSplitTiles = 32;        // split plan: longest split in key tiles
constexpr int kMaxMergeSplits = 1024;     // split plan: splits the merge takes at most
constexpr int kTileRows = kWaves * 32;    // stacked query rows per workgroup (one unit)
static_assert(kTileRows == plan::kUnitRows && kKT == plan::kKeyTile, "unit shape");

struct MergeDesc;

struct MfmaArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* block_table;
  const int32_t* prefix_len;
  const int32_t* parents;
  const int32_t* n_nodes;
  uint16_t* ws_o;  // [2W][256][128] bf16: a piece's O / l (slot 2s or 2s + 1)
  float* ws_ml;    // [2W][256][2]: max (log2 units), sum l
  MergeDesc* ws_desc;  // [units]: each unit's merge (after a 64-byte header: the unit count)
  int max_units;       // units the launch can have at most (table entries)
  uint16_t* out;
  const int32_t* status;
  int B, Nmax, Hq, Hkv, G, kv_rows, max_blocks, max_prefix;
  int kv_shift;  // log2(kv_rows) when kv_rows is a power of two, else -1
  int W;  // stream plan: workgroups of the grid (a power of two)
  // split plan: prefix keys per split, splits of the longest sequence, whether
  // the tree may take a split of its own, row tiles per (sequence, kv head)
  int split_keys, max_splits, tree_alone, row_tiles;
  float scale_log2;
  float lazy_gap;  // kLazyMax / scale_log2: the raw-score margin of the lazy max
};

// A-row i of a 32-key block reads key sigma(i); accumulator register r of lane
// half h then holds key 16*h + r.
__device__ __forceinline__ int sigma(int i) {
  return 16 * ((i >> 2) & 1) + 4 * (i >> 3) + (i & 3);
}
__device__ __forceinline__ int swz_v(int key) { return 4 * (key & 3); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// x of lane (l xor 32), with v_permlane32_swap (a VALU op; __shfl_xor goes
// through the LDS crossbar, where it queues behind the tile's fragment reads).
// The swap of x with itself leaves the upper half's values in the lower half
// of the second result and the lower half's in the upper half of the first.
__device__ __forceinline__ float xor32(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (__lane_id() & 32) ? r[0] : r[1]);
}

// KV splits of a sequence with prefix P and n tree nodes.  The prefix is cut
// into ranges of split_keys keys (at least one range).  The tree's keys join
// the last range, except when the plan sets tree_alone, the prefix has two or
// more ranges and the last one would then hold more tiles than a full range:
// the tree is then a split of its own, after the prefix ranges.
__host__ __device__ __forceinline__ int n_splits_of(int P, int n, int split_keys, int tree_alone) {
  const int pre = (P + split_keys - 1) / split_keys;
  if (pre <= 1) return 1;
  if (tree_alone) {
    const int last_tiles = (P - (pre - 1) * split_keys + kKT - 1) / kKT;
    if (last_tiles + (n + kKT - 1) / kKT > split_keys / kKT) return pre + 1;
  }
  return pre;
}

// The larger of x in lanes l and l ^ 32, in every lane: the swap of x with
// itself leaves the lower half's values in both halves of the first result and
// the upper half's in both halves of the second.
__device__ __forceinline__ float max_xor32(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  // (the halves are copied out first: hipcc folds a bit-cast of element 1 of
  // the result to element 0)
  const uint32_t lo = r[0], hi = r[1];
  return __builtin_elementwise_maximum(__builtin_bit_cast(float, lo), __builtin_bit_cast(float, hi));
}

__device__ __forceinline__ lds_void* as_lds(const void* p) { return (lds_void*)(p); }
__device__ __forceinline__ global_cvoid* as_global(const void* p) { return (global_cvoid*)(p); }

// Transposed 4-key x 16-dim read of a 16-lane group (ds_read_b64_tr_b16):
// supplier lane s of the group addresses key k0 + s/4, dims d0 + 4*(s%4)..+3;
// lane p then receives keys k0..k0+3 of dim d0 + p.
__device__ __forceinline__ s16x4 lds_read_tr(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)as_lds(p));
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Direct global->LDS loads of 16 bytes per lane (global_load_lds_dwordx4;
// lane i's bytes land at M0 + 16*i).  They are issued as inline assembly on
// purpose: the compiler does not track them, so it does not put a full
// vector-memory wait in front of every later LDS read (which would drain the
// prefetch ring every tile).  The kernel waits for them itself (wait_vmcnt)
// and orders them across waves with bare barriers.  Nothing else in these
// kernels uses M0.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(as_lds(p))));
}
// Base pointer that the compiler must keep in scalar registers (the SADDR
// form of the load takes a 64-bit SGPR pair).
__device__ __forceinline__ const void* scalar_ptr(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo);
}
__device__ __forceinline__ void dma16(uint32_t lds, const void* uniform_base, uint32_t lane_off) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               ::"s"(lds), "v"(lane_off), "s"(scalar_ptr(uniform_base))
               : "memory");
}
__device__ __forceinline__ void dma16(uint32_t lds, const void* lane_ptr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(lane_ptr)
               : "memory");
}
// Direct global->LDS load of 4 bytes per lane (lane i's word lands at M0 + 4*i).
__device__ __forceinline__ void dma4(uint32_t lds, const void* lane_ptr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(lds), "v"(lane_ptr)
               : "memory");
}
// Workgroup barrier without the memory fence __syncthreads() adds (that fence
// would also wait for every outstanding direct load).
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

constexpr int kMaxSplitBlocks = 3072;  // paged block ids one unit's share may span

// One share of a workgroup's work (a unit's key range), planned by wave 0 and
// read by every wave before it runs the share.
struct ShareDesc {
  int32_t b, g, rt, P, n, key_begin, n_pre, tree, whole, slot;
};
constexpr int kMaxShares = 16;  // shares planned per round

struct Smem {
  unsigned char kv[kStages][kTileBytes];
  ShareDesc share[kMaxShares];
  int64_t next_pos;  // where the next planning round resumes
  int32_t n_share, first;
  uint32_t anc[LTD_MAX_NODES][kAncWords];
  int16_t jump[LTD_MAX_NODES];     // jump pointers of the mask build
  int32_t par[LTD_MAX_NODES];      // the tree's parent links (mask build)
  int32_t blk[kMaxSplitBlocks];  // physical block ids of this split's rows (paged)
};
// The Q rows are loaded into ring slots 2 and 3 (8 KiB per wave) before the
// first two tiles; the loop first writes those slots after its first barrier.
static_assert(kStages >= 4 && 2 * kTileBytes >= kWaves * 32 * kD * 2, "Q fits ring slots 2-3");

// This lane's share of a tile's direct loads: for load u (0..3) the tile row
// of its K chunk and of its V chunk, the chunk's byte offset within the row,
// and the wave-uniform LDS byte offset of the wave's 1 KiB destination block.
struct LoadPlan {
  int k_key[kKLoads], k_off[kKLoads], v_key[kKLoads], v_off[kKLoads], lds_pos[kKLoads];
};

__device__ __forceinline__ LoadPlan make_load_plan(int wave, int lane) {
  LoadPlan lp;
#pragma unroll
  for (int u = 0; u < kKLoads; ++u) {
    const int blk = u * kWaves + wave;    // 1 KiB block = 4 LDS rows of 256 B
    const int i = blk * 4 + (lane >> 4);  // LDS row
    const int pc = lane & 15;             // physical 16-byte chunk in the row
    lp.k_key[u] = (i & 32) + sigma(i & 31);
    lp.k_off[u] = (pc ^ (i & 15)) * 16;
    lp.v_key[u] = i;
    lp.v_off[u] = (pc ^ swz_v(i)) * 16;
    lp.lds_pos[u] = blk * 1024;
  }
  return lp;
}

// The attention of one workgroup over its share of one unit: the prefix keys
// [key_begin, key_begin + n_pre) and, with kTree, also the tree's keys
// [P, P + n) under the ancestor mask.  Tiles t < tA cover the first range, the
// rest the second; a tile never spans both.  With final_out the share is the
// whole unit and the normalised output goes to `out`; otherwise the share's
// partial result goes to workspace slot `slot`.
// The cache layout (kPaged) is a compile-time choice, so each kernel's tile
// loop keeps only its own layout's addressing state in scalar registers (the
// contiguous instantiation of the split kernel then spills none of them).
template <bool kTree, int HD, bool kPaged>
__device__ __forceinline__ void attend(const MfmaArgs& a, Smem& sm, int b, int g, int row0,
                                       int valid_rows, int key_begin, int n_pre, int P, int n,
                                       bool final_out, int slot) {
  // (an opaque copy of the thread index: a workgroup runs this once per share,
  // and without it the compiler hoists every per-lane address out of the share
  // loop and keeps it live, and spilled, across all of them)
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int wave = tid / kWave;
  const int lane = tid % kWave;
  const int h = lane >> 5;
  const int l32 = lane & 31;
  const int n_tree = kTree ? n : 0;  // keys of the second range
  const int tA = (n_pre + kKT - 1) / kKT;
  const int n_tiles = tA + (n_tree + kKT - 1) / kKT;
  // Tile t: its first logical cache row, the keys of its range from there on
  // (more than kKT for all but a range's last tile), and whether it is a tree
  // tile (then `rel` is its first key relative to P).
  struct TileRef {
    int row, left, rel;
    bool tree;
  };
  auto tile_ref = [&](int t) -> TileRef {
    if (!kTree || t < tA) return TileRef{key_begin + t * kKT, n_pre - t * kKT, 0, false};
    const int rel = (t - tA) * kKT;
    return TileRef{P + rel, n_tree - rel, rel, true};
  };

  // ---- Q rows and parent links, straight into LDS ahead of everything else
  // (the tile loads queue behind them, and the wait for them below leaves the
  // first tiles in flight).  Wave w's 32 stacked rows row0 + 32w + R land at
  // 256*R in its 8 KiB block, with 16-byte chunk c at c ^ (R & 15), the
  // layout the K operand also uses; rows past valid_rows repeat the last
  // valid row (their results are never stored).
  const int qrow_idx = row0 + wave * 32 + l32;
  const bool qvalid = qrow_idx < valid_rows;
  // A wave whose 32 rows are all padding only loads tiles and takes part in
  // the barriers.
  const bool active = row0 + wave * 32 < valid_rows;
  const int qnode = qvalid ? qrow_idx / a.G : 0;
  unsigned char* q_lds = &sm.kv[2][0] + wave * (32 * kD * 2);
  if (active) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int R = 4 * j + (lane >> 4);
      const int idx = min(row0 + wave * 32 + R, valid_rows - 1);
      const int lc = (lane & 15) ^ (R & 15);
      const uint16_t* src = a.q +
          ((static_cast<int64_t>(b) * a.Nmax + idx / a.G) * a.Hq + g * a.G + idx % a.G) * HD +
          (lc & (HD / 8 - 1)) * 8;
      dma16(lds_addr(q_lds + j * 1024), src);
    }
  }
  constexpr int kNodesPerLane = LTD_MAX_NODES / kWave;
  const int nslots = (n + kWave - 1) / kWave;  // node slots holding a node of this tree
  if (kTree && wave == 0) {
#pragma unroll
    for (int k = 0; k < kNodesPerLane; ++k)
      if (k < nslots)
        dma4(lds_addr(&sm.par[kWave * k]),
             a.parents + static_cast<int64_t>(b) * a.Nmax + min(lane + kWave * k, n - 1));
  }

  // ---- direct K/V tile loads
  const LoadPlan lp = make_load_plan(wave, lane);
  const unsigned char* kbase = reinterpret_cast<const unsigned char*>(a.k);
  const unsigned char* vbase = reinterpret_cast<const unsigned char*>(a.v);
  constexpr bool paged = kPaged;  // a paged cache (block table) or one contiguous range per (b, g)
  // Paged caches: this split's block ids are staged in LDS first, so address
  // generation never waits on a global load.  The split's rows are one
  // contiguous logical range (for the last split the tree rows follow the
  // prefix rows directly).
  int first_blk = 0;
  if (paged) {
    first_blk = key_begin / a.kv_rows;
    const int n_blk = (key_begin + n_pre + n_tree - 1) / a.kv_rows - first_blk + 1;
    const int32_t* bt = a.block_table + static_cast<int64_t>(b) * a.max_blocks + first_blk;
    // (stored as the block's row group of head g, blk * Hkv + g: its first
    // row is that times kv_rows)
    for (int j = tid; j < n_blk; j += kThreads) sm.blk[j] = bt[j] * a.Hkv + g;
    __syncthreads();
  }
  auto row_byte = [&](int row) -> int64_t {  // byte offset of logical cache row `row`
    if (!paged) return ((static_cast<int64_t>(b) * a.Hkv + g) * a.kv_rows + row) * (HD * 2);
    if (a.kv_shift >= 0) {  // power-of-two blocks: shifts and masks, no division
      const int64_t rg = sm.blk[(row >> a.kv_shift) - first_blk];
      return ((rg << a.kv_shift) + (row & (a.kv_rows - 1))) * (HD * 2);
    }
    const int64_t rg = sm.blk[row / a.kv_rows - first_blk];
    return (rg * a.kv_rows + row % a.kv_rows) * (HD * 2);
  };
  // A lane's byte offset of its chunk within a cache row.  The LDS tile keeps
  // 128-dim rows whatever the head size; with 64 dims each row's 8 chunks
  // fill both halves of its LDS row (the upper half is never read).
  int k_off[kKLoads], v_off[kKLoads];
  uint32_t k_voff[kKLoads], v_voff[kKLoads];
#pragma unroll
  for (int u = 0; u < kKLoads; ++u) {
    k_off[u] = lp.k_off[u] & (HD * 2 - 1);
    v_off[u] = lp.v_off[u] & (HD * 2 - 1);
    k_voff[u] = static_cast<uint32_t>(lp.k_key[u] * (HD * 2) + k_off[u]);
    v_voff[u] = static_cast<uint32_t>(lp.v_key[u] * (HD * 2) + v_off[u]);
  }
  // Paged caches with power-of-two blocks of at least 4 rows: the 4 keys a
  // load instruction covers are 4-aligned, so in a full prefix tile (which
  // starts at a multiple of 64) they lie in one block.  Each instruction then
  // takes a wave-uniform base, from its block id, in scalar registers, plus a
  // loop-invariant per-lane offset within the block.
  const bool paged_uniform = paged && a.kv_shift >= 2;
  const int in_blk = (a.kv_rows < kKT ? a.kv_rows : kKT) - 1;  // key bits inside a block (of a tile)
  uint32_t k_poff[kKLoads], v_poff[kKLoads];
  int k_grp[kKLoads], v_grp[kKLoads];  // first tile key of each instruction (lane 0's)
#pragma unroll
  for (int u = 0; u < kKLoads; ++u) {
    k_poff[u] = static_cast<uint32_t>((lp.k_key[u] & in_blk) * (HD * 2) + k_off[u]);
    v_poff[u] = static_cast<uint32_t>((lp.v_key[u] & in_blk) * (HD * 2) + v_off[u]);
    k_grp[u] = __builtin_amdgcn_readfirstlane(lp.k_key[u]);
    v_grp[u] = __builtin_amdgcn_readfirstlane(lp.v_key[u]);
  }
  // For a full prefix tile (rows from a multiple of 64) the block of load u is
  // the tile's first block plus k_grp[u] >> kv_shift (0 for blocks of 64 rows
  // or more); a row group's first byte is rg << rg_shift.
  int k_lix[kKLoads], v_lix[kKLoads];
#pragma unroll
  for (int u = 0; u < kKLoads; ++u) {
    k_lix[u] = a.kv_shift <= 6 ? k_grp[u] >> a.kv_shift : 0;
    v_lix[u] = a.kv_shift <= 6 ? v_grp[u] >> a.kv_shift : 0;
  }
  const int rg_shift = a.kv_shift + (HD == 128 ? 8 : 7);
  // LDS byte addresses of the ring and of this wave's 1 KiB block in a slot,
  // worked out once: a slot's load targets are then scalar adds.
  const uint32_t ring_lds = lds_addr(&sm.kv[0][0]);
  uint32_t pos_lds[kKLoads];
#pragma unroll
  for (int u = 0; u < kKLoads; ++u) pos_lds[u] = __builtin_amdgcn_readfirstlane(lp.lds_pos[u]);
  auto issue_tile = [&](int t) {
    const uint32_t k_lds = ring_lds + (t % kStages) * kTileBytes;
    const uint32_t v_lds = k_lds + kKBytes;
    const TileRef tr = tile_ref(t);
    if (paged_uniform && !tr.tree && tr.left >= kKT && (tr.row & (kKT - 1)) == 0) {
      const int64_t in_row = a.kv_rows > kKT ? static_cast<int64_t>(tr.row & (a.kv_rows - 1)) * (HD * 2) : 0;
      const int tb = (tr.row >> a.kv_shift) - first_blk;  // the tile's first block
      int bk[kKLoads], bv[kKLoads];
#pragma unroll
      for (int u = 0; u < kKLoads; ++u) {
        bk[u] = sm.blk[tb + k_lix[u]];
        bv[u] = sm.blk[tb + v_lix[u]];
      }
#pragma unroll
      for (int u = 0; u < kKLoads; ++u) {
        const int64_t kr = __builtin_amdgcn_readfirstlane(bk[u]);
        const int64_t vr = __builtin_amdgcn_readfirstlane(bv[u]);
        dma16(k_lds + pos_lds[u], kbase + ((kr << rg_shift) + in_row), k_poff[u]);
        dma16(v_lds + pos_lds[u], vbase + ((vr << rg_shift) + in_row), v_poff[u]);
      }
    } else if (!paged && tr.left >= kKT) {
      // contiguous rows: a uniform tile base plus per-lane 32-bit offsets
      const int64_t base = row_byte(tr.row);
#pragma unroll
      for (int u = 0; u < kKLoads; ++u) {
        dma16(k_lds + pos_lds[u], kbase + base, k_voff[u]);
        dma16(v_lds + pos_lds[u], vbase + base, v_voff[u]);
      }
    } else {
      // paged rows, or a range's last partial tile (keys past the range's end
      // read its last row and are masked out)
#pragma unroll
      for (int u = 0; u < kKLoads; ++u) {
        const int kk = tr.row + min(lp.k_key[u], tr.left - 1);
        const int vk = tr.row + min(lp.v_key[u], tr.left - 1);
        dma16(k_lds + pos_lds[u], kbase + row_byte(kk) + k_off[u]);
        dma16(v_lds + pos_lds[u], vbase + row_byte(vk) + v_off[u]);
      }
    }
  };

  // The first tiles, behind Q.
#pragma unroll
  for (int t = 0; t < kStages - 2; ++t)
    if (t < n_tiles) issue_tile(t);
  // This wave's Q rows and parent links have landed once no more than the
  // tiles' loads are outstanding.
  if (n_tiles >= 2)
    wait_vmcnt<2 * kLoadsPerTile>();
  else if (n_tiles == 1)
    wait_vmcnt<kLoadsPerTile>();
  else
    wait_vmcnt<0>();

  // ---- Q fragment (B operand of S^T): lane holds row l32 of the wave's
  // 32-row block, dims 16*kk + 8*h .. +7.  All waves have read theirs before
  // the loop's first barrier, after which tile 2 overwrites the slot.
  bf16x8 qf[HD / 16];
  if (active) {
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk)
      qf[kk] = *reinterpret_cast<const bf16x8*>(q_lds + l32 * (kD * 2) +
                                                (((2 * kk + h) ^ (l32 & 15)) << 4));
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");

  // The tree's parent links, for wave 0 (lane l handles nodes l + 64*k).
  int my_parent[kNodesPerLane];
#pragma unroll
  for (int k = 0; k < kNodesPerLane; ++k) {
    const int i = lane + kWave * k;
    my_parent[k] = -1;
    if (kTree && wave == 0 && i > 0 && i < n) my_parent[k] = sm.par[i];
  }

  // ---- ancestor masks (tree split): wave 0 builds them by pointer doubling
  // over the parent links, anc(i) |= anc(jump(i)), jump(i) = jump(jump(i)).
  // Each lane keeps the sets and jump pointers of its nodes (i = lane + 64*k)
  // in registers; a round publishes them to LDS, orders the wave's LDS
  // traffic with one wave-level fence, and reads the jump targets' entries.
  // The rounds stop once every jump pointer has passed the root (after
  // ceil(log2(depth + 1)) rounds).  The other waves go on to the tile loop,
  // whose first barrier publishes the masks.
  if (kTree && wave == 0) {
    typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
    u32x8 anc_r[kNodesPerLane];
    int jmp[kNodesPerLane];
#pragma unroll
    for (int k = 0; k < kNodesPerLane; ++k) {
      const int i = lane + kWave * k;
#pragma unroll
      for (int w = 0; w < kAncWords; ++w) anc_r[k][w] = (i < n && (i >> 5) == w) ? (1u << (i & 31)) : 0u;
      jmp[k] = my_parent[k];
    }
    u32x8* anc_lds = reinterpret_cast<u32x8*>(&sm.anc[0][0]);
    for (int r = 0; r < 8; ++r) {
#pragma unroll
      for (int k = 0; k < kNodesPerLane; ++k) {
        if (k < nslots) {
          const int i = lane + kWave * k;
          anc_lds[i] = anc_r[k];
          sm.jump[i] = static_cast<int16_t>(jmp[k]);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      bool live = false;
#pragma unroll
      for (int k = 0; k < kNodesPerLane; ++k) {
        if (k < nslots) {
          const int j = jmp[k];
          const int jc = j >= 0 ? j : 0;
          const u32x8 other = anc_lds[jc];
          const int jj = sm.jump[jc];
          if (j >= 0) {
            anc_r[k] |= other;
            jmp[k] = jj;
          }
          live |= jmp[k] >= 0;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      if (__builtin_amdgcn_ballot_w64(live) == 0) break;
    }
#pragma unroll
    for (int k = 0; k < kNodesPerLane; ++k) {
      const int i = lane + kWave * k;
      if (i < n) anc_lds[i] = anc_r[k];
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }

  // ---- online softmax state (raw score units) and O^T accumulators
  // m starts at the most negative finite float: the first key that is not
  // masked moves it (a score at that very value gets weight 2^0), and no step
  // needs a case for -inf.
  float m_run = kNoMax, l_run = 0.f;
  f32x16 o_acc[HD / 32];
#pragma unroll
  for (int db = 0; db < HD / 32; ++db) o_acc[db] = f32x16{};
  const float c = a.scale_log2;

  // LDS read offsets (bytes within a tile), all loop-invariant:
  //  K operand, 16-dim step kk: row l32 of the 32-row block, chunk
  //  (2*kk + h) ^ (l32 & 15).
  int k_rd[HD / 16];
#pragma unroll
  for (int kk = 0; kk < HD / 16; ++kk)
    k_rd[kk] = l32 * (kD * 2) + (((2 * kk + h) ^ (l32 & 15)) << 4);
  //  V^T operand: 16-lane group q reads key 16*(q/2) + s/4 (+ the k-step's
  //  base, a multiple of 4), dims 32*db + 16*(q%2) + 4*(s%4).
  const int tr_q = lane >> 4, tr_s = lane & 15;
  const int tr_key = 16 * (tr_q >> 1) + (tr_s >> 2);
  int v_rd[HD / 32];
#pragma unroll
  for (int db = 0; db < HD / 32; ++db) {
    const int dim = 32 * db + 16 * (tr_q & 1) + 4 * (tr_s & 3);
    v_rd[db] = tr_key * (kD * 2) + (((dim >> 3) ^ swz_v(tr_key)) << 4) + (dim & 7) * 2;
  }

  // K fragments of a tile (A operand of S^T), read into registers one phase
  // ahead of their MFMAs.
  bf16x8 af[2][HD / 16];
  auto load_k = [&](int t) {
    const unsigned char* k_s = sm.kv[t % kStages];
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        af[kb][kk] = *reinterpret_cast<const bf16x8*>(k_s + kb * 32 * (kD * 2) + k_rd[kk]);
  };
  // S^T = K Q^T from the fragments in af, the two 32-key blocks interleaved.
  auto scores = [&](f32x16(&s)[2]) {
    s[0] = s[1] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[kb][kk], qf[kk], s[kb], 0, 0, 0);
  };

  // The online softmax of a tile in three parts: the key mask (tiles that
  // hold tree keys or end their range), the exponentials (writes the P^T
  // fragments; the reference max m moves only when a score exceeds it by
  // 2^kLazyMax) and the finish, which rescales O and l when some lane's m
  // moved.  The finish must come after the previous tile's P.V product.
  auto mask_scores = [&](int t, f32x16(&s)[2]) {
    const TileRef tr = tile_ref(t);
    if (tr.tree || tr.left < kKT) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int kfirst = kb * 32 + 16 * h;  // tile key of register r = kfirst + r
        uint32_t vis = 0xFFFFu;
        if (kfirst + 16 > tr.left) vis = (kfirst >= tr.left) ? 0u : ((1u << (tr.left - kfirst)) - 1u);
        if (tr.tree) vis &= (sm.anc[qnode][(tr.rel + kb * 32) >> 5] >> (16 * h)) & 0xFFFFu;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (!((vis >> r) & 1u)) s[kb][r] = -INFINITY;
      }
    }
  };
  float m_new = kNoMax, psum = 0.f;
  auto exponentials = [&](f32x16(&s)[2], bf16x8(&pf)[2][2]) {
    // IEEE maximum (NaN-propagating) needs no operand canonicalisation and
    // maps to three-input v_maximum3_f32.
    float tmax = __builtin_elementwise_maximum(s[0][0], s[0][1]);
#pragma unroll
    for (int r = 2; r < 32; r += 2)
      tmax = __builtin_elementwise_maximum(__builtin_elementwise_maximum(tmax, s[r >> 4][r & 15]),
                                           s[r >> 4][(r & 15) + 1]);
    tmax = max_xor32(tmax);
    // (scale > 0, so the lazy test can run on raw scores)
    m_new = tmax > m_run + a.lazy_gap ? tmax : m_run;
    const float neg = -m_new * c;
    // The row sum adds the rounded bf16 probabilities, two per
    // v_dot2_f32_bf16 with ones: the very weights P.V multiplies.
    const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
    float ps = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        u32x4 pk;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p0 = exp2_fast(__builtin_fmaf(s[kb][8 * kk + 2 * j], c, neg));
          const float p1 = exp2_fast(__builtin_fmaf(s[kb][8 * kk + 2 * j + 1], c, neg));
          // (summed before it goes into the vector: hipcc folds a bf16x2
          // bit-cast of element j of a u32x4 to element 0)
          const bf16x2 w = __builtin_convertvector((f32x2){p0, p1}, bf16x2);
          ps = __builtin_amdgcn_fdot2_f32_bf16(w, ones, ps, false);
          pk[j] = __builtin_bit_cast(uint32_t, w);
        }
        pf[kb][kk] = __builtin_bit_cast(bf16x8, pk);
      }
    }
    psum = ps;
  };
  auto finish_softmax = [&]() {
    if (__builtin_amdgcn_ballot_w64(m_new != m_run) != 0) {
      const float alpha = exp2_fast((m_run - m_new) * c);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < HD / 32; ++db) o_acc[db] *= alpha;
    }
    l_run += psum;
    m_run = m_new;
  };

  // O^T += V^T P^T for tile t; k-step kc = 2*kb + kk covers keys 32*kb +
  // 16*h + 8*kk .. +7, read as two transposed 4-key reads.
  auto accumulate = [&](int t, const bf16x8(&pf)[2][2]) {
    const unsigned char* v_s = sm.kv[t % kStages] + kKBytes;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      const int koff = (32 * (kc >> 1) + 8 * (kc & 1)) * (kD * 2);
      bf16x8 vf[HD / 32];
#pragma unroll
      for (int db = 0; db < HD / 32; ++db) {
        const s16x4 lo = lds_read_tr(v_s + v_rd[db] + koff);
        const s16x4 hi = lds_read_tr(v_s + v_rd[db] + koff + 4 * (kD * 2));
        vf[db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int db = 0; db < HD / 32; ++db)
        o_acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db], pf[kc >> 1][kc & 1], o_acc[db], 0, 0, 0);
    }
  };

  // ---- tile loop, software-pipelined by one phase: iteration t runs the
  // P.V product of tile t-1 together with the softmax of tile t (one block
  // of MFMAs and independent vector work for the scheduler to interleave),
  // then publishes tile t+1, reads its K fragments and issues its S MFMAs.
  // V of tile t-1 is still read in iteration t, so loads run kAhead =
  // kStages - 2 tiles ahead and never refill a slot that is in use: the
  // barrier that publishes tile t+1 comes after the last read of tile t-1.
  constexpr int kAhead = kStages - 2;
  static_assert(kAhead == 2, "the vmcnt waits below assume two tiles of look-ahead");
  auto publish = [&](int t) {  // wait for tile t, publish it, start loading tile t + kAhead
    if (t + 1 < n_tiles) wait_vmcnt<kLoadsPerTile>();  // tile t+1 may stay in flight
    else wait_vmcnt<0>();
    barrier_only();  // tile t landed for all waves; every wave is done with tile t-2
    if (t + kAhead < n_tiles) issue_tile(t + kAhead);
  };
  // The P^T fragments alternate between two register sets (the loop is
  // unrolled by two), so tile t-1's are never copied.
  f32x16 s_acc[2];
  bf16x8 pfa[2][2], pfb[2][2];
  auto body = [&](int t, const bf16x8(&pf_prev)[2][2], bf16x8(&pf)[2][2]) {
    publish(t);
    if (active) {
      load_k(t);
      scores(s_acc);
      mask_scores(t, s_acc);
      accumulate(t - 1, pf_prev);  // tile t-1's P.V ...
      exponentials(s_acc, pf);     // ... interleaved with tile t's softmax
      // (pins P and its row sum ahead of the rescale branch: otherwise the
      // compiler sinks the exponentials past it, out of reach of the P.V
      // MFMAs they can overlap)
      asm volatile("" : "+v"(pf[0][0]), "+v"(pf[0][1]), "+v"(pf[1][0]), "+v"(pf[1][1]), "+v"(psum));
      finish_softmax();            // after P.V(t-1): may rescale O
    }
  };
  if (n_tiles > 0) {
    publish(0);
    if (active) {
      load_k(0);
      scores(s_acc);
      mask_scores(0, s_acc);
      exponentials(s_acc, pfa);
      finish_softmax();
    }
  }
  int t = 1;
  for (; t + 1 < n_tiles; t += 2) {
    body(t, pfa, pfb);
    body(t + 1, pfb, pfa);
  }
  if (t < n_tiles) {
    body(t, pfa, pfb);
    if (active) accumulate(n_tiles - 1, pfb);
  } else if (n_tiles > 0 && active) {
    accumulate(n_tiles - 1, pfa);
  }

  // ---- results.  For a whole unit the normalised output O / l goes straight
  // to `out`.  Otherwise the share's partial result: (max in log2 units, sum)
  // in fp32 and O / l in bf16 (half the bytes of raw fp32 partials; the merge
  // weights each piece by 2^(m - M) * l), at the unit's row r in slot `slot`.
  // The O rows pass through LDS so that every store writes whole 256-byte rows
  // (a wave's 32 partial rows are one contiguous 8 KiB block of the
  // workspace).  Partials are stored non-temporally: keeping them dirty in
  // this XCD's L2 only lengthens the write-back at the end of the kernel.
  constexpr int kRowPitch = kD * 2 + 16;  // padded LDS row (bank spread)
  static_assert(kWaves * 32 * kRowPitch <= kStages * kTileBytes, "staging fits the ring");
  const int64_t part = static_cast<int64_t>(slot) * kTileRows - row0;  // + absolute row
  barrier_only();  // every wave is done with the K/V ring; reuse it for staging
  if (!active) return;
  unsigned char* stage = &sm.kv[0][0] + wave * (32 * kRowPitch);  // spans ring slots
  {
    const float lsum = l_run + xor32(l_run);
    if (!final_out && qvalid && h == 0) {
      f32x2 ml = {lsum > 0.f ? m_run * c : -INFINITY, lsum};
      __builtin_nontemporal_store(ml, reinterpret_cast<f32x2*>(a.ws_ml + (part + qrow_idx) * 2));
    }
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    unsigned char* srow = stage + l32 * kRowPitch;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint2 v;
        v.x = pack_bf16x2(o_acc[db][4 * j] * inv, o_acc[db][4 * j + 1] * inv);
        v.y = pack_bf16x2(o_acc[db][4 * j + 2] * inv, o_acc[db][4 * j + 3] * inv);
        *reinterpret_cast<uint2*>(srow + (db * 32 + 8 * j + 4 * h) * 2) = v;
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  constexpr int kRowChunks = HD * 2 / 16;       // 16-byte chunks of an output row
  constexpr int kChunks = 32 * kRowChunks;       // ... of this wave's rows
  static_assert(kChunks % kWave == 0, "whole store rounds");
  const int wrow0 = row0 + wave * 32;
  // (an opaque copy of the lane index: otherwise the compiler shares the
  // chunk indices below with the parent-link loads before the tile loop and
  // keeps them live, and spills them, across it)
  int lane_e = lane;
  asm volatile("" : "+v"(lane_e));
  if (final_out) {
    // stacked row r = node * G + head in group -> out[b][node][g * G + head]
#pragma unroll
    for (int i = 0; i < kChunks / kWave; ++i) {
      const int cidx = i * kWave + lane_e;
      const int r = cidx / kRowChunks, col = cidx % kRowChunks;
      const int row = wrow0 + r;
      if (row < valid_rows) {
        uint16_t* orow =
            a.out + ((static_cast<int64_t>(b) * a.Nmax + row / a.G) * a.Hq + g * a.G + row % a.G) * HD;
        *reinterpret_cast<u32x4*>(orow + col * 8) =
            *reinterpret_cast<const u32x4*>(stage + r * kRowPitch + col * 16);
      }
    }
    return;
  }
  unsigned char* gbase = reinterpret_cast<unsigned char*>(a.ws_o + (part + wrow0) * kD);
#pragma unroll
  for (int i = 0; i < kChunks / kWave; ++i) {
    const int cidx = i * kWave + lane_e;
    const int r = cidx / kRowChunks, col = cidx % kRowChunks;
    if (wrow0 + r < valid_rows)
      __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(stage + r * kRowPitch + col * 16),
                                  reinterpret_cast<u32x4*>(gbase + r * (kD * 2) + col * 16));
  }
}

// ---- the call's work axis (stream_plan.hpp), computed by each wave on its
// own: lane l holds sequence c * 64 + l of chunk c.  Prefix lengths and node
// counts are clamped into the range the launch was sized for, so malformed
// data without validation cannot move any position off the planned axis.

__device__ __forceinline__ plan::SeqCost lane_cost(const MfmaArgs& a, int b, int* P, int* n) {
  *P = 0;
  *n = 1;
  if (b < a.B) {
    *P = min(max(a.prefix_len[b], 0), a.max_prefix);
    *n = min(max(a.n_nodes[b], 1), a.Nmax);
  }
  return plan::seq_cost(*P, *n, a.G);
}

__device__ __forceinline__ int64_t shfl_up_i64(int64_t v, int d) {
  const int lo = __shfl_up(static_cast<int>(v), d, kWave);
  const int hi = __shfl_up(static_cast<int>(v >> 32), d, kWave);
  return (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
}
__device__ __forceinline__ int64_t readlane_i64(int64_t v, int l) {
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(v), l);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(v >> 32), l);
  return (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
}

// The call's sequence table on the axis, one sequence per lane: lane l of a
// wave holds sequence l (its clamped prefix length and node count, first axis
// position and axis length), and every lane holds the total length C.  With
// more than 64 sequences the lanes hold the first 64 and positions past them
// are found by rescanning the table (axis_find).
struct Axis {
  int P, n;
  int64_t start, len;
  int ubase;  // index of this lane's sequence's first unit
  int64_t C;
  int units;  // units of the whole call
};

// Inclusive prefix sum over the wave.
__device__ __forceinline__ int64_t wave_scan_i64(int64_t x) {
  const int lane = __lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t y = shfl_up_i64(x, d);
    if (lane >= d) x += y;
  }
  return x;
}

__device__ Axis axis_load(const MfmaArgs& a) {
  const int lane = __lane_id();
  Axis ax{};
  if (a.B == 1) {
    // one sequence: scalar loads (a short round trip) and no scans
    const int P = min(max(a.prefix_len[0], 0), a.max_prefix);
    const int n = min(max(a.n_nodes[0], 1), a.Nmax);
    const plan::SeqCost c = plan::seq_cost(P, n, a.G);
    ax.P = P;
    ax.n = n;
    ax.start = 0;
    ax.ubase = 0;
    ax.len = lane == 0 ? a.Hkv * c.per_head : 0;
    ax.C = a.Hkv * c.per_head;
    ax.units = a.Hkv * c.rt;
    return ax;
  }
  int64_t base = 0;
  int ubase = 0;
  for (int c0 = 0; c0 < a.B; c0 += kWave) {
    int P, n;
    const plan::SeqCost c = lane_cost(a, c0 + lane, &P, &n);
    const int64_t len = c0 + lane < a.B ? a.Hkv * c.per_head : 0;
    const int64_t x = wave_scan_i64(len);
    const int nu = c0 + lane < a.B ? a.Hkv * c.rt : 0;
    const int xu = static_cast<int>(wave_scan_i64(nu));
    if (c0 == 0) {
      ax.P = P;
      ax.n = n;
      ax.start = x - len;
      ax.len = len;
      ax.ubase = xu - nu;
    }
    base += readlane_i64(x, kWave - 1);
    ubase += __builtin_amdgcn_readlane(xu, kWave - 1);
  }
  ax.C = base;
  ax.units = ubase;
  return ax;
}

// The sequence whose units hold axis position p (0 <= p < C).
__device__ plan::SeqAt axis_find(const MfmaArgs& a, const Axis& ax, int64_t p) {
  plan::SeqAt r{};
  const uint64_t hit = __ballot(ax.len > 0 && ax.start <= p && p < ax.start + ax.len);
  if (hit != 0) {
    const int l = __ffsll(static_cast<long long>(hit)) - 1;
    r.b = l;
    r.P = __builtin_amdgcn_readlane(ax.P, l);
    r.n = __builtin_amdgcn_readlane(ax.n, l);
    r.pre = readlane_i64(ax.start, l);
    r.ubase = __builtin_amdgcn_readlane(ax.ubase, l);
    r.c = plan::seq_cost(r.P, r.n, a.G);
    return r;
  }
  // past the first 64 sequences: rescan the table from the second chunk on
  const int lane = __lane_id();
  int64_t base = readlane_i64(ax.start + ax.len, kWave - 1);
  int ubase = __builtin_amdgcn_readlane(ax.ubase, kWave - 1) +
              __builtin_amdgcn_readlane(a.Hkv * plan::seq_cost(ax.P, ax.n, a.G).rt, kWave - 1);
  for (int c0 = kWave; c0 < a.B; c0 += kWave) {
    int P, n;
    const plan::SeqCost c = lane_cost(a, c0 + lane, &P, &n);
    const int64_t len = c0 + lane < a.B ? a.Hkv * c.per_head : 0;
    const int64_t x = wave_scan_i64(len);
    const int nu = c0 + lane < a.B ? a.Hkv * c.rt : 0;
    const int xu = static_cast<int>(wave_scan_i64(nu));
    const int64_t start = base + x - len;
    const uint64_t h = __ballot(len > 0 && start <= p && p < start + len);
    if (h != 0) {
      const int l = __ffsll(static_cast<long long>(h)) - 1;
      r.b = c0 + l;
      r.P = __builtin_amdgcn_readlane(P, l);
      r.n = __builtin_amdgcn_readlane(n, l);
      r.pre = readlane_i64(start, l);
      r.ubase = ubase + __builtin_amdgcn_readlane(xu - nu, l);
      r.c = plan::seq_cost(r.P, r.n, a.G);
      return r;
    }
    base += readlane_i64(x, kWave - 1);
    ubase += __builtin_amdgcn_readlane(xu, kWave - 1);
  }
  return r;  // not reached for p < C
}

// What the merge kernel needs of a unit: whether it was cut and, if so, its
// pieces (plan::MergeJob), written by the attention workgroup that owns the
// unit's tree block so that the merge workgroups do not redo the partition's
// arithmetic.  Entry i of the table is the call's unit i; the table's header
// holds the call's unit count (entries past it are left from other calls).
struct MergeDesc {
  int32_t active, b, g, rt, n, sa, sa_first, t_pre;
  int64_t U, C;
  int32_t w, pad[3];
};
static_assert(sizeof(MergeDesc) == 64, "descriptor layout");

// Workgroup w of the grid takes stream index s: the workgroups on one XCD
// (w mod 8; the hardware deals workgroups to the 8 XCDs round robin) take one
// contiguous eighth of the axis, in launch order, so the row tiles of one
// (sequence, kv head), which read the same keys, run side by side on one L2.
__device__ __forceinline__ int stream_index(int w, int W) { return (w % 8) * (W / 8) + w / 8; }

// ---- split plan (one sequence): grid = (b * Hkv + g, row tile, KV split).
// Each (sequence, kv head, row tile) unit is cut into KV splits of
// split_keys prefix keys; the tree's keys join the last split or take one of
// their own.  (sequence, kv head) is the fastest grid dimension: workgroups
// are dealt to the 8 XCDs by linear id modulo 8, so each kv head's splits
// share one XCD (its L2 holds their common Q rows and K/V).  A unit with one
// split writes its output directly; otherwise split sp leaves its partial in
// slot (bg * max_splits + sp) * row_tiles + row tile.
template <int HD, bool kPaged>
__global__ void __launch_bounds__(kThreads, 1) attn_split_kernel(MfmaArgs a) {
  __shared__ __attribute__((aligned(16))) Smem sm;
  const int bg = blockIdx.x;
  const int rtile = blockIdx.y;
  const int split = blockIdx.z;
  const int b = bg / a.Hkv;
  const int g = bg % a.Hkv;
  if (halted(a.status)) return;
  const int P = a.prefix_len[b];
  const int n = a.n_nodes[b];
  const int nsp = n_splits_of(P, n, a.split_keys, a.tree_alone);
  if (split >= nsp) return;
  const int valid_rows = a.G * n;
  const int row0 = rtile * kTileRows;
  if (row0 >= valid_rows) return;
  // Prefix keys [key_begin, key_begin + n_pre); a tree split of its own
  // starts at P with none.
  const int key_begin = min(split * a.split_keys, P);
  const int n_pre = min(a.split_keys, P - key_begin);
  const int slot = (bg * a.max_splits + split) * a.row_tiles + rtile;
  if (split == nsp - 1)
    attend<true, HD, kPaged>(a, sm, b, g, row0, valid_rows, key_begin, n_pre, P, n, nsp == 1, slot);
  else
    attend<false, HD, kPaged>(a, sm, b, g, row0, valid_rows, key_begin, n_pre, P, n, nsp == 1, slot);
}

// Split plan merge, one wave per stacked row: combine the splits' partials
//   out = sum_s w_s * Ohat_s / sum_s w_s,  w_s = 2^(m_s - M) * l_s,  M = max_s m_s,
// where Ohat_s = O_s / l_s is the split's normalised output (bf16).  Lane s
// takes split s's (m, l); the 4 groups of 16 lanes each read one split's row
// (16 bytes = 8 dims per lane) per step, so 4 splits' rows are in flight per
// load, and the groups' sums are added with two lane exchanges.  The kernel
// is latency-bound, so the (m, l) pairs and the first 16 splits' rows are
// requested before the sequence's prefix length and node count arrive: every
// row of the grid is inside the workspace's Mpad rows, and every split index
// below max_splits inside its splits.
template <int HD>
__global__ void __launch_bounds__(256) attn_split_merge_kernel(MfmaArgs a) {
  __shared__ float w_s[4][kMaxMergeSplits];
  constexpr int kFirst = 16;  // splits whose rows are requested up front
  const int bg = blockIdx.x;
  const int b = bg / a.Hkv;
  const int g = bg % a.Hkv;
  if (halted(a.status)) return;
  const int wv = threadIdx.x / kWave;
  const int row = blockIdx.y * 4 + wv;
  const int lane = threadIdx.x % kWave;
  const int grp = lane >> 4, col = lane & 15;  // split offset, 8-dim chunk
  const int Mpad = a.row_tiles * kTileRows;  // rows of a (sequence, kv head) unit set
  const int64_t part0 = static_cast<int64_t>(bg) * a.max_splits * Mpad + row;
  const unsigned char* op = reinterpret_cast<const unsigned char*>(a.ws_o + part0 * kD) + col * 16;
  const int64_t stride = static_cast<int64_t>(Mpad) * kD * 2;  // bytes between splits
  f32x2 ml0 = {-INFINITY, 0.f};
  if (lane < a.max_splits) ml0 = *reinterpret_cast<const f32x2*>(a.ws_ml + (part0 + lane * Mpad) * 2);
  u32x4 o0[kFirst / 4];
#pragma unroll
  for (int u = 0; u < kFirst / 4; ++u) {
    const int sp = 4 * u + grp;
    o0[u] = sp < a.max_splits ? *reinterpret_cast<const u32x4*>(op + sp * stride)
                              : (u32x4){0u, 0u, 0u, 0u};
  }
  const int n = a.n_nodes[b];
  const int P = a.prefix_len[b];
  if (row >= a.G * n) return;
  // (clamped so that a prefix above the planned maximum cannot index past the
  // workspace; such input is malformed and caught when validation is on)
  const int n_splits = min(n_splits_of(P, n, a.split_keys, a.tree_alone), a.max_splits);
  if (n_splits == 1) return;  // the attention kernel wrote this row's output
  float M = lane < n_splits ? ml0.x : -INFINITY;
  for (int s = lane + kWave; s < n_splits; s += kWave) M = fmaxf(M, a.ws_ml[(part0 + s * Mpad) * 2]);
  M = wave_max(M);
  float wsum = 0.f;
  for (int s = lane; s < n_splits; s += kWave) {
    const f32x2 ml = s == lane ? ml0 : *reinterpret_cast<const f32x2*>(a.ws_ml + (part0 + s * Mpad) * 2);
    const float w = exp2_fast(ml.x - M) * ml.y;
    w_s[wv][s] = w;
    wsum += w;
  }
  wsum = wave_sum(wsum);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  auto fold = [&](const u32x4& o, float w) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += w * bf16_to_f32(static_cast<uint16_t>(o[e] & 0xFFFFu));
      acc[2 * e + 1] += w * bf16_to_f32(static_cast<uint16_t>(o[e] >> 16));
    }
  };
#pragma unroll
  for (int u = 0; u < kFirst / 4; ++u) {
    const int sp = 4 * u + grp;
    if (sp < n_splits) fold(o0[u], w_s[wv][sp]);
  }
  for (int s0 = kFirst; s0 < n_splits; s0 += 16) {
    u32x4 o[4];
    float w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int sp = s0 + 4 * u + grp;
      o[u] = (u32x4){0u, 0u, 0u, 0u};
      w[u] = 0.f;
      if (sp < n_splits) {
        o[u] = *reinterpret_cast<const u32x4*>(op + sp * stride);
        w[u] = w_s[wv][sp];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) fold(o[u], w[u]);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    acc[e] += __shfl_xor(acc[e], 16, kWave);
    acc[e] += __shfl_xor(acc[e], 32, kWave);
  }
  if (grp == 0 && col < HD / 8) {  // (lanes past the head's dims summed unused workspace)
    const float inv = 1.f / wsum;
    const int node = row / a.G;
    const int hq = g * a.G + row % a.G;
    uint16_t* orow = a.out + ((static_cast<int64_t>(b) * a.Nmax + node) * a.Hq + hq) * HD;
    u32x4 v;
    v.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    v.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
    v.z = pack_bf16x2(acc[4] * inv, acc[5] * inv);
    v.w = pack_bf16x2(acc[6] * inv, acc[7] * inv);
    *reinterpret_cast<u32x4*>(orow + col * 8) = v;
  }
}


// ---- stream plan (batches): the workgroup's shares are planned in rounds of up to kMaxShares by wave 0
// into LDS, then run one by one by the whole workgroup: the partition's state
// (the sequence table, positions) is dead while the tile loop runs, which
// keeps it out of the loop's registers.
template <int HD, bool kPaged>
__global__ void __launch_bounds__(kThreads, 1) attn_stream_kernel(MfmaArgs a) {
  __shared__ __attribute__((aligned(16))) Smem sm;
  if (halted(a.status)) return;
  const int s = stream_index(blockIdx.x, a.W);
  const int wave = threadIdx.x / kWave;
  bool started = false;
  for (int round = 0;; ++round) {
    if (wave == 0) {
      const Axis ax = axis_load(a);
      auto find = [&](int64_t p) { return axis_find(a, ax, p); };
      const plan::Grid gr = plan::make_grid(ax.C, a.W);
      if (blockIdx.x == 0 && round == 0 && threadIdx.x == 0)
        *reinterpret_cast<int32_t*>(a.ws_desc) = ax.units;  // the merge table's header
      bool first = round == 0 ? true : sm.first != 0;
      const int64_t pos = round == 0 ? plan::range_lo(gr, s) : sm.next_pos;
      int k = 0;
      const int64_t next = plan::walk_shares(
          s, gr, pos, first, kMaxShares, find,
          [&](const plan::SeqAt& q, const plan::Unit& u, int64_t U, const plan::Share& sh,
              bool whole, int slot) {
            const plan::KeyRange keys = plan::share_keys(sh, q.P);
            if (threadIdx.x == 0)
              sm.share[k] = ShareDesc{q.b, u.g, u.rt, q.P, q.n, keys.begin, keys.count,
                                      sh.tree ? 1 : 0, whole ? 1 : 0, slot};
            ++k;
            if (sh.tree) {  // this workgroup owns the unit's last item: its merge entry
              const plan::MergeJob job = plan::unit_job(q, u, U, s, gr, find);
              if (threadIdx.x == 0) {
                MergeDesc d{};
                d.active = job.active;
                d.b = q.b;
                d.g = u.g;
                d.rt = u.rt;
                d.n = q.n;
                d.sa = job.sa;
                d.sa_first = job.sa_first;
                d.t_pre = q.c.t_pre;
                d.U = U;
                d.C = ax.C;
                d.w = u.w;
                a.ws_desc[1 + plan::unit_index(q, u)] = d;
              }
            }
          });
      if (threadIdx.x == 0) {
        sm.n_share = k;
        sm.first = first ? 1 : 0;
        sm.next_pos = next < plan::range_lo(gr, s + 1) ? next : -1;
      }
    }
    __syncthreads();
    const int n_share = sm.n_share;
    const int64_t next_pos = sm.next_pos;
    for (int i = 0; i < n_share; ++i) {
      if (started) __syncthreads();  // the last share's staging is done with the ring
      started = true;
      const ShareDesc d = sm.share[i];
      const int row0 = d.rt * kTileRows;
      if (d.tree)
        attend<true, HD, kPaged>(a, sm, d.b, d.g, row0, a.G * d.n, d.key_begin, d.n_pre, d.P, d.n,
                     d.whole != 0, d.slot);
      else
        attend<false, HD, kPaged>(a, sm, d.b, d.g, row0, a.G * d.n, d.key_begin, d.n_pre, d.P, d.n,
                      d.whole != 0, d.slot);
    }
    if (next_pos < 0) break;
    __syncthreads();  // every wave has read this round's shares
  }
}

// Merge of a unit cut between workgroups: out = sum_p w_p * Ohat_p / sum_p w_p,
// w_p = 2^(m_p - M) * l_p, M = max_p m_p, over the unit's pieces p in
// workgroup order, where Ohat_p = O_p / l_p is the piece's normalised output
// (bf16).  blockIdx.x = the unit (its entry in the merge table says whether it
// was cut), blockIdx.y picks 64 of its rows: each wave takes 16 rows, 4 lanes
// per row and a quarter of the head's dims per lane.  Lane k of a wave works out the
// slot of piece k once (64 pieces per round); every lane then walks the
// pieces in batches of 4 with all their loads in flight, keeping a running
// max (each batch rescales the sums at most once), so a unit of up to 4
// pieces takes a single round of loads.
template <int HD>
__global__ void __launch_bounds__(256) attn_stream_merge_kernel(MfmaArgs a) {
  constexpr int kBatch = 4;
  constexpr int kQD = HD / 4;       // dims per lane (4 lanes per row)
  constexpr int kQC = kQD / 8;      // 16-byte chunks per lane
  if (halted(a.status)) return;
  const int units = *reinterpret_cast<const int32_t*>(a.ws_desc);
  const MergeDesc d = a.ws_desc[1 + blockIdx.x];
  if (static_cast<int>(blockIdx.x) >= units || !d.active) return;
  const int wv = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int rows = min(a.G * d.n - d.rt * kTileRows, kTileRows);
  const int r0 = blockIdx.y * 64 + wv * 16;
  if (r0 >= rows) return;
  const int r = min(r0 + (lane >> 2), rows - 1);  // (rows past the unit's compute its last, unstored)
  const int quarter = lane & 3;                    // dims kQD * quarter .. + kQD - 1
  plan::MergeJob job{};
  job.active = true;
  job.sa = d.sa;
  job.sa_first = d.sa_first != 0;
  job.U = d.U;
  job.u.w = d.w;
  job.q.c.t_pre = d.t_pre;
  const plan::Grid gr = plan::make_grid(d.C, a.W);
  const int npieces = plan::owner(gr, plan::tree_item(d.U, d.w, d.t_pre)) - d.sa + 1;
  float acc[kQD];
#pragma unroll
  for (int e = 0; e < kQD; ++e) acc[e] = 0.f;
  float wsum = 0.f;
  float M = -INFINITY;  // running max: acc and wsum are relative to 2^M
  for (int c0 = 0; c0 < npieces; c0 += kWave) {
    const int cnt = min(kWave, npieces - c0);
    const int my_slot = lane < cnt ? plan::merge_piece_slot(job, c0 + lane, gr) : -1;
    for (int k0 = 0; k0 < cnt; k0 += kBatch) {
      f32x2 ml[kBatch];
      u32x4 o[kBatch][kQC];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int slot = k0 + j < cnt ? __builtin_amdgcn_readlane(my_slot, k0 + j) : -1;
        ml[j] = (f32x2){-INFINITY, 0.f};
#pragma unroll
        for (int c = 0; c < kQC; ++c) o[j][c] = (u32x4){0u, 0u, 0u, 0u};
        if (slot >= 0) {
          const int64_t row = static_cast<int64_t>(slot) * kTileRows + r;
          ml[j] = *reinterpret_cast<const f32x2*>(a.ws_ml + row * 2);
          const u32x4* src = reinterpret_cast<const u32x4*>(a.ws_o + row * kD + quarter * kQD);
#pragma unroll
          for (int c = 0; c < kQC; ++c) o[j][c] = src[c];
        }
      }
      // the batch's pieces join the running sums (one rescale per batch)
      float Mb = M;
#pragma unroll
      for (int j = 0; j < kBatch; ++j) Mb = fmaxf(Mb, ml[j].x);
      if (Mb > M) {
        const float alpha = M == -INFINITY ? 0.f : exp2_fast(M - Mb);
        wsum *= alpha;
#pragma unroll
        for (int e = 0; e < kQD; ++e) acc[e] *= alpha;
        M = Mb;
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const float w = ml[j].y > 0.f ? exp2_fast(ml[j].x - M) * ml[j].y : 0.f;
        wsum += w;
#pragma unroll
        for (int c = 0; c < kQC; ++c)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[8 * c + 2 * e] += w * bf16_to_f32(static_cast<uint16_t>(o[j][c][e] & 0xFFFFu));
            acc[8 * c + 2 * e + 1] += w * bf16_to_f32(static_cast<uint16_t>(o[j][c][e] >> 16));
          }
      }
    }
  }
  if (r0 + (lane >> 2) >= rows) return;
  const float inv = 1.f / wsum;
  const int row = d.rt * kTileRows + r;  // stacked row = node * G + head in group
  const int node = row / a.G;
  const int hq = d.g * a.G + row % a.G;
  u32x4* dst = reinterpret_cast<u32x4*>(
      a.out + ((static_cast<int64_t>(d.b) * a.Nmax + node) * a.Hq + hq) * HD + quarter * kQD);
#pragma unroll
  for (int c = 0; c < kQC; ++c) {
    u32x4 v;
    v.x = pack_bf16x2(acc[8 * c + 0] * inv, acc[8 * c + 1] * inv);
    v.y = pack_bf16x2(acc[8 * c + 2] * inv, acc[8 * c + 3] * inv);
    v.z = pack_bf16x2(acc[8 * c + 4] * inv, acc[8 * c + 5] * inv);
    v.w = pack_bf16x2(acc[8 * c + 6] * inv, acc[8 * c + 7] * inv);
    dst[c] = v;
  }
}

}  // namespace

namespace {

constexpr int kMinTilesPerWg = 2;   // a share shorter than this is mostly fixed cost
constexpr int kMaxGrid = 1024;      // workgroups of the attention grid at most

// Stacked-row tiles and key tiles of the longest unit the launch allows.
int64_t max_unit_tiles(const AttnShape& s) {
  return (s.max_prefix + kKT - 1) / kKT + (s.Nmax + kKT - 1) / kKT;
}
int64_t max_units(const AttnShape& s) {
  const int64_t rows = static_cast<int64_t>(s.Hq / s.Hkv) * s.Nmax;
  return static_cast<int64_t>(s.B) * s.Hkv * ((rows + kTileRows - 1) / kTileRows);
}

// Whether every workgroup's share of a grid of W fits the paged block table
// staged in LDS: a share is at most one unit's keys and, on the axis, at most
// (C / W) / 2 + 1 key tiles (the smallest tile weight is 2), plus the tree.
bool share_fits(const AttnShape& s, int W) {
  if (s.max_blocks <= 0) return true;  // contiguous cache: no table
  const int64_t unit_rows = static_cast<int64_t>(s.max_prefix) + s.Nmax;
  const int64_t axis_tiles =
      max_units(s) *
      plan::unit_extent(static_cast<int>((s.max_prefix + kKT - 1) / kKT), (s.Nmax + kKT - 1) / kKT) *
      plan::tile_weight(8);
  const int64_t share_rows =
      std::min(unit_rows, (axis_tiles / W / 2 + 2) * kKT + static_cast<int64_t>(s.Nmax));
  return share_rows / s.kv_rows + 2 <= kMaxSplitBlocks;
}

// Stream plan grid: W workgroups, a power of two of at least 8 (one eighth of
// the axis per XCD; the partition's arithmetic is then shifts),
// at most one resident round (one workgroup per compute unit), each with at
// least kMinTilesPerWg key tiles of the largest call the shape allows.  It
// does not depend on the cache layout, so neither does the workspace.
int choose_grid(const AttnShape& s, int num_cus) {
  const int64_t tiles = max_units(s) * max_unit_tiles(s);
  const int64_t want = std::min<int64_t>(std::min(num_cus, kMaxGrid), tiles / kMinTilesPerWg);
  int W = 8;
  while (2 * W <= want) W *= 2;
  return W;
}

constexpr size_t kSlotBytes = static_cast<size_t>(kTileRows) * (kD * sizeof(uint16_t) + 2 * sizeof(float));
constexpr size_t kDescBytes = 64;  // sizeof(MergeDesc)

}  // namespace

// Single sequences take the split plan (every unit has the same length, and
// the plan's cost model picks the split length and whether the tree keys get
// a split of their own); batches take the stream plan, which balances units
// of different lengths, unless a paged layout's blocks are so small that a
// workgroup's share could span more block ids than the LDS table holds (the
// split plan shortens its splits for those).
bool use_stream(const AttnShape& s) { return s.B > 1 && share_fits(s, choose_grid(s, 256)); }

// Longest split (in keys, a multiple of the key tile) whose paged block ids
// fit the LDS table: the last split's rows (its prefix keys plus up to Nmax
// tree keys) span at most (keys + Nmax) / kv_rows + 2 blocks.  A contiguous
// cache has no such bound.
int64_t split_key_cap(const AttnShape& s) {
  if (s.max_blocks <= 0) return int64_t{1} << 40;
  const int64_t cap = static_cast<int64_t>(kMaxSplitBlocks - 2) * s.kv_rows - s.Nmax;
  return cap / kKT * kKT;
}

// The smallest cap over every cache layout (paged with 1-row blocks); the
// supported range and the workspace size use it, so that neither depends on
// the layout of the call.
int64_t worst_split_key_cap(const AttnShape& s) {
  AttnShape w = s;
  w.kv_rows = 1;
  w.max_blocks = 1;
  return split_key_cap(w);
}

static double plan_cost(int64_t P, int n, int64_t sk, bool alone, int64_t units, int64_t target) {
  constexpr double kFixedTiles = 3.0, kMaskTiles = 0.5, kMergeTiles = 2.5;
  const int64_t tps = sk / kKT;
  const int64_t tree_tiles = (n + kKT - 1) / kKT;
  const int64_t pre = (P + sk - 1) / sk;
  const int S = n_splits_of(static_cast<int>(P), n, static_cast<int>(sk), alone);
  double longest;
  if (pre <= 1) {
    longest = static_cast<double>((P + kKT - 1) / kKT + tree_tiles) + kMaskTiles;
  } else {
    const int64_t last = (P - (pre - 1) * sk + kKT - 1) / kKT;
    const double tree_split =
        static_cast<double>(S > pre ? tree_tiles : last + tree_tiles) + kMaskTiles;
    longest = std::max(static_cast<double>(tps), tree_split);
  }
  const int64_t rounds = (units * S + target - 1) / target;
  return static_cast<double>(rounds) * (longest + kFixedTiles) +
         (S > 1 ? kMergeTiles + S / 32.0 : 0.0);
}

void plan_split(const AttnShape& s, int num_cus, AttnPlan* p) {
  const int G = s.Hq / s.Hkv;
  const int rows = G * s.Nmax;
  p->row_tiles = (rows + kTileRows - 1) / kTileRows;
  // A (sequence, kv head, row tile) unit is split along the keys into about
  // as many workgroups as keep one resident round of one workgroup per
  // compute unit busy (a second, nearly empty round would double the kernel
  // time).  That gives the shortest split considered; a split holds at least
  // two key tiles, at most the paged table's cap, and the merge kernel's
  // table bounds the number of splits.
  const int64_t units = static_cast<int64_t>(s.B) * s.Hkv * p->row_tiles;
  const int64_t target = num_cus;
  const int64_t want = std::max<int64_t>(1, target / units);
  const int64_t mp = s.max_prefix;
  const int64_t cap = std::min(split_key_cap(s), static_cast<int64_t>(kMaxSplitTiles) * kKT);
  int64_t sk0 = (mp + want - 1) / want;
  sk0 = std::max<int64_t>(sk0, (mp + kMaxMergeSplits - 1) / kMaxMergeSplits);
  sk0 = std::max<int64_t>((sk0 + kKT - 1) / kKT * kKT, 2 * kKT);
  sk0 = std::min(sk0, cap);
  // From there up to the cap, the split length (and whether the tree takes a
  // split of its own) with the lowest estimated time: this balances the
  // split that carries the tree against the others.
  int64_t best_sk = sk0;
  bool best_alone = false;
  double best = plan_cost(mp, s.Nmax, sk0, false, units, target);
  for (int64_t sk = sk0; sk <= cap; sk += kKT) {
    for (int alone = 0; alone < 2; ++alone) {
      if (alone && n_splits_of(static_cast<int>(mp), s.Nmax, static_cast<int>(sk), 1) >
                       kMaxMergeSplits)
        continue;
      const double c = plan_cost(mp, s.Nmax, sk, alone != 0, units, target);
      if (c < best) {
        best = c;
        best_sk = sk;
        best_alone = alone != 0;
      }
    }
  }
  p->split_keys = static_cast<int>(best_sk);
  p->tree_alone = best_alone;
  p->max_splits = n_splits_of(static_cast<int>(mp), s.Nmax, p->split_keys, best_alone);
  // Workspace for partials, sized from the shortest split considered (the
  // most splits any plan of this shape can have), so that a layout with a
  // smaller cap never needs more than the size reported for the worst one.
  // None when no sequence can have more than one split.
  const int64_t pre0 = (mp + sk0 - 1) / sk0;
  const int64_t bound = pre0 <= 1 ? 1 : std::min<int64_t>(pre0 + 1, kMaxMergeSplits);
  const int64_t Mpad = static_cast<int64_t>(p->row_tiles) * kTileRows;
  const int64_t slots = static_cast<int64_t>(s.B) * s.Hkv * bound * Mpad;
  p->workspace_bytes =
      bound > 1 ? static_cast<size_t>(slots) * (kD * sizeof(uint16_t) + 2 * sizeof(float)) : 0;
  p->mfma = true;
  p->stream = false;
  p->grid = s.B * s.Hkv * p->row_tiles * p->max_splits;
}

// The split plan needs splits of at least two key tiles whose block ids fit
// the LDS table even with one-row blocks, and at most kMaxMergeSplits of them.
bool mfma_supported(const AttnShape& s) {
  if (s.dtype != LTD_DTYPE_BF16 || (s.d != 128 && s.d != 64)) return false;
  if (use_stream(s)) return true;
  const int64_t cap = worst_split_key_cap(s);
  return cap >= 2 * kKT && s.max_prefix <= cap * kMaxMergeSplits;
}

int attention_grid(const AttnPlan& p) { return p.mfma ? p.grid : 0; }

// Stream plan: two partial slots per workgroup and the merge table (a 64-byte
// header and one entry per unit the call can have).
void plan_stream(const AttnShape& s, int num_cus, AttnPlan* p) {
  p->mfma = true;
  p->stream = true;
  p->grid = choose_grid(s, num_cus);
  p->workspace_bytes = 2 * static_cast<size_t>(p->grid) * kSlotBytes + (1 + max_units(s)) * kDescBytes;
}

void plan_mfma(const AttnShape& s, int num_cus, AttnPlan* p) {
  if (use_stream(s))
    plan_stream(s, num_cus, p);
  else
    plan_split(s, num_cus, p);
}

hipError_t launch_attn_mfma(const AttnShape& s, const AttnPlan& p, const void* q,
                            const void* k_cache, const void* v_cache, const int32_t* block_table,
                            const int32_t* prefix_len, const int32_t* parents,
                            const int32_t* n_nodes, void* out, float scale, void* workspace,
                            const int32_t* status, hipStream_t stream) {
  MfmaArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_cache);
  a.v = static_cast<const uint16_t*>(v_cache);
  a.block_table = block_table;
  a.prefix_len = prefix_len;
  a.parents = parents;
  a.n_nodes = n_nodes;
  a.out = static_cast<uint16_t*>(out);
  a.status = status;
  a.B = s.B;
  a.Nmax = s.Nmax;
  a.Hq = s.Hq;
  a.Hkv = s.Hkv;
  a.G = s.Hq / s.Hkv;
  a.kv_rows = s.kv_rows;
  a.kv_shift = -1;
  for (int k = 0; k < 31; ++k)
    if ((1 << k) == s.kv_rows) a.kv_shift = k;
  a.max_blocks = s.max_blocks;
  a.max_prefix = s.max_prefix;
  a.scale_log2 = scale * kLog2e;
  a.lazy_gap = kLazyMax / a.scale_log2;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  a.ws_o = static_cast<uint16_t*>(workspace);
  if (!p.stream) {
    a.split_keys = p.split_keys;
    a.max_splits = p.max_splits;
    a.tree_alone = p.tree_alone ? 1 : 0;
    a.row_tiles = p.row_tiles;
    const size_t slots = static_cast<size_t>(s.B) * s.Hkv * p.max_splits * p.row_tiles * kTileRows;
    a.ws_ml = reinterpret_cast<float*>(ws + slots * kD * 2);
    const dim3 grid(s.B * s.Hkv, p.row_tiles, p.max_splits);
    const bool paged = a.block_table != nullptr;
    if (s.d == 64 && paged)
      hipLaunchKernelGGL((attn_split_kernel<64, true>), grid, dim3(kThreads), 0, stream, a);
    else if (s.d == 64)
      hipLaunchKernelGGL((attn_split_kernel<64, false>), grid, dim3(kThreads), 0, stream, a);
    else if (paged)
      hipLaunchKernelGGL((attn_split_kernel<128, true>), grid, dim3(kThreads), 0, stream, a);
    else
      hipLaunchKernelGGL((attn_split_kernel<128, false>), grid, dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.max_splits == 1) return e;  // one split: the output is final
    // (sequence, kv head) fastest, as for the attention grid: a head's merge
    // runs on the XCD whose workgroups wrote its partials.
    const dim3 mgrid(s.B * s.Hkv, static_cast<unsigned>((p.row_tiles * kTileRows + 3) / 4));
    if (s.d == 64)
      hipLaunchKernelGGL(attn_split_merge_kernel<64>, mgrid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(attn_split_merge_kernel<128>, mgrid, dim3(256), 0, stream, a);
    return hipGetLastError();
  }
  const size_t slots = static_cast<size_t>(2) * p.grid * kTileRows;
  a.ws_ml = reinterpret_cast<float*>(ws + slots * kD * 2);
  a.ws_desc = reinterpret_cast<MergeDesc*>(ws + slots * (kD * 2 + 2 * sizeof(float)));
  a.W = p.grid;
  a.max_units = static_cast<int>(max_units(s));
  const bool paged = a.block_table != nullptr;
  if (s.d == 64 && paged)
    hipLaunchKernelGGL((attn_stream_kernel<64, true>), dim3(p.grid), dim3(kThreads), 0, stream, a);
  else if (s.d == 64)
    hipLaunchKernelGGL((attn_stream_kernel<64, false>), dim3(p.grid), dim3(kThreads), 0, stream, a);
  else if (paged)
    hipLaunchKernelGGL((attn_stream_kernel<128, true>), dim3(p.grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((attn_stream_kernel<128, false>), dim3(p.grid), dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // One merge workgroup column per possible unit, 64 rows per workgroup.
  if (s.d == 64)
    hipLaunchKernelGGL(attn_stream_merge_kernel<64>, dim3(a.max_units, kTileRows / 64), dim3(256),
                       0, stream, a);
  else
    hipLaunchKernelGGL(attn_stream_merge_kernel<128>, dim3(a.max_units, kTileRows / 64), dim3(256),
                       0, stream, a);
  return hipGetLastError();
}

}  // namespace ltd
