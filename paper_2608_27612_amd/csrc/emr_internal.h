// Internal data layout shared by the host runtime and the gfx950 kernels.
//
// A packed population is one device array of 32-bit words ("blob") plus one ProgDesc per
// (genome, query direction). For a direction, the CPPN inputs split into two that vary with the
// grid position (the position's x and y) and three that do not (the source's x and y, and the
// constant 1). Every live node is then either position-dependent ("varying") or a per-(genome,
// source) constant ("uniform"):
//   - the varying program is what one GPU lane interprets per position;
//   - the uniform program is evaluated once per (genome, source) by the bind kernel, which folds
//     every uniform contribution into a per-step bias (and, when the output itself is uniform,
//     produces the output constant).
#pragma once
#include <stdint.h>

#if defined(__HIPCC__) || defined(__HIP__)
#define EMR_HD __host__ __device__
#else
#define EMR_HD
#endif

namespace emr {

// Kernel window sizes (register slots per source) the kernels are instantiated for.
constexpr int kWindows[] = {4, 8, 16, 32};
constexpr int kMaxWindow = 32;
// Sources evaluated together by one lane (same genome, same direction).
constexpr int kMaxGroup = 4;
// Parts of a launch: one per (sources per walk, register window) variant present (9 at most),
// each split at most 5 ways by chunk size (16 .. 1 tiles) when the launch has a schedule.
constexpr int kMaxBuckets = 9;
constexpr int kMaxParts = 5 * kMaxBuckets;
// Register budget of the value windows: S sources x P positions x W slots <= 128 VGPRs per lane.
constexpr int kWindowRegs = 128;
// Positions per wave iteration and iterations per tile.
constexpr int kWave = 64;
constexpr int kTileIters = 4;
constexpr int kTile = kWave * kTileIters;  // 256 = 4^4 positions
constexpr int kFirstAlignedLevel = 4;     // first level whose size is a multiple of kTile

// ---------------------------------------------------------------- varying program
// At blob[var_off] (a multiple of 16 words): n_rec records of 16 words, in topological order of the
// position-dependent nodes. A node with e node-to-node edges takes max(1, ceil(e / 11)) records:
//   word 0: meta   bits 0..3  tail: 0 = more records of this node follow;
//                             1 + a = the node ends with activation a and its value is stored to
//                                     the dst slot (a in 0..5, EMR_ACT_*);
//                             7 + a = the node is the output: activation a, value kept
//                  bit 4      first record of a node: the accumulator starts at bias + ax x + ay y
//                  bit 5      (first record) the node's value does not depend on the source: no
//                             path reaches it from the source's coordinates, so its bias rows
//                             are equal for every source and it takes the same value for every
//                             source at a position (never set for the output node)
//                  bits 8..12 dst slot
//                  bits 16..19 number of edges in this record (0..11)
//   word 1: float bits of the summed weights of the node's edges from the position's x (first
//           record only, else 0)
//   word 2: the same for y
//   word 3: source slots of record positions 0..5, 5 bits each (position k at bit 5k)
//   word 4: source slots of positions 6..10, 5 bits each
//   words 5..15: float bits of the edge weights of positions 0..10
// A record with n edges uses positions 0..n-1 and they are accumulated from position n-1 down
// to 0, so the packer stores the node's edges in reverse.
// The node's bias is not stored here: it is the per-source folded bias from the bind kernel.
constexpr uint32_t kRecWords = 16;
constexpr uint32_t kRecEdges = 11;
constexpr uint32_t kRecTailMask = 15u;
constexpr uint32_t kRecTailStore = 1u;   // + activation
constexpr uint32_t kRecTailOutput = 7u;  // + activation
constexpr uint32_t kRecFirst = 1u << 4;
constexpr uint32_t kRecShared = 1u << 5;
constexpr uint32_t kRecDstShift = 8;
constexpr uint32_t kRecEdgeShift = 16;
constexpr uint32_t kSlotBits = 5;

// ---------------------------------------------------------------- uniform program
// At blob[uni_off]:
//   header 4 words: n_unodes, out_u (index into U of the output, or kNone when it varies),
//                   n_steps (of the varying program), 0
//   n_unodes records of 4 words: act, n_edges, edge_off, bias bits      -> U[5 + k]
//   n_steps  records of 4 words: n_fold, fold_off, bias bits, r         -> folded bias of varying
//            node i, for its first program record r
//   edges: {u_src, w bits}; U[0..4] hold the five input roles (x1, y1, x2, y2, 1).
// edge_off and fold_off count words from uni_off, so a genome's words can be moved as a block.
constexpr uint32_t kNone = 0xFFFFFFFFu;

struct ProgDesc {
  uint32_t var_off;   // word offset of the record stream
  uint32_t n_rec;     // records
  uint32_t n_steps;   // varying nodes
  uint32_t uni_off;   // word offset of the uniform program
  uint32_t flags;     // bit 0: output varies with position; bits 8..15: register window needed
  uint32_t uni_end;   // word offset one past the uniform program and its edges
  uint32_t pad[2];
};

// One unit of kernel work: up to kMaxGroup sources of one genome sharing a direction.
// Its bias rows (4 floats each, one per source slot) start at bias_off, a multiple of 4: row 0 holds
// the output constants (used when the output is uniform), row 1 + r the folded bias of the node
// whose first program record is r (rows of other records are unused). The group owns n_rec + 2
// rows: the walk reads row 1 + r with record r, for r up to n_rec (the prefetch past the end).
struct Group {
  uint32_t var_off;
  uint32_t n_rec;
  uint32_t n_steps;
  uint32_t flags;      // copied from ProgDesc
  uint32_t bias_off;   // float offset into the bias table
  uint32_t code_off;   // compiled tier: byte offset of the group's program in the code area
  uint32_t pad[2];
  uint32_t pair[kMaxGroup];  // global pair ids of the sources (unused entries repeat the last)
};

// Device error bits (word kFlagErr of a call's flag slot).
constexpr uint32_t kErrTable = 2u;     // a table entry pointed outside its table (entry skipped)
constexpr uint32_t kMaxSteps = 256;
constexpr uint32_t kMaxRecords = kMaxSteps + 4096 / kRecEdges + 1;

// One (genome, direction, source) evaluated by the bind kernel.
struct Member {
  uint32_t desc;       // ProgDesc index = 2 * genome + dir
  uint32_t source;     // source index
  uint32_t bias_base;  // its group's bias_off + its slot in the group
  uint32_t bias_rows;  // rows owned by its group (n_rec + 2)
};

// Positions per lane per program walk. A lane holds whole sibling quads: the four children of
// one parent (P = 4) or of a parent in each of P / 4 consecutive tiles (P = 8, 16), so a cell's
// variance is computed inside the lane. S sources of one genome share the walk (M = S P
// instances); a (S, P, W) combination fits when the M value windows fit the register budget and
// the estimated VGPR total (accumulators, windows, positions, per-source variances and ~16
// others) leaves room for 3 waves per SIMD. The record step's scalar work is shared by the M
// instances, so the largest P that fits is taken.
EMR_HD constexpr bool fits_lane(int S, int P, int W) {
  return S * P * W <= kWindowRegs && 16 + S * P + S * P * W + 2 * P + 2 * S <= 168;
}
EMR_HD constexpr int positions_per_lane(int S, int W) {
  return fits_lane(S, 16, W) ? 16 : fits_lane(S, 8, W) ? 8 : 4;
}
// Sources per walk for window W: the most (up to 3) that fit with P = 4.
EMR_HD constexpr int max_group(int W) {
  return fits_lane(3, 4, W) ? 3 : fits_lane(2, 4, W) ? 2 : 1;
}

// Level helpers shared by host and device.
EMR_HD inline int64_t level_offset(int level) {  // first grid index of level >= 1
  return ((int64_t(1) << (2 * level)) - 4) / 3;
}
EMR_HD inline int64_t n_positions(int depth) { return level_offset(depth + 1); }
EMR_HD inline int64_t n_parents(int depth) {
  return depth <= 0 ? 0 : ((int64_t(1) << (2 * depth)) - 1) / 3;
}
// Tiles per (pair, depth): one "head" tile for levels 1..kFirstAlignedLevel-1 (or all levels when
// the depth is smaller), then kTile-sized tiles that never straddle a level.
EMR_HD inline int64_t tiles_per_pair(int depth) {
  if (depth < kFirstAlignedLevel) return 1;
  return 1 + (n_positions(depth) - level_offset(kFirstAlignedLevel)) / kTile;
}

// First parent index of a pair's tile T (T = tiles_per_pair(depth) gives n_parents(depth)): tile 0
// holds the parents of levels 0..2 (or all of them when the depth is smaller), every other tile 64.
EMR_HD inline int64_t tile_parent_offset(int64_t T, int depth) {
  if (T == 0) return 0;
  if (depth < kFirstAlignedLevel) return n_parents(depth);
  return level_offset(kFirstAlignedLevel) / 4 + (T - 1) * (kTile / 4);
}


// ---------------------------------------------------------------- discover launch scalars
// One launch covers every group of a call, in up to kMaxParts parts: runs of groups with S
// sources per walk and register window W, each with one chunk size (costliest part first). The
// launch's chunks are those of its parts, one after the other.
struct DiscoverPart {
  uint32_t S, W, group0;                     // sources per walk, window; the part's first group
  uint32_t n_chunks, chunks_per_group, chunk_tiles;
};
struct DiscoverScalars {
  int64_t cap, n_pos;  // cap: records the pool holds
  // The launch covers tiles tile_lo .. tile_lo + tiles - 1 of every pair.
  uint32_t tile_lo, tiles;
  uint32_t n_parts, n_chunks;  // chunks of all parts
  DiscoverPart part[kMaxParts];
  int32_t depth;
  float theta16;  // 16 theta
  uint32_t code_bytes;  // compiled tier: size of the code area (0 for the interpreter)
  // Records over more than 2 groups of 64 tiles: bit g % 64 of nz[pair * nz_words + g / 64]
  // marks a group g of the range that kept a cell (k_move visits only those).
  uint64_t* nz;
  uint32_t nz_words;
  uint32_t blob_words, n_pairs;
  uint32_t bias_floats;  // the host keeps the bias table below 2^32 floats
  uint32_t head_parents;  // parents in a pair's tile 0 (levels 1..3, or all levels of a shallower grid)
  // Record mode: the pool's reservation counter, the pool, and the per-pair record totals (each
  // chunk adds its sources' counts; zero when the launch starts).
  uint64_t* pool_ctr;
  uint32_t* pool_parent;
  float* pool_w4;
  uint32_t* pair_total;
  // The workgroups' chunk lists, or NULL for round-robin chunks (chunk c of the launch to
  // workgroup c mod workgroups): workgroup b's waves take the entries sched[b * sched_stride + j],
  // j = 0, 1, ..., up to the first kNoChunk, each naming a chunk as its part << kEntryPartShift |
  // its index in the part. The lists were made for exactly sched_lists workgroups (the launch's
  // grid); sched_stride is a multiple of 64, at most kListLds.
  const uint32_t* sched;
  uint32_t sched_stride, sched_lists;
};
constexpr uint32_t kNoChunk = 0xFFFFFFFFu;
constexpr uint32_t kEntryPartShift = 24;  // a listed part holds fewer than 2^24 chunks
static_assert(kMaxParts < (1 << (32 - kEntryPartShift)) - 1, "part ids of list entries");

// A discover workgroup fills one CU: 3 waves on each of its 4 SIMDs (the kernels' register budget
// allows 3), taking their workgroup's chunks one at a time from a counter in LDS. A SIMD issues
// for its oldest wave first, so waves of one workgroup progress at different speeds; taking chunks
// as they free up keeps every wave busy until the CU's share runs out.
constexpr int kDiscoverWaves = 12;
constexpr int kDiscoverThreads = kDiscoverWaves * kWave;
constexpr uint32_t kListLds = 2048;  // the longest list: a discover workgroup holds it in LDS

// Output modes: raw CPPN outputs; records of kept cells, each walk's reserved in a pool with one
// atomic, each tile's pool offset and count left in its status word and each chunk's count added
// to its pair's total, for k_scan (pair offsets) and k_move (per-pair contiguous lists).
constexpr int kModeRaw = 0, kModeRecords = 1;

// A tile's status word in record mode: its records' pool offset << 8 | their count (<= 64).
constexpr uint32_t kStatusCountBits = 8;

// Call flag words (a library-owned slot of kSlotWords words per call, zero when a call takes it and
// cleared again by the call's last kernel).
constexpr int kFlagErr = 0;      // error bits
constexpr int kFlagMax = 1;      // largest pair count (saturating u32)
constexpr int kFlagPool = 2;     // u64: the pool's reservation counter (words 2, 3)
constexpr int kFlagTotal = 6;    // u64: records found by the call (words 6, 7)
constexpr int kFlagWords = 8;

// ---------------------------------------------------------------- compiled tier
// A walk calls its group's compiled program (machine code written at run time into the code area
// of the template code object) with this register convention, shared by the call site in the
// kernel and the host code generator. For M = S P instances:
//   v[kJitAcc + m]                    accumulator of instance m (the program's outputs)
//   v[jit_window(M, W, m) + k]        slot k of instance m's value window (k < W)
//   v[jit_xr(M, W, j)], v[jit_yr(...)] the x and y of position j (read only). Position
//                                     4 k + c is child c of the lane's parent in tile k, whose
//                                     x depends on c & 1 and y on c >> 1 only: each is held once,
//                                     x at jit_x + 4 k + (c & 1), y at jit_x + P + 4 k + (c & 2)
//                                     (the registers between are not part of the convention)
//   v[jit_x(M, W) + 2 P ...]          jit_temps(S, P, W) bias copies (for S > 1 the last source's
//                                     accumulators hold the partial sums)
//   s[kJitRow .. kJitRow + 15]        bias rows 1 .. kJitRowBlock of the group (the rows of records
//                                     0 .. 3), loaded by the caller once per chunk (in and out:
//                                     a program that needs later rows loads them here, and then
//                                     loads its first rows itself too)
//   s[kJitBp, kJitBp + 1]             the group's bias rows (row 0 outputs of a program without
//                                     records, row 1 + r the biases of the node starting at record r)
//   s[kJitRet, kJitRet + 1]           the return address
// A program touches nothing else: no memory writes, no exec, vcc or m0, no other registers.
constexpr int kJitAcc = 4;
constexpr int kJitRow = 40;
constexpr int kJitRowBlock = 4;  // records whose bias rows are loaded together
constexpr int kJitBp = 56;
constexpr int kJitRet = 58;
constexpr uint32_t kJitTailPad = 1024;  // s_endpgm bytes kept after the last program
EMR_HD constexpr int jit_window(int M, int W, int m) { return ((kJitAcc + M + 1) & ~1) + m * W; }
EMR_HD constexpr int jit_x(int M, int W) { return jit_window(M, W, M); }
EMR_HD constexpr int jit_xr(int M, int W, int j) { return jit_x(M, W) + (j & ~3) + (j & 1); }
EMR_HD constexpr int jit_yr(int M, int W, int P, int j) {
  return jit_x(M, W) + P + (j & ~3) + (j & 2);
}
// Bias copies of a variant: one per source, where they fit below kJitTop (the highest register
// any variant needs); a variant without them adds the biases from their SGPRs.
constexpr int kJitTop = 148;
EMR_HD constexpr int jit_temps(int S, int P, int W) {
  return S == 1 ? 1 : (jit_x(S * P, W) + 2 * P + S <= kJitTop ? S : 0);
}

// Tiles of one chunk at most (a chunk's record counts are held one per lane, 16 per source).
constexpr uint32_t kChunkTilesMax = 16;
// Group marks of the compaction: a range of more than kNzMinGroups groups of 64 tiles has
// nz_words(tiles) words of marks per pair, one bit per group.
constexpr uint32_t kNzMinGroups = 2;
EMR_HD constexpr uint32_t nz_words(uint32_t tiles) { return ((tiles + 63u) / 64u + 63u) / 64u; }
// Rows of zeros after the last tile of the tile geometry table: a walk of TPW <= 4 tiles loads
// the next walk's TPW rows, up to 2 TPW - 1 rows past its first tile, with no bound per load.
constexpr uint32_t kGeoPadRows = 8;

struct DiscoverArgs {
  const uint32_t* geo;     // tile geometry table of the depth (k_tile_geo), geo_rows rows
  uint32_t geo_rows;       // with the kGeoPadRows rows of padding
  const uint32_t* blob;
  const Group* groups;     // the plan's group table (parts index into it)
  const float* bias_tab;
  uint64_t* status;        // [n_pairs * tiles] tile status words of the range
  uint64_t* nz;            // group marks (DiscoverScalars::nz)
  uint32_t* err;           // the call's flag words (kFlag*)
  uint32_t* pool_parent;   // record mode: the pool (cap records)
  float* pool_w4;
  uint32_t* pair_total;    // record mode: per-pair record totals
  float* raw;              // raw-output mode: [pair][N]
  int64_t cap;             // records the pool holds
  int64_t n_pos;           // N(depth)
  // The launch's parts: groups part_group0[k] .. + part_groups[k] - 1, with part_S[k] sources
  // per walk and register window part_W[k], in launch order.
  uint32_t n_parts;
  uint32_t part_S[kMaxParts], part_W[kMaxParts], part_group0[kMaxParts], part_groups[kMaxParts];
  // the part's chunk size in tiles: a power of two from one walk's tiles to kChunkTilesMax, or 0
  // for the launcher's rule
  uint32_t part_chunk[kMaxParts];
  uint32_t tile_lo;        // first tile of the launch (of every pair)
  uint32_t tiles;          // tiles of the launch per pair
  int32_t depth;
  float theta;
  uint32_t blob_words;     // size of the population table
  uint32_t n_pairs;        // pairs of the call (bound for pair ids)
  uint64_t bias_floats;    // size of the bias table
  const uint32_t* sched;   // the workgroups' chunk lists (DiscoverScalars::sched), or NULL
  uint32_t sched_stride, sched_lists;
};

// Arguments of the compaction of one record-mode range: k_scan (the pairs' offsets, one
// workgroup) then k_move (one wave per pair).
struct ScanArgs {
  uint32_t* pair_total;  // [n_pairs] per-pair totals of the range (cleared by k_scan after use)
  int64_t* pair_count;   // [n_pairs] out
  int64_t* pair_offset;  // [n_pairs + 1] out
  uint32_t* flags;       // the call's flag words (kFlag*)
  uint32_t* host;        // non-NULL: the call's pinned flag words (device view); k_scan then
                         // hands the flags over and clears them (the call's last flag writer)
  int64_t* host_counts;  // non-NULL: pinned words (device view) that also get the counts, and at
                         // [n_pairs] the call's error bits (a streamed chunk's check before its
                         // delivery)
  uint32_t n_pairs;
};
struct MoveArgs {
  const uint64_t* status;  // [n_pairs * tiles]
  const uint32_t* pool_parent;
  const float* pool_w4;
  uint32_t* parent;
  float* w4;
  const int64_t* pair_count;
  const int64_t* pair_offset;
  uint64_t* nz;
  const uint8_t* skip;   // per pair: 1 = its groups were left out of the launch (no records)
  int64_t cap;
  uint32_t tiles, n_pairs, nz_words;
};

// ---------------------------------------------------------------- after discovery (phase2.hip)
// The records of a checked discover call (CSR) and each pair's genome, direction and source.
struct RecordsIn {
  const uint32_t* parent;
  const float* w4;
  const int64_t* count;   // [n_pairs]
  const int64_t* offset;  // [n_pairs + 1]
  int64_t cap;            // records the buffers hold (entries beyond it are not read)
  const uint32_t* pair_info;  // [2 n_pairs]: genome << 1 | dir, source index
  const float* src_xy;        // [2 n_sources]
  uint32_t n_pairs;
  int32_t depth;
};

struct HiddenArgs {
  RecordsIn rec;
  uint32_t* fresh;         // [n_genomes * words] cells found by this call (cleared before it)
  uint32_t* known;         // [n_genomes * words] or NULL
  uint32_t* totals;        // [n_genomes] new cells per genome
  const int64_t* offsets;  // [n_genomes + 1] from k_scan
  uint32_t* out_src;       // [3 cap] emr_source records (x, y bits, dir)
  uint32_t* out_cell;      // [cap] or NULL
  int64_t cap;
  int64_t words;
  uint32_t n_genomes;
};

struct ExpressArgs {
  RecordsIn rec;
  uint32_t type_mask;
  float w_min;
  uint32_t* totals;           // [n_pairs]
  const int64_t* out_offset;  // [n_pairs + 1] from k_scan
  uint32_t* out_cell;
  float* out_w;
  int64_t cap;
};

struct ChainArgs {
  RecordsIn rec;
  uint32_t* member;           // [n_pairs * qwords] bit P: parent P is a record of the pair
  int64_t qwords;
  uint32_t* totals;           // [n_pairs]
  const int64_t* out_offset;  // [n_pairs + 1] from k_scan
  uint32_t* out_parent;
  float* out_w4;
  int64_t cap;
};

struct BindArgs {
  const uint32_t* blob;
  const ProgDesc* desc;
  const Member* members;
  const float* src_xy;     // [n_sources * 2]
  float* bias_tab;
  uint32_t* err;
  uint32_t n_members;
  uint32_t n_desc;         // entries of desc
  uint32_t n_sources;
  uint32_t blob_words;
  uint64_t bias_floats;
};

}  // namespace emr
