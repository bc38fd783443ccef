// gfx950 kernels for eager multi-resolution substrate discovery.
//
//   k_grid      writes the cell centres of every queried position (Section 3.1, Eq. 1).
//   k_fill      clears the look-back status words and counters of a workspace.
//   k_bind      evaluates the position-independent part of each (genome, source) CPPN once and
//               folds it into per-step biases (one wave per pair).
//   k_discover  the hot path: one lane per parent cell; each lane interprets the varying CPPN
//               program for S sources of one genome at the cell's four children at once
//               (Section 3.1, the batched query W), reduces the four siblings to their variance
//               in registers, applies var > theta (Section 3.2, Eq. 2), and places the kept cells
//               with a wave ballot at per-tile slots (compacted by k_compact) or through a
//               per-pair decoupled look-back scan, so every pair's records land in ascending
//               parent order with no atomics on the output.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/emr.h"
#include "emr_internal.h"

namespace emr {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x32 __attribute__((ext_vector_type(32)));

// ------------------------------------------------------------------------ activations
// The bind kernel's activations (uniform nodes): hardware v_exp_f32 (2^x), v_rcp_f32 and
// v_sin_f32 (sin of 2*pi*x) with the range reductions their inputs need. Errors stay near 1e-7
// absolute for |z| up to a few hundred. (Varying nodes are activated inside the record step.)
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kInv2Pi = 0.159154943091895336f;
constexpr float k2PiHi = 6.28318548202514648f;      // nearest float to 2*pi
constexpr float k2PiLo = -1.74845553146951720e-07f; // 2*pi - k2PiHi

__device__ __forceinline__ float act_sigmoid(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-kLog2e * z));
}
__device__ __forceinline__ float act_tanh(float z) {
  // tanh z = 2 / (1 + e^{-2z}) - 1; absolute error ~2 ulp(1) near 0, exact +-1 in the tails.
  return __builtin_fmaf(2.0f, __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-2.0f * kLog2e * z)),
                        -1.0f);
}
__device__ __forceinline__ float act_gauss(float z) {
  return __builtin_amdgcn_exp2f(-kLog2e * (z * z));
}
__device__ __forceinline__ float act_sine(float z) {
  // Cody-Waite reduction by 2*pi (two-part constant), then the hardware sine in revolutions.
  float k = __builtin_rintf(z * kInv2Pi);
  float r = __builtin_fmaf(-k, k2PiHi, z);
  r = __builtin_fmaf(-k, k2PiLo, r);
  return __builtin_amdgcn_sinf(r * kInv2Pi);
}
__device__ __forceinline__ float act_apply(uint32_t a, float z) {
  switch (a) {
    case EMR_ACT_SIGMOID: return act_sigmoid(z);
    case EMR_ACT_TANH: return act_tanh(z);
    case EMR_ACT_GAUSS: return act_gauss(z);
    case EMR_ACT_SINE: return act_sine(z);
    case EMR_ACT_ABS: return __builtin_fabsf(z);
    default: return z;
  }
}

// ------------------------------------------------------------------------ position decode
__device__ __forceinline__ uint32_t compact_even(uint32_t x) {  // bits 0,2,4,.. -> 0,1,2,..
  x &= 0x55555555u;
  x = (x | (x >> 1)) & 0x33333333u;
  x = (x | (x >> 2)) & 0x0F0F0F0Fu;
  x = (x | (x >> 4)) & 0x00FF00FFu;
  x = (x | (x >> 8)) & 0x0000FFFFu;
  return x;
}
__device__ __forceinline__ float pow2_neg(int l) {  // 2^-l, exact
  return __int_as_float((127 - l) << 23);
}
// Level of grid index p: 3(p+1)+1 lies in [4^l, 4^(l+1)).
__device__ __forceinline__ int level_of(uint32_t p) {
  return (31 - __builtin_clz(3u * p + 4u)) >> 1;
}

// ------------------------------------------------------------------------ wave helpers
__device__ __forceinline__ uint32_t lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}
// The lane id read where it is used: values derived from it on rarely taken paths are then
// computed there instead of being hoisted to the kernel start and held in registers throughout.
__device__ __forceinline__ uint32_t lane_id_here() {
  uint32_t l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n v_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ uint32_t popc64(uint64_t m) { return __builtin_popcountll(m); }
__device__ __forceinline__ uint32_t mbcnt64(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ------------------------------------------------------------------------ register windows
// Walker<S, P, W>: the M = S * P instances' accumulators and varying values in pinned VGPRs, and
// step(), which runs one program record for all of them in a single asm statement (generated,
// see gen_regwin.py). s_set_gpr_idx_on also writes M0; M0 is reserved by the compiler and this
// kernel has no other use of it (no LDS DMA, no message or GWS instructions), which the ISA check
// in the tests enforces.
#include "regwin_gen.h"

// Raises *p to at least v. The plain read first keeps the many waves whose value is not larger
// from all queueing on the one word.
__device__ __forceinline__ void raise_max(uint32_t* p, uint32_t v) {
  if (v > __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) atomicMax(p, v);
}

// ------------------------------------------------------------------------ look-back scan
// Tile status words of one pair, indexed by tile. A tile publishes its local count as an
// aggregate, sums predecessors (64 per probe, one per lane) back to the nearest inclusive
// prefix, then publishes its own inclusive prefix. The kernel is launched cooperatively (every
// wave is resident) and each wave walks its tiles in increasing order, so the lowest unfinished
// tile always belongs to a running wave whose earlier tiles are done: waits always end. Each wait
// is also bounded and, if the bound were ever hit, raises an error flag instead of spinning on.
constexpr uint32_t kSpinLimit = 1u << 22;

__device__ __forceinline__ void status_store(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t status_load(uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ uint64_t lookback(uint64_t* row, uint32_t tile, uint64_t count, uint32_t* err) {
  const uint32_t lane = lane_id();
  if (tile == 0) {
    if (lane == 0) status_store(&row[0], kStatusInclusive | count);
    return 0;
  }
  if (lane == 0) status_store(&row[tile], kStatusAggregate | count);
  uint64_t prefix = 0;
  int64_t j = (int64_t)tile - 1;
  uint32_t spins = 0;
  for (;;) {
    const int64_t idx = j - (int64_t)lane;
    const uint64_t s = idx >= 0 ? status_load(&row[idx]) : kStatusInclusive;
    const uint64_t flag = s >> 62;
    const uint64_t incl = ballot(flag == 2);
    const uint64_t empty = ballot(flag == 0);
    const uint32_t first = incl ? (uint32_t)__builtin_ctzll(incl) : 64u;
    const uint64_t upto = first >= 63 ? ~0ull : ((2ull << first) - 1ull);
    if (empty & upto) {
      if (++spins > kSpinLimit) {
        if (lane == 0) atomicOr(err, kErrLookback);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      continue;
    }
    const uint64_t mine = ((upto >> lane) & 1ull) ? (s & kStatusValueMask) : 0ull;
    prefix += wave_sum_u64(mine);
    if (first < 64) break;
    j -= 64;
  }
  if (lane == 0) status_store(&row[tile], kStatusInclusive | (prefix + count));
  return prefix;
}

// ------------------------------------------------------------------------ discover kernel
// Pointers are passed as separate restrict-qualified parameters so the compiler can prove that
// the program, group and bias tables are never written by the kernel and read them with scalar
// loads through the scalar cache.
//
// One launch covers every group of a call, in up to kMaxParts parts: the groups with S sources
// per walk and register window W, one part per (S, W) present (costliest part first). The
// launch's chunks are those of its parts, one after the other.
struct DiscoverPart {
  uint32_t S, W, group0;                     // sources per walk, window; the part's first group
  uint32_t n_chunks, chunks_per_group, chunk_tiles;
};
struct DiscoverScalars {
  int64_t cap, n_pos;
  // The launch covers tiles tile_lo .. tile_lo + tiles - 1 of every pair; record slots of a pair
  // region count from parent_lo, the first parent index of tile tile_lo.
  uint32_t tile_lo, parent_lo, tiles;
  uint32_t n_parts, n_chunks;  // chunks of all parts
  DiscoverPart part[kMaxParts];
  int32_t depth;
  float theta16;  // 16 theta
  uint32_t blob_words, n_pairs;
  uint32_t bias_floats;  // the host keeps the bias table below 2^32 floats
  uint32_t head_parents;  // parents in a pair's tile 0 (levels 1..3, or all levels of a shallower grid)
};

// Output modes: raw CPPN outputs; records at fixed per-tile slots (pair_capacity >= Q(D)),
// compacted afterwards by k_compact; records placed directly through the look-back scan (any
// capacity).
constexpr int kModeRaw = 0, kModePadded = 1, kModeLookback = 2;

// Read-only tables are read through the constant address space: the kernel never writes them
// during a launch, and uniform loads from it are always scalar loads (s_load through the scalar
// cache), whatever the kernel stores elsewhere.
typedef __attribute__((address_space(4))) const uint32_t cu32;
typedef __attribute__((address_space(4))) const float cf32;

// One Group record (12 words) through the constant address space.
__device__ __forceinline__ Group load_group(cu32* p) {
  Group g;
  g.var_off = p[0];
  g.n_rec = p[1];
  g.n_steps = p[2];
  g.flags = p[3];
  g.bias_off = p[4];
  g.pad[0] = g.pad[1] = g.pad[2] = 0;
#pragma unroll
  for (int k = 0; k < kMaxGroup; ++k) g.pair[k] = p[8 + k];
  return g;
}
static_assert(sizeof(Group) == 12 * sizeof(uint32_t), "Group layout");


// ------------------------------------------------------------------------ compaction
// First parent index of a pair's tile T: tile 0 holds the parents of levels 1..3, every other tile
// 64 parents.
__device__ __forceinline__ uint32_t tile_parent_offset(uint32_t T) {
  return T == 0 ? 0u : (uint32_t)(level_offset(kFirstAlignedLevel) / 4) + (T - 1) * (kTile / 4);
}

// Compaction of one pair by one wave, once every tile of the range has left its records at the
// tile's own slots and its count in counts[pair * tiles + t]: scans the counts, 64 tiles at a time,
// and moves the records down to their final, contiguous place, then writes the pair's count and
// returns it.
__device__ uint32_t compact_pair(const uint64_t* __restrict__ counts, uint32_t* __restrict__ parent,
                                 float* __restrict__ w4, int64_t* __restrict__ pair_count,
                                 int64_t cap, uint32_t tile_lo, uint32_t tiles, uint32_t pair,
                                 uint32_t head_slots, uint32_t lane) {
  const uint32_t parent_lo = tile_parent_offset(tile_lo);
  const uint64_t* row = counts + (int64_t)pair * tiles;
  const int64_t region = (int64_t)pair * cap;
  uint32_t running = 0;
  for (uint32_t t0 = 0; t0 < tiles; t0 += kWave) {
    // a tile holds at most its own slot count (64, or the head tile's parents)
    const uint32_t t_lane = t0 + lane;
    const uint32_t slots = tile_lo + t_lane == 0 ? head_slots : (uint32_t)(kTile / 4);
    const uint32_t c = t_lane < tiles ? min((uint32_t)row[t_lane], slots) : 0u;
    // inclusive scan over the wave, bit-sliced: c < 128, so the counts of the lanes below are
    // the sum over bits b of 2^b times the number of lanes below with bit b set (mbcnt)
    uint32_t incl = c;
#pragma unroll
    for (int b = 0; b < 7; ++b) incl += mbcnt64(ballot((c >> b) & 1u)) << b;
    // These tiles' records in batches of 64, lane l moving the batch's l-th record: its tile is
    // the one (among the tiles with records) whose scan range holds it. A batch's loads all come
    // before its stores, and no record moves up, so a batch never overwrites a later batch's
    // records before they are read.
    const uint32_t total = __builtin_amdgcn_readlane(incl, kWave - 1);
    const uint64_t nz = ballot(c != 0u);
    for (uint32_t b = 0; b < total; b += kWave) {
      const uint32_t q = b + lane;  // the record's rank among these tiles' records
      uint32_t src = running + q;
      for (uint64_t m = nz; m != 0ull; m &= m - 1ull) {
        const uint32_t i = (uint32_t)__builtin_ctzll(m);
        const uint32_t hi = __builtin_amdgcn_readlane(incl, i);
        const uint32_t lo = hi - __builtin_amdgcn_readlane(c, i);
        if (q >= lo && q < hi) src = tile_parent_offset(tile_lo + t0 + i) - parent_lo + (q - lo);
      }
      const uint32_t dst = running + q;
      if (q < total && src != dst) {
        const uint32_t pv = parent[region + src];
        const float4 wv = reinterpret_cast<const float4*>(w4)[region + src];
        parent[region + dst] = pv;
        reinterpret_cast<float4*>(w4)[region + dst] = wv;
      }
    }
    running += total;
  }
  if (lane == 0) pair_count[pair] = running;
  return running;
}

// Each wave takes pairs pair = wave, wave + n_waves, ...: compacts them once every discover launch
// of the range has finished, and the workgroup's largest count is raised into *max_count with one
// atomic.
constexpr int kCompactWaves = 4;

__global__ void __launch_bounds__(kCompactWaves * kWave)
    k_compact(const uint64_t* __restrict__ counts, uint32_t* __restrict__ parent,
              float* __restrict__ w4, int64_t* __restrict__ pair_count,
              uint32_t* __restrict__ max_count, int64_t cap, uint32_t tile_lo, uint32_t tiles,
              uint32_t n_pairs, uint32_t head_slots) {
  __shared__ uint32_t wave_max[kCompactWaves];
  const uint32_t lane = lane_id();
  const uint32_t wv = threadIdx.x / kWave;
  const uint32_t n_waves = gridDim.x * kCompactWaves;
  uint32_t my_max = 0;
  for (uint32_t pair = __builtin_amdgcn_readfirstlane(blockIdx.x * kCompactWaves + wv);
       pair < n_pairs; pair += n_waves) {
    my_max = max(my_max, compact_pair(counts, parent, w4, pair_count, cap, tile_lo, tiles, pair,
                                      head_slots, lane));
  }
  if (lane == 0) wave_max[wv] = my_max;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t m = 0;
    for (int k = 0; k < kCompactWaves; ++k) m = max(m, wave_max[k]);
    raise_max(max_count, m);
  }
}

// Where a level-aligned tile (a pair's tile T >= 1, 256 positions of one level) lies: its level
// and the column and row of its 16 x 16 block of cells within the level, whose Morton index is z.
// Consecutive tiles are stepped with a Morton increment instead of a fresh bit de-interleave.
struct TileGeo {
  uint32_t T, lvl, z, cx, cy;
};
__device__ __forceinline__ void tile_geo_set(TileGeo& g, uint32_t T) {
  const uint32_t p0 = (uint32_t)(level_offset(kFirstAlignedLevel) + (int64_t)(T - 1) * kTile);
  g.T = T;
  g.lvl = (uint32_t)level_of(p0);
  g.z = (p0 - (uint32_t)level_offset((int)g.lvl)) >> 8;
  g.cx = compact_even(g.z);
  g.cy = compact_even(g.z >> 1);
}
__device__ __forceinline__ void tile_geo_next(TileGeo& g) {
  g.T++;
  if (g.z + 1u == 1u << (2u * (g.lvl - (uint32_t)kFirstAlignedLevel))) {  // the level's last tile
    g.lvl++;
    g.z = g.cx = g.cy = 0;
    return;
  }
  // z + 1 clears z's t trailing ones (ceil(t/2) column bits, floor(t/2) row bits) and sets bit t
  const uint32_t t = (uint32_t)__builtin_ctz(~g.z);
  g.z++;
  g.cx &= ~((1u << ((t + 1u) >> 1)) - 1u);
  g.cy &= ~((1u << (t >> 1)) - 1u);
  if (t & 1u)
    g.cy |= 1u << (t >> 1);
  else
    g.cx |= 1u << (t >> 1);
}

// Per-lane constants of the position decode. Lane l holds parent q0 + l of a tile whose first
// parent is q0. In a level-aligned tile the children's Morton indices are m0 + 4 l + c (m0 a
// multiple of 256): lane bits 0, 2, 4 are the cell column's bits 1..3, lane bits 1, 3, 5 the row's,
// and child c adds column bit 0 = c & 1 and row bit 0 = c >> 1. Eq. 1: x = (2 column + 1)
// 2^-level - 1, and likewise y; xl, yl hold the lane's and child's part of 2 column and 2 row.
struct LaneGeo {
  float xl[2], yl[2];
};

// The tables and outputs of a launch.
struct DiscoverPtrs {
  cu32* blob;
  cu32* groups;
  cf32* bias;
  uint64_t* status;
  uint32_t* err;
  uint32_t* parent;
  float* w4;
  int64_t* pair_count;
  float* raw;
};

// One chunk (chunk_tiles consecutive tiles of one group) of a part with S sources per walk. A lane
// holds the four children (grid indices 4 q .. 4 q + 3) of TPW = P / 4 parent cells q, one in each
// tile of the walk, and evaluates the S sources at those P positions at once (M = S * P
// instances; instance m = s * P + 4 k + c is source s at child c of the lane's parent in tile k).
// One walk of the program therefore serves M queries per lane, and a cell's variance is formed
// inside the lane.
template <int S, int W, int MODE>
__device__ __forceinline__ void discover_chunk(uint32_t c, const DiscoverPart& pt,
                                               const DiscoverScalars& a, const DiscoverPtrs& d,
                                               const LaneGeo& geo, uint32_t lane) {
  constexpr int P = positions_per_lane(S, W);
  static_assert(P == 4 || P == 8 || P == 16, "a lane holds whole sibling quads");
  constexpr int M = S * P;
  constexpr int TPW = P / kTileIters;  // tiles per walk
  // (the launcher makes chunk_tiles a multiple of TPW, so a walk's tiles lie in one chunk)
  const uint32_t gi = pt.group0 + c / pt.chunks_per_group;
  const uint32_t chunk_tile = (c % pt.chunks_per_group) * pt.chunk_tiles;
  const Group G = load_group(d.groups + 12 * gi);
  // Every table-derived offset, count and id is checked before use: an entry that points outside
  // its table raises an error flag and the chunk is skipped instead of reading or writing wild.
  // The walk reads records var_off .. var_off + 16 n_rec (one past the last: the prefetch) and
  // bias rows inside the group's n_rec + 2.
  // (32-bit arithmetic throughout: n_rec is bounded first, and no sum below can wrap.)
  {
    const uint32_t rec_words = kRecWords * (G.n_rec + 1), row_floats = 4u * (G.n_rec + 2);
    bool ok = G.n_rec <= kMaxRecords && G.n_steps <= G.n_rec &&
              (G.var_off & (kRecWords - 1)) == 0 && (G.bias_off & 3u) == 0 &&
              rec_words <= a.blob_words && G.var_off <= a.blob_words - rec_words &&
              row_floats <= a.bias_floats && G.bias_off <= a.bias_floats - row_floats;
#pragma unroll
    for (int s = 0; s < S; ++s) ok = ok && G.pair[s] < a.n_pairs;
    if (!ok) {
      if (lane == 0) atomicOr(d.err, kErrTable);
      return;
    }
  }
  const uint32_t n_rec = (G.flags & 1u) != 0 ? G.n_rec : 0u;  // no records: a uniform output
  const uint32_t chunk_end = min(chunk_tile + pt.chunk_tiles, a.tiles);
  if constexpr (MODE != kModeRaw) {
    if (n_rec == 0 && !(0.0f > a.theta16)) {
      // A uniform output has variance 0 everywhere: with theta >= 0 every tile of the chunk keeps
      // nothing, and its counts (padded) or inclusive prefixes (look-back: all zero, no
      // predecessor needed) are written at once.
      if (lane == 0) {
        for (uint32_t t = chunk_tile; t < chunk_end; ++t)
#pragma unroll
          for (int s = 0; s < S; ++s) {
            uint64_t* w = d.status + (int64_t)G.pair[s] * a.tiles + t;
            if constexpr (MODE == kModePadded) {
              *w = 0ull;
            } else {
              status_store(w, kStatusInclusive);
              if (t + 1 == a.tiles) d.pair_count[G.pair[s]] = 0;
            }
          }
      }
      return;
    }
  }

  Walker<S, P, W> R;
  TileGeo tg{0u, 0u, 0u, 0u, 0u};  // T = 0: not set yet
  for (uint32_t t0 = chunk_tile; t0 < chunk_end; t0 += TPW) {
    // ---- geometry of the walk's tiles (t0 counts from the launch's first tile, tile_lo). The
    // pair's tile 0 holds the parents of levels 1..3 (21 of them; the positions decoded one by
    // one); every other tile 64 parents of one level, whose 256 children start at grid index p0.
    uint32_t p0[TPW];
    uint64_t vmask[TPW];  // lanes holding a queried parent
    float px[P], py[P];
#pragma unroll
    for (int k = 0; k < TPW; ++k) {
      const uint32_t tile = a.tile_lo + t0 + k;  // the pair's tile index
      const bool in_range = t0 + k < a.tiles;
      if (tile == 0) {
        p0[k] = 0;
        vmask[k] = !in_range ? 0ull
                   : a.head_parents >= 64u ? ~0ull
                                           : (1ull << a.head_parents) - 1ull;
        const uint32_t ln = lane_id_here();
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const uint32_t p = 4u * ln + (uint32_t)c4;
          const int l = level_of(p);
          const uint32_t mm = p - (uint32_t)level_offset(l);
          const float sc = pow2_neg(l);
          px[4 * k + c4] = __builtin_fmaf((float)(2u * compact_even(mm) + 1u), sc, -1.0f);
          py[4 * k + c4] = __builtin_fmaf((float)(2u * compact_even(mm >> 1) + 1u), sc, -1.0f);
        }
      } else {
        p0[k] = (uint32_t)(level_offset(kFirstAlignedLevel) + (int64_t)(tile - 1) * kTile);
        vmask[k] = in_range ? ~0ull : 0ull;
        if (tg.T != 0u && tile == tg.T + 1u)
          tile_geo_next(tg);
        else
          tile_geo_set(tg, tile);
        const float sc = pow2_neg((int)tg.lvl);
        const float bx = __builtin_fmaf((float)(32u * tg.cx + 1u), sc, -1.0f);
        const float by = __builtin_fmaf((float)(32u * tg.cy + 1u), sc, -1.0f);
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          px[4 * k + c4] = __builtin_fmaf(geo.xl[c4 & 1], sc, bx);
          py[4 * k + c4] = __builtin_fmaf(geo.yl[c4 >> 1], sc, by);
        }
      }
    }

    // ---- CPPN (Section 2): the varying program in topological order, M instances at once, in
    // one statement (the record step, generated): record r reads bias row 1 + r, and the next
    // record and row are loaded while the current one is computed. A uniform output is the
    // constant of row 0 (its program has no records).
    R.def();
    R.walk((uint64_t)(d.blob + G.var_off), (uint64_t)(d.bias + G.bias_off), n_rec, px, py);
    // the output node's activation was applied by its record's tail
    const float* w = R.acc;

    if constexpr (MODE == kModeRaw) {
#pragma unroll
      for (int s = 0; s < S; ++s)
#pragma unroll
        for (int k = 0; k < TPW; ++k)
          if ((vmask[k] >> lane) & 1ull) {
            float* o = d.raw + (int64_t)G.pair[s] * a.n_pos + p0[k] + 4u * lane;
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4) o[c4] = w[s * P + 4 * k + c4];
          }
      continue;
    }
    // ---- variance of the four siblings (Section 3.2) and the threshold test (Eq. 2), inside
    // the lane, from the pairwise split of the sum of squared deviations from the mean:
    // 16 var = 2 (w0 - w1)^2 + 2 (w2 - w3)^2 + ((w0 + w1) - (w2 + w3))^2, tested as
    // 16 var > 16 theta (both scalings by 16 exact, barring overflow or a subnormal variance).
    float s2[S][TPW];
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int k = 0; k < TPW; ++k) {
        const float* q = w + s * P + 4 * k;
        const float c = q[0] - q[1], d = q[2] - q[3];
        const float e = (q[0] + q[1]) - (q[2] + q[3]);
        s2[s][k] = __builtin_fmaf(__builtin_fmaf(d, d, c * c), 2.0f, e * e);
      }
    // Nearly every cell is dropped: one test on the maximum decides whether any record is kept.
    float mx = s2[0][0];
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int k = 0; k < TPW; ++k) mx = __builtin_fmaxf(mx, s2[s][k]);
    const bool some = ballot(mx > a.theta16) != 0ull;

    if constexpr (MODE == kModePadded) {
      uint32_t run[S][TPW];  // records per source and tile
      if (some) {
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
          for (int k = 0; k < TPW; ++k) {
            const uint64_t kb = ballot(s2[s][k] > a.theta16) & vmask[k];
            run[s][k] = popc64(kb);
            if ((kb >> lane) & 1ull) {
              // a tile's records start at its first parent index within the pair
              const int64_t slot = (int64_t)G.pair[s] * a.cap + ((p0[k] >> 2) - a.parent_lo) +
                                   mbcnt64(kb);
              d.parent[slot] = (p0[k] >> 2) + lane;
#pragma unroll
              for (int c4 = 0; c4 < 4; ++c4) d.w4[slot * 4 + c4] = w[s * P + 4 * k + c4];
            }
          }
      } else {
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
          for (int k = 0; k < TPW; ++k) run[s][k] = 0;
      }
      if (lane == 0) {
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
          for (int k = 0; k < TPW; ++k)
            if (t0 + k < a.tiles) d.status[(int64_t)G.pair[s] * a.tiles + t0 + k] = run[s][k];
      }
    }
    if constexpr (MODE == kModeLookback) {
      // ---- each tile learns its exact offset within each pair from the look-back scan, in
      // increasing tile order
#pragma unroll
      for (int k = 0; k < TPW; ++k) {
        const uint32_t tile = t0 + k;
        if (tile >= a.tiles) break;
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const uint64_t kb = some ? ballot(s2[s][k] > a.theta16) & vmask[k] : 0ull;
          const uint64_t cnt = popc64(kb);
          const uint32_t pair = G.pair[s];
          const uint64_t base = lookback(d.status + (int64_t)pair * a.tiles, tile, cnt, d.err);
          if (tile + 1 == a.tiles && lane == 0) {
            d.pair_count[pair] = (int64_t)(base + cnt);
            raise_max(d.err + 1, (uint32_t)min(base + cnt, (uint64_t)0xFFFFFFFFu));
          }
          if ((kb >> lane) & 1ull) {
            const int64_t idx = (int64_t)base + (int64_t)mbcnt64(kb);
            if (idx < a.cap) {
              const int64_t slot = (int64_t)pair * a.cap + idx;
              d.parent[slot] = (p0[k] >> 2) + lane;
#pragma unroll
              for (int c4 = 0; c4 < 4; ++c4) d.w4[slot * 4 + c4] = w[s * P + 4 * k + c4];
            }
          }
        }
      }
    }
  }
}

// One launch: every part, each chunk dispatched to the code of its part's (S, W). Chunks are
// handed out round-robin over the waves: chunk c goes to wave c mod n_waves. A group's chunks go
// to consecutive waves, so a pair's tiles are computed concurrently, and each wave visits its
// tiles in increasing order.
template <int MODE>
__global__ void __launch_bounds__(256)
    k_discover(const uint32_t* __restrict__ blob, const Group* __restrict__ groups,
               const float* __restrict__ bias_tab, uint64_t* __restrict__ status,
               uint32_t* __restrict__ err, uint32_t* __restrict__ parent, float* __restrict__ w4,
               int64_t* __restrict__ pair_count, float* __restrict__ raw, DiscoverScalars a) {
  const uint32_t lane = lane_id();
  const uint32_t i_lo = (lane & 1u) | ((lane >> 1) & 2u) | ((lane >> 2) & 4u);
  const uint32_t j_lo = ((lane >> 1) & 1u) | ((lane >> 2) & 2u) | ((lane >> 3) & 4u);
  const LaneGeo geo{{(float)(4u * i_lo), (float)(4u * i_lo + 2u)},
                    {(float)(4u * j_lo), (float)(4u * j_lo + 2u)}};
  const DiscoverPtrs d{(cu32*)blob, (cu32*)groups, (cf32*)bias_tab, status, err,
                       parent, w4, pair_count, raw};
  const uint32_t n_waves = gridDim.x * (blockDim.x / kWave);
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / kWave) +
                                                       threadIdx.x / kWave);
  for (uint32_t c = wave; c < a.n_chunks; c += n_waves) {
    // the chunk's part, and its index within the part
    uint32_t k = 0, cl = c;
    while (k + 1 < a.n_parts && cl >= a.part[k].n_chunks) {
      cl -= a.part[k].n_chunks;
      ++k;
    }
    const DiscoverPart pt = a.part[k];
    switch (pt.W * 4u + pt.S) {
      case 4 * 4 + 3: discover_chunk<3, 4, MODE>(cl, pt, a, d, geo, lane); break;
      case 4 * 4 + 2: discover_chunk<2, 4, MODE>(cl, pt, a, d, geo, lane); break;
      case 4 * 4 + 1: discover_chunk<1, 4, MODE>(cl, pt, a, d, geo, lane); break;
      case 8 * 4 + 3: discover_chunk<3, 8, MODE>(cl, pt, a, d, geo, lane); break;
      case 8 * 4 + 2: discover_chunk<2, 8, MODE>(cl, pt, a, d, geo, lane); break;
      case 8 * 4 + 1: discover_chunk<1, 8, MODE>(cl, pt, a, d, geo, lane); break;
      case 16 * 4 + 2: discover_chunk<2, 16, MODE>(cl, pt, a, d, geo, lane); break;
      case 16 * 4 + 1: discover_chunk<1, 16, MODE>(cl, pt, a, d, geo, lane); break;
      case 32 * 4 + 1: discover_chunk<1, 32, MODE>(cl, pt, a, d, geo, lane); break;
      default:
        if (lane == 0) atomicOr(err, kErrTable);
    }
  }
}
static_assert(max_group(4) == 3 && max_group(8) == 3 && max_group(16) == 2 && max_group(32) == 1,
              "the (S, W) variants of k_discover");

// ------------------------------------------------------------------------ bind kernel
// One wave per member (genome, direction, source). The wave copies the genome's uniform program
// into LDS with one coalesced pass, evaluates the uniform nodes in topological order (every lane
// computes the same values, fmaf in edge order), then each lane folds the uniform contributions
// of one varying node into that node's bias row entry.
constexpr int kMaxU = 5 + 256;
constexpr int kBindWaves = 4;
constexpr uint32_t kBindProgWords = 1024;  // larger uniform programs are read from global memory

__global__ void __launch_bounds__(kBindWaves * kWave)
    k_bind(const uint32_t* __restrict__ blob, const ProgDesc* __restrict__ desc,
           const Member* __restrict__ members, const float* __restrict__ src_xy,
           float* __restrict__ bias_tab, uint32_t* __restrict__ err, uint32_t n_members,
           uint32_t n_desc, uint32_t n_sources, uint32_t blob_words, uint64_t bias_floats) {
  __shared__ float U_all[kBindWaves][kMaxU];
  __shared__ uint32_t prog_all[kBindWaves][kBindProgWords];
  const uint32_t lane = lane_id();
  const uint32_t wv = threadIdx.x / kWave;
  const uint32_t i = __builtin_amdgcn_readfirstlane(blockIdx.x * kBindWaves + wv);
  if (i >= n_members) return;
  float* U = U_all[wv];
  const Member m = members[i];
  bool ok = m.desc < n_desc && m.source < n_sources;
  const ProgDesc d = desc[ok ? m.desc : 0];
  ok = ok && d.uni_off + 4ull <= d.uni_end && d.uni_end <= blob_words;
  const uint32_t words = ok ? d.uni_end - d.uni_off : 0u;
  // Program words relative to uni_off, from LDS when they fit.
  const uint32_t* prog = blob + d.uni_off;
  if (ok && words <= kBindProgWords) {
    for (uint32_t k = lane; k < words; k += kWave) prog_all[wv][k] = prog[k];
    prog = prog_all[wv];
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  uint32_t n_un = 0, out_u = kNone, n_steps = 0;
  if (ok) {
    n_un = prog[0];
    out_u = prog[1];
    n_steps = prog[2];
    // The member's bias rows: row 0 and rows 1..n_steps, all inside the group's rows.
    const uint64_t row0 = m.bias_base & ~3u;
    ok = n_un <= kMaxU - 5 && n_steps <= kMaxSteps && n_steps + 2 <= m.bias_rows &&
         4ull + 4ull * (n_un + n_steps) <= words && (out_u == kNone || out_u < 5 + n_un) &&
         row0 + 4ull * m.bias_rows <= bias_floats;
  }
  if (!ok) {
    if (lane == 0) atomicOr(err, kErrTable);
    return;
  }
  const uint32_t dir = m.desc & 1u;
  const float sx = src_xy[2 * m.source], sy = src_xy[2 * m.source + 1];
  // Input roles: the source fills (x1, y1) for outgoing queries and (x2, y2) for incoming ones;
  // the position-dependent roles are never read by the uniform program.
  if (lane < 5) {
    const float in5[5] = {dir == 0 ? sx : 0.0f, dir == 0 ? sy : 0.0f, dir == 0 ? 0.0f : sx,
                          dir == 0 ? 0.0f : sy, 1.0f};
    U[lane] = in5[lane];
  }
  // Edge lists are word offsets from uni_off and must lie inside this uniform program.
  auto edges_ok = [&](uint32_t off, uint32_t cnt) { return (uint64_t)off + 2ull * cnt <= words; };
  bool bad = false;
  for (uint32_t k = 0; k < n_un && !bad; ++k) {
    const uint32_t* rec = prog + 4 + 4 * k;
    const uint32_t act = rec[0], cnt = rec[1], off = rec[2];
    float z = __uint_as_float(rec[3]);
    if (!edges_ok(off, cnt)) {
      bad = true;
      break;
    }
    const uint32_t* ep = prog + off;
    for (uint32_t e = 0; e < cnt; ++e)
      z = __builtin_fmaf(__uint_as_float(ep[2 * e + 1]), U[min(ep[2 * e], 4u + k)], z);
    // every lane computed the same value and stores it to the same word
    U[5 + k] = act_apply(act, z);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const uint32_t* fold = prog + 4 + 4 * n_un;
  for (uint32_t t = lane; t < n_steps && !bad; t += kWave) {
    float z = __uint_as_float(fold[4 * t + 2]);
    const uint32_t cnt = fold[4 * t], off = fold[4 * t + 1], rec = fold[4 * t + 3];
    if (!edges_ok(off, cnt) || rec + 2 >= m.bias_rows) {
      bad = true;
      break;
    }
    const uint32_t* ep = prog + off;
    for (uint32_t e = 0; e < cnt; ++e)
      z = __builtin_fmaf(__uint_as_float(ep[2 * e + 1]), U[min(ep[2 * e], 4u + n_un)], z);
    bias_tab[m.bias_base + 4 * (1 + rec)] = z;
  }
  if (bad) atomicOr(err, kErrTable);
  if (lane == 0) bias_tab[m.bias_base] = out_u == kNone ? 0.0f : U[out_u];
}

// ------------------------------------------------------------------------ gather
// Packs the compacted records of all pairs into one contiguous list, pair after pair: pair r's
// min(count_r, cap) records go to offset sum_{q < r} min(count_q, cap). Workgroup b handles pairs
// 64 b .. 64 b + 63; it sums the counts before its first pair itself, so no other pass is needed.
constexpr int kGatherPairs = 64;

__global__ void __launch_bounds__(256)
    k_gather(const int64_t* __restrict__ counts, const uint32_t* __restrict__ parent,
             const float* __restrict__ w4, int64_t cap, uint32_t n_pairs,
             uint32_t* __restrict__ out_parent, float* __restrict__ out_w4) {
  __shared__ uint64_t part[256];
  __shared__ uint64_t offs[kGatherPairs + 1];
  const uint32_t first = blockIdx.x * kGatherPairs;
  auto clamp = [&](uint32_t r) -> uint64_t {
    const int64_t c = counts[r];
    return (uint64_t)(c < 0 ? 0 : (c < cap ? c : cap));
  };
  uint64_t mine = 0;
  for (uint32_t r = threadIdx.x; r < first; r += blockDim.x) mine += clamp(r);
  part[threadIdx.x] = mine;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t base = 0;
    for (int k = 0; k < 256; ++k) base += part[k];
    offs[0] = base;
    for (int i = 0; i < kGatherPairs; ++i)
      offs[i + 1] = offs[i] + (first + i < n_pairs ? clamp(first + i) : 0ull);
  }
  __syncthreads();
  const uint32_t lane = lane_id();
  for (uint32_t i = threadIdx.x / kWave; i < (uint32_t)kGatherPairs && first + i < n_pairs;
       i += blockDim.x / kWave) {
    const uint64_t n = offs[i + 1] - offs[i], dst = offs[i];
    const int64_t src = (int64_t)(first + i) * cap;
    for (uint64_t e = lane; e < n; e += kWave) {
      out_parent[dst + e] = parent[src + e];
      reinterpret_cast<float4*>(out_w4)[dst + e] = reinterpret_cast<const float4*>(w4)[src + e];
    }
  }
}

// ------------------------------------------------------------------------ small kernels
__global__ void k_fill(uint32_t* p, int64_t n_words, uint32_t value) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_words;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = value;
}

__global__ void k_grid(float* xy, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t p = (uint32_t)i;
    const int l = level_of(p);
    const uint32_t m = p - (uint32_t)level_offset(l);
    const float scale = pow2_neg(l);
    xy[2 * i] = __builtin_fmaf((float)(2u * compact_even(m) + 1u), scale, -1.0f);
    xy[2 * i + 1] = __builtin_fmaf((float)(2u * compact_even(m >> 1) + 1u), scale, -1.0f);
  }
}

}  // namespace emr

// ------------------------------------------------------------------------ launchers
// Called by the host runtime (runtime.cpp); each returns the hipError_t of its launch.
extern "C" hipError_t emr_launch_fill(void* p, int64_t n_words, uint32_t value, hipStream_t s) {
  if (n_words <= 0) return hipSuccess;
  int64_t blocks = (n_words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(emr::k_fill, dim3((uint32_t)blocks), dim3(256), 0, s, (uint32_t*)p, n_words,
                     value);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_grid(float* xy, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(emr::k_grid, dim3((uint32_t)blocks), dim3(256), 0, s, xy, n);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_bind(const emr::BindArgs* a, hipStream_t s) {
  if (a->n_members == 0) return hipSuccess;
  hipLaunchKernelGGL(emr::k_bind, dim3((a->n_members + emr::kBindWaves - 1) / emr::kBindWaves),
                     dim3(emr::kBindWaves * emr::kWave), 0, s, a->blob, a->desc,
                     a->members, a->src_xy, a->bias_tab, a->err, a->n_members, a->n_desc,
                     a->n_sources, a->blob_words, a->bias_floats);
  return hipGetLastError();
}

template <int MODE>
static hipError_t launch_discover_t(const emr::DiscoverArgs* a, uint32_t blocks, hipStream_t s,
                                    hipEvent_t start, hipEvent_t stop) {
  auto kern = emr::k_discover<MODE>;
  int dev = 0, cus = 0;
  hipError_t e;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
    return e;
  if (cus <= 0) cus = 1;
  // Workgroups of this kernel that fit on one CU (a property of the compiled kernel).
  static const int per_cu = [&] {
    int n = 0;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, 256, 0) == hipSuccess && n > 0
               ? n
               : 1;
  }();
  if (a->n_parts == 0 || a->n_parts > (uint32_t)emr::kMaxParts) return hipErrorInvalidValue;
  uint64_t groups = 0;
  for (uint32_t k = 0; k < a->n_parts; ++k) {
    const int S = (int)a->part_S[k], W = (int)a->part_W[k];
    if ((W != 4 && W != 8 && W != 16 && W != 32) || S < 1 || S > emr::max_group(W))
      return hipErrorInvalidValue;
    groups += a->part_groups[k];
  }
  // Chunks of 4 tiles when the launch has work for at least 4 such chunks per SIMD; else each
  // chunk is one walk's worth of tiles, for parallelism.
  const bool big = groups * a->tiles >= 16ull * 4ull * (uint64_t)cus;
  emr::DiscoverScalars sc{};
  sc.cap = a->cap;
  sc.n_pos = a->n_pos;
  sc.tile_lo = a->tile_lo;
  sc.parent_lo = a->parent_lo;
  sc.tiles = a->tiles;
  sc.n_parts = a->n_parts;
  uint64_t chunks = 0;
  for (uint32_t k = 0; k < a->n_parts; ++k) {
    const int S = (int)a->part_S[k], W = (int)a->part_W[k];
    const uint32_t tpw = (uint32_t)emr::positions_per_lane(S, W) / emr::kTileIters;
    const uint32_t chunk = big ? 4u : tpw;
    const uint32_t cpg = (a->tiles + chunk - 1) / chunk;
    sc.part[k] = emr::DiscoverPart{(uint32_t)S, (uint32_t)W, a->part_group0[k],
                                   a->part_groups[k] * cpg, cpg, chunk};
    chunks += (uint64_t)a->part_groups[k] * cpg;
  }
  if (chunks > 0xFFFFFFFFull) return hipErrorInvalidValue;
  sc.n_chunks = (uint32_t)chunks;
  sc.depth = a->depth;
  sc.theta16 = 16.0f * a->theta;
  sc.blob_words = a->blob_words;
  sc.n_pairs = a->n_pairs;
  sc.bias_floats = (uint32_t)a->bias_floats;
  sc.head_parents =
      (uint32_t)(a->depth < emr::kFirstAlignedLevel ? emr::n_parents(a->depth)
                                                    : emr::level_offset(emr::kFirstAlignedLevel) / 4);
  // Clamp the grid to what can be resident at once: the waves walk their chunks. The look-back
  // mode is launched cooperatively (the runtime refuses a grid that cannot be resident all at
  // once), which its forward progress relies on; the other modes have no waits between waves.
  const uint32_t resident = (uint32_t)per_cu * (uint32_t)cus;
  const uint32_t needed = (uint32_t)((chunks + 3) / 4);  // one wave per chunk, 4 per workgroup
  if (blocks > needed) blocks = needed;
  if (blocks > resident) blocks = resident;
  if (blocks == 0) {
    // nothing to run: the events still bracket the (empty) launch position
    if (start && (e = hipEventRecord(start, s)) != hipSuccess) return e;
    if (stop && (e = hipEventRecord(stop, s)) != hipSuccess) return e;
    return hipSuccess;
  }
  const uint32_t* blob = a->blob;
  const emr::Group* grp = a->groups;
  const float* bias_tab = a->bias_tab;
  uint64_t* status = a->status;
  uint32_t* err = a->err;
  uint32_t* parent = a->parent;
  float* w4 = a->w4;
  int64_t* pair_count = a->pair_count;
  float* raw = a->raw;
  if (start && (e = hipEventRecord(start, s)) != hipSuccess) return e;
  if constexpr (MODE == emr::kModeLookback) {
    void* args[] = {&blob, &grp, &bias_tab, &status, &err, &parent, &w4, &pair_count, &raw, &sc};
    e = hipLaunchCooperativeKernel((const void*)kern, dim3(blocks), dim3(256), args, 0, s);
  } else {
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, s, blob, grp, bias_tab, status, err,
                       parent, w4, pair_count, raw, sc);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  return stop ? hipEventRecord(stop, s) : hipSuccess;
}

// One launch for all the parts (sources per walk and register window) listed in *a. blocks: the
// most 256-thread workgroups (4 waves each) to launch; the launch uses at most one wave per chunk
// of tiles and no more workgroups than can be resident at once; every wave walks its share of the
// chunks. start, stop: events recorded on s around the launch, or NULL.
// mode: 0 raw outputs, 1 padded records (then emr_launch_compact), 2 look-back records.
extern "C" hipError_t emr_launch_discover(const emr::DiscoverArgs* a, int mode, uint32_t blocks,
                                          hipStream_t s, hipEvent_t start, hipEvent_t stop) {
  switch (mode) {
    case emr::kModeRaw: return launch_discover_t<emr::kModeRaw>(a, blocks, s, start, stop);
    case emr::kModePadded: return launch_discover_t<emr::kModePadded>(a, blocks, s, start, stop);
    case emr::kModeLookback:
      return launch_discover_t<emr::kModeLookback>(a, blocks, s, start, stop);
    default: return hipErrorInvalidValue;
  }
}

extern "C" hipError_t emr_launch_gather(const int64_t* counts, const uint32_t* parent,
                                        const float* w4, int64_t cap, uint32_t n_pairs,
                                        uint32_t* out_parent, float* out_w4, hipStream_t s) {
  if (n_pairs == 0) return hipSuccess;
  hipLaunchKernelGGL(emr::k_gather, dim3((n_pairs + emr::kGatherPairs - 1) / emr::kGatherPairs),
                     dim3(256), 0, s, counts, parent, w4, cap, n_pairs, out_parent, out_w4);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_compact(const uint64_t* counts, uint32_t* parent, float* w4,
                                         int64_t* pair_count, uint32_t* max_count, int64_t cap,
                                         uint32_t tile_lo, uint32_t tiles, uint32_t n_pairs,
                                         uint32_t head_slots, hipStream_t s) {
  if (n_pairs == 0) return hipSuccess;
  uint32_t blocks = (n_pairs + emr::kCompactWaves - 1) / emr::kCompactWaves;
  if (blocks > 1024) blocks = 1024;  // waves loop over pairs beyond this
  hipLaunchKernelGGL(emr::k_compact, dim3(blocks), dim3(emr::kCompactWaves * emr::kWave), 0, s,
                     counts, parent, w4, pair_count, max_count, cap, tile_lo, tiles, n_pairs,
                     head_slots);
  return hipGetLastError();
}
