// The discover kernel's body, shared by the interpreting kernel (kernels.hip) and the kernels of
// the template code object for compiled programs (jit.hip): one lane per parent cell; each lane
// evaluates the varying CPPN program for S sources of one genome at the cell's four children at
// once (Section 3.1, the batched query W), reduces the four siblings to their variance in
// registers, applies var > theta (Section 3.2, Eq. 2), and writes the kept cells to a record pool
// (one reservation per walk that keeps any), leaving each tile's pool offset and count in its
// status word and each chunk's counts in its pairs' totals; k_scan and k_move then place every
// pair's records contiguously in ascending parent order.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/emr.h"
#include "emr_internal.h"

namespace emr {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x32 __attribute__((ext_vector_type(32)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));

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
// A 64-bit value of lane i (uniform i) / of the first active lane. The lane builtins return int:
// each half is taken as unsigned before widening (a sign-extended low half would set the high
// word whenever its bit 31 is set).
__device__ __forceinline__ uint64_t read_lane64(uint64_t v, uint32_t i) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, (int)i);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), (int)i);
  return ((uint64_t)hi << 32) | (uint64_t)lo;
}
__device__ __forceinline__ uint64_t first_lane64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | (uint64_t)lo;
}
__device__ __forceinline__ uint32_t popc64(uint64_t m) { return __builtin_popcountll(m); }
__device__ __forceinline__ uint32_t mbcnt64(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
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

// ------------------------------------------------------------------------ discover kernel
// Pointers are passed as separate restrict-qualified parameters so the compiler can prove that
// the program, group and bias tables are never written by the kernel and read them with scalar
// loads through the scalar cache.
// (DiscoverPart, DiscoverScalars and the output modes are in emr_internal.h.)

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
  g.code_off = p[5];
  g.pad[0] = g.pad[1] = 0;
#pragma unroll
  for (int k = 0; k < kMaxGroup; ++k) g.pair[k] = p[8 + k];
  return g;
}
static_assert(sizeof(Group) == 12 * sizeof(uint32_t), "Group layout");


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
  cu32* geo;  // tile geometry rows {bx, by, 2^-level, p0} (k_tile_geo)
  cu32* blob;
  cu32* groups;
  cf32* bias;
  uint64_t* status;
  uint32_t* err;
  float* raw;
};

// Record mode: the status words of a chunk's tiles, source s and tile chunk_tile + k held in lane
// 16 s + k (pool offset of the tile's records and their count), stored by those lanes at once (the
// status words of the tiles outside the launch range are never written); and each source's
// records of the chunk (totals[s], wave-uniform) added to its pair's total.
template <int S>
__device__ __forceinline__ void store_chunk_counts(const DiscoverPtrs& d, const DiscoverScalars& a,
                                                   const Group& G, uint32_t chunk_tile,
                                                   uint32_t chunk_end, uint32_t counts,
                                                   uint32_t bases, const uint32_t* totals,
                                                   uint32_t lane) {
#pragma unroll
  for (int s = 0; s < S; ++s)
    if (lane == 0 && totals[s] != 0u) atomicAdd(a.pair_total + G.pair[s], totals[s]);
  // one store per source (its pair id uniform), lanes 16 s .. 16 s + 15
  const uint32_t k = lane & 15u;
#pragma unroll
  for (int s = 0; s < S; ++s)
    if ((lane >> 4) == (uint32_t)s && chunk_tile + k < chunk_end)
      d.status[(int64_t)G.pair[s] * a.tiles + chunk_tile + k] =
          ((uint64_t)bases << kStatusCountBits) | (uint64_t)counts;
  // A chunk (a whole number of chunks fills a group of 64 tiles) that kept a cell marks its
  // group, so that the compaction of a long range visits only the groups with records.
  if (a.tiles > kNzMinGroups * kWave) {
    const uint64_t kept = ballot(counts != 0u);
    const uint32_t g = chunk_tile / kWave;
#pragma unroll
    for (int s = 0; s < S; ++s)
      if (lane == 0 && ((kept >> (16 * s)) & 0xFFFFull) != 0ull)
        atomicOr((unsigned long long*)(a.nz + (int64_t)G.pair[s] * a.nz_words + g / 64u),
                 1ull << (g % 64u));
  }
}

// One chunk (chunk_tiles consecutive tiles of one group) of a part with S sources per walk. A lane
// holds the four children (grid indices 4 q .. 4 q + 3) of TPW = P / 4 parent cells q, one in each
// tile of the walk, and evaluates the S sources at those P positions at once (M = S * P
// instances; instance m = s * P + 4 k + c is source s at child c of the lane's parent in tile k).
// One walk of the program therefore serves M queries per lane, and a cell's variance is formed
// inside the lane.
//
// JIT selects how the program runs: the interpreter (the record step) or the group's compiled
// program, called at code_base + its code offset.
template <int S, int W, int MODE, bool JIT>
__device__ __forceinline__ void discover_chunk(uint32_t c, const DiscoverPart& pt,
                                               const DiscoverScalars& a, const DiscoverPtrs& d,
                                               const LaneGeo& geo, uint32_t lane,
                                               uint64_t code_base) {
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
    // a compiled program lies inside the code area (its end is checked by the host)
    if constexpr (JIT) ok = ok && G.code_off < a.code_bytes && (G.code_off & 3u) == 0;
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
      // nothing, and its counts are written at once.
      const uint32_t none[S] = {};
      store_chunk_counts<S>(d, a, G, chunk_tile, chunk_end, 0u, 0u, none, lane);
      return;
    }
  }

  Walker<S, P, W> R;
  JitCall<S, P, W> J;
  // Compiled programs find the group's bias rows 1 .. 4 in their scalar registers: loaded once
  // per chunk (the workspace keeps 16 floats of padding after the bias table, so the load stays
  // inside it for the last group).
  u32x16 rows;
  if constexpr (JIT)
    rows = *reinterpret_cast<const __attribute__((address_space(4))) u32x16*>(
        d.bias + G.bias_off + 4u);
  // Record mode: the chunk's record counts and pool offsets, source s and tile chunk_tile + k in
  // lane 16 s + k; they stay zero unless a walk keeps a cell, and go out with one store per chunk.
  uint32_t chunk_counts = 0, chunk_bases = 0;
  uint32_t chunk_total[S];  // records of the chunk per source (wave-uniform)
#pragma unroll
  for (int s = 0; s < S; ++s) chunk_total[s] = 0u;
  // The geometry rows of the walk's tiles, loaded one walk ahead from gp (the rows of the next
  // walk's tiles). The host sizes the table for the launch's range plus kGeoPadRows rows of
  // padding (emr_discover_setup), which the last walks' loads reach; a walk past the range end
  // keeps nothing.
  uint32_t gnext[TPW][4];
  cu32* gp = d.geo + 4u * (a.tile_lo + chunk_tile);
  auto load_geo = [&]() {
#pragma unroll
    for (int k = 0; k < TPW; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) gnext[k][q] = gp[4 * k + q];
    gp += 4 * TPW;
  };
  load_geo();
  for (uint32_t t0 = chunk_tile; t0 < chunk_end; t0 += TPW) {
    uint32_t gcur[TPW][4];
#pragma unroll
    for (int k = 0; k < TPW; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) gcur[k][q] = gnext[k][q];
    // ---- geometry of the walk's tiles (t0 counts from the launch's first tile, tile_lo). The
    // pair's tile 0 holds the parents of levels 1..3 (21 of them; the positions decoded one by
    // one); every other tile 64 parents of one level, whose 256 children start at grid index p0,
    // with its block's corner and the level's cell size from the geometry table.
    uint32_t p0[TPW];
    uint64_t vmask[TPW];  // lanes holding a queried parent
    float px[P], py[P];
#pragma unroll
    for (int k = 0; k < TPW; ++k) {
      const uint32_t tile = a.tile_lo + t0 + k;  // the pair's tile index
      const bool in_range = t0 + k < a.tiles;
      if (k == 0 && tile == 0) {
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
        const float bx = __uint_as_float(gcur[k][0]), by = __uint_as_float(gcur[k][1]);
        const float sc = __uint_as_float(gcur[k][2]);
        p0[k] = gcur[k][3];
        vmask[k] = in_range ? ~0ull : 0ull;
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
    // The output node's activation was applied by its record's tail (or the compiled program).
    // The next walk's geometry rows are loaded while this walk runs: by the call statement before
    // it jumps to the program (the compiler waits for every pending scalar load before an asm
    // statement, so a load issued ahead of it in C++ would be waited for at once), or before the
    // interpreter's walk.
    const float* w;
    if constexpr (JIT) {
      typename JitCall<S, P, W>::Geo g;
      J.call(code_base + G.code_off, (uint64_t)(d.bias + G.bias_off), px, py, rows, (uint64_t)gp,
             g);
      gp += 4 * TPW;
#pragma unroll
      for (int k = 0; k < TPW; ++k)
#pragma unroll
        for (int q = 0; q < 4; ++q) gnext[k][q] = g[4 * k + q];
      w = J.acc;
    } else {
      load_geo();
      R.def();
      R.walk((uint64_t)(d.blob + G.var_off), (uint64_t)(d.bias + G.bias_off), n_rec, px, py);
      w = R.acc;
    }

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

    if constexpr (MODE == kModeRecords) {
      if (some) {
        // The walk's kept cells, source s and tile k: one pool reservation for all of them (one
        // atomic per walk that keeps anything), then each (s, k) segment in (s, k) order.
        uint64_t kb[S][TPW];
        uint32_t n_walk = 0;
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
          for (int k = 0; k < TPW; ++k) {
            kb[s][k] = ballot(s2[s][k] > a.theta16) & vmask[k];
            n_walk += popc64(kb[s][k]);
          }
        uint64_t off = 0;
        if (lane == 0)
          off = atomicAdd((unsigned long long*)a.pool_ctr, (unsigned long long)n_walk);
        off = first_lane64(off);
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
          for (int k = 0; k < TPW; ++k) {
            const uint32_t cnt = popc64(kb[s][k]);
            chunk_total[s] += cnt;
            if (lane == 16u * (uint32_t)s + min(t0 + (uint32_t)k - chunk_tile, 15u)) {
              chunk_counts = cnt;
              chunk_bases = (uint32_t)off;  // (a pool offset beyond 2^32 exceeds any capacity)
            }
            if ((kb[s][k] >> lane) & 1ull) {
              const uint64_t idx = off + mbcnt64(kb[s][k]);
              if (idx < (uint64_t)a.cap) {
                a.pool_parent[idx] = (p0[k] >> 2) + lane;
#pragma unroll
                for (int c4 = 0; c4 < 4; ++c4) a.pool_w4[idx * 4 + c4] = w[s * P + 4 * k + c4];
              }
            }
            off += cnt;
          }
      }
    }
  }
  if constexpr (MODE == kModeRecords)
    store_chunk_counts<S>(d, a, G, chunk_tile, chunk_end, chunk_counts, chunk_bases, chunk_total,
                          lane);
}

// One launch: every part, each chunk dispatched to the code of its part's (S, W). A workgroup
// (one CU) owns a share of the chunks: the entries of its list when the launch has a schedule
// (lists balanced across CUs by the host's cost model, costliest chunk first), else chunks
// b, b + n_wg, ... (round-robin); its waves take them in that order, one at a time, from a
// counter in LDS. Chunks are independent: each writes its own tiles' status words, records and raw
// outputs, and adds to counters, so neither their order nor their wave matters for the result.
// (The body of the discover kernels: k_discover below runs the interpreter, the template code
// object's kernels the compiled programs.)
template <int MODE, bool JIT>
__device__ __forceinline__ void discover_body(const uint32_t* __restrict__ geo_tab,
                                              const uint32_t* __restrict__ blob,
                                              const Group* __restrict__ groups,
                                              const float* __restrict__ bias_tab,
                                              uint64_t* __restrict__ status, uint32_t* __restrict__ err,
                                              float* __restrict__ raw, const DiscoverScalars& a,
                                              uint64_t code_base) {
  const uint32_t lane = lane_id();
  const uint32_t i_lo = (lane & 1u) | ((lane >> 1) & 2u) | ((lane >> 2) & 4u);
  const uint32_t j_lo = ((lane >> 1) & 1u) | ((lane >> 2) & 2u) | ((lane >> 3) & 4u);
  const LaneGeo geo{{(float)(4u * i_lo), (float)(4u * i_lo + 2u)},
                    {(float)(4u * j_lo), (float)(4u * j_lo + 2u)}};
  const DiscoverPtrs d{(cu32*)geo_tab, (cu32*)blob, (cu32*)groups, (cf32*)bias_tab, status, err,
                       raw};
  const uint32_t n_wg = gridDim.x, wg = blockIdx.x;
  // (the launcher accepts a schedule only when it was made for this grid: sched_lists == n_wg,
  // so row wg and its sched_stride entries lie inside the table; the interpreter, which runs the
  // calls without lists, leaves the list path out)
  const bool listed = JIT && a.sched != nullptr;
  // The workgroup's next share entry, and its list (at most kListLds entries), copied to LDS (a
  // wave then takes a chunk with two LDS accesses); one barrier before any wave takes one.
  __shared__ uint32_t next;
  __shared__ uint32_t list[kListLds];
  if (threadIdx.x == 0) next = 0u;
  if (listed)
    for (uint32_t i = threadIdx.x; i < a.sched_stride; i += blockDim.x)
      list[i] = a.sched[wg * a.sched_stride + i];
  __syncthreads();
  for (;;) {
    // The wave's share entry: every lane adds to `next`, lane 0 one and the others zero, so lane
    // 0 reads the entry it took. (One asm statement: as a lane-0 branch around an atomicAdd the
    // compiler keeps values live across the loop in a way that spills.)
    uint32_t e, one, addr;
    asm volatile(
        "v_mbcnt_lo_u32_b32 %1, -1, 0\n\t"
        "v_cmp_eq_u32_e32 vcc, 0, %1\n\t"
        "v_cndmask_b32_e64 %1, 0, 1, vcc\n\t"
        "v_mov_b32 %2, %3\n\t"
        "ds_add_rtn_u32 %0, %2, %1\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=v"(e), "=&v"(one), "=&v"(addr)
        : "s"((uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)&next)
        : "vcc", "memory");
    e = __builtin_amdgcn_readfirstlane(e);
    // the chunk, as a list entry: its part << kEntryPartShift | its index in the part
    uint32_t entry;
    if (listed) {
      if (e >= a.sched_stride) break;
      entry = __builtin_amdgcn_readfirstlane(list[e]);
      if (entry == kNoChunk) break;
    } else {
      // (each wave takes one entry past the share's end at most, so c < n_chunks + 13 n_wg,
      // which does not wrap with n_chunks < 2^31)
      uint32_t c = wg + e * n_wg;
      if (c >= a.n_chunks) break;
      uint32_t p = 0;
      while (p + 1 < a.n_parts && c >= a.part[p].n_chunks) {
        c -= a.part[p].n_chunks;
        ++p;
      }
      entry = p << kEntryPartShift | c;  // (setup bounds an unlisted part below 2^24 chunks)
    }
    // (the launcher checked every listed entry's index against its part when it made the lists;
    // a round-robin entry's index is inside its part by the scan)
    const uint32_t k = entry >> kEntryPartShift, cl = entry & ((1u << kEntryPartShift) - 1u);
    if (k >= a.n_parts) {
      if (lane == 0) atomicOr(err, kErrTable);
      break;
    }
    const DiscoverPart pt = a.part[k];
    switch (pt.W * 4u + pt.S) {
      case 4 * 4 + 3: discover_chunk<3, 4, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 4 * 4 + 2: discover_chunk<2, 4, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 4 * 4 + 1: discover_chunk<1, 4, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 8 * 4 + 3: discover_chunk<3, 8, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 8 * 4 + 2: discover_chunk<2, 8, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 8 * 4 + 1: discover_chunk<1, 8, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 16 * 4 + 2: discover_chunk<2, 16, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 16 * 4 + 1: discover_chunk<1, 16, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      case 32 * 4 + 1: discover_chunk<1, 32, MODE, JIT>(cl, pt, a, d, geo, lane, code_base); break;
      default:
        if (lane == 0) atomicOr(err, kErrTable);
    }
  }
}
static_assert(max_group(4) == 3 && max_group(8) == 3 && max_group(16) == 2 && max_group(32) == 1,
              "the (S, W) variants of the discover kernels");

}  // namespace emr
