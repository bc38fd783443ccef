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

#include <mutex>

#include "../../include/emr.h"
#include "emr_internal.h"
#include "discover.h"

namespace emr {

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

// ------------------------------------------------------------------------ compaction
// First parent index of a pair's tile T: tile 0 holds the parents of levels 1..3, every other tile
// 64 parents.
__device__ __forceinline__ uint32_t tile_parent_offset(uint32_t T) {
  return T == 0 ? 0u : (uint32_t)(level_offset(kFirstAlignedLevel) / 4) + (T - 1) * (kTile / 4);
}

// Compaction of one pair by one wave, once every tile of the range has left its records at the
// tile's own slots and its count in counts[pair * tiles + t]. The tiles go in groups of 64 in
// increasing order: a group's counts are scanned and its records moved down to their final,
// contiguous place. A range of more than two groups visits only the groups whose bit the discover
// kernel set in the pair's words of `nz` (a group that kept nothing has no records to move), and
// clears those words for the next range. Writes the pair's count and returns it.
__device__ uint32_t compact_pair(const uint64_t* __restrict__ counts, uint32_t* __restrict__ parent,
                                 float* __restrict__ w4, int64_t* __restrict__ pair_count,
                                 uint64_t* __restrict__ nz, int64_t cap, uint32_t tile_lo,
                                 uint32_t tiles, uint32_t pair, uint32_t head_slots,
                                 uint32_t lane) {
  const uint32_t parent_lo = tile_parent_offset(tile_lo);
  const uint64_t* row = counts + (int64_t)pair * tiles;
  const int64_t region = (int64_t)pair * cap;
  const uint32_t n_groups = (tiles + kWave - 1) / kWave;
  uint32_t running = 0;
  // lane's tile count in group g (a tile holds at most its own slot count: 64, or the head
  // tile's parents)
  auto load_count = [&](uint32_t g) -> uint32_t {
    const uint32_t t_lane = g * kWave + lane;
    const uint32_t slots = tile_lo + t_lane == 0 ? head_slots : (uint32_t)(kTile / 4);
    return t_lane < tiles ? min((uint32_t)row[t_lane], slots) : 0u;
  };
  auto group = [&](uint32_t g, uint32_t c) {
    const uint32_t t0 = g * kWave;
    // inclusive scan over the wave, bit-sliced: c < 128, so the counts of the lanes below are
    // the sum over bits b of 2^b times the number of lanes below with bit b set (mbcnt)
    uint32_t incl = c;
#pragma unroll
    for (int b = 0; b < 7; ++b) incl += mbcnt64(ballot((c >> b) & 1u)) << b;
    // The group's records in batches of 64, lane l moving the batch's l-th record: its tile is
    // the one (among the tiles with records) whose scan range holds it. A batch's loads all come
    // before its stores, and no record moves up, so a batch never overwrites a later batch's
    // records before they are read.
    const uint32_t total = __builtin_amdgcn_readlane(incl, kWave - 1);
    const uint64_t has = ballot(c != 0u);
    for (uint32_t b = 0; b < total; b += kWave) {
      const uint32_t q = b + lane;  // the record's rank among the group's records
      uint32_t src = running + q;
      for (uint64_t m = has; m != 0ull; m &= m - 1ull) {
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
  };
  if (n_groups <= kNzMinGroups) {
    // Both groups' counts are requested at once, and both groups' records move in one sequence
    // of batches (rank q < total0 in group 0, else rank q - total0 in group 1), so a pair with
    // few records waits for one round of record loads. Ranks ascend with the source slots and
    // every record moves down, as within one group.
    const uint32_t c0 = load_count(0), c1 = n_groups > 1 ? load_count(1) : 0u;
    auto scan = [&](uint32_t c) {
      uint32_t incl = c;
#pragma unroll
      for (int b = 0; b < 7; ++b) incl += mbcnt64(ballot((c >> b) & 1u)) << b;
      return incl;
    };
    const uint32_t incl0 = scan(c0), incl1 = scan(c1);
    const uint32_t total0 = __builtin_amdgcn_readlane(incl0, kWave - 1);
    const uint32_t total = total0 + __builtin_amdgcn_readlane(incl1, kWave - 1);
    const uint64_t has0 = ballot(c0 != 0u), has1 = ballot(c1 != 0u);
    for (uint32_t b = 0; b < total; b += kWave) {
      const uint32_t q = b + lane, q1 = q - total0;  // (q1 wraps above every range for q < total0)
      uint32_t src = q;
      for (uint64_t m = has0; m != 0ull; m &= m - 1ull) {
        const uint32_t i = (uint32_t)__builtin_ctzll(m);
        const uint32_t hi = __builtin_amdgcn_readlane(incl0, i);
        const uint32_t lo = hi - __builtin_amdgcn_readlane(c0, i);
        if (q >= lo && q < hi) src = tile_parent_offset(tile_lo + i) - parent_lo + (q - lo);
      }
      for (uint64_t m = has1; m != 0ull; m &= m - 1ull) {
        const uint32_t i = (uint32_t)__builtin_ctzll(m);
        const uint32_t hi = __builtin_amdgcn_readlane(incl1, i);
        const uint32_t lo = hi - __builtin_amdgcn_readlane(c1, i);
        if (q1 >= lo && q1 < hi)
          src = tile_parent_offset(tile_lo + kWave + i) - parent_lo + (q1 - lo);
      }
      if (q < total && src != q) {
        const uint32_t pv = parent[region + src];
        const float4 wv = reinterpret_cast<const float4*>(w4)[region + src];
        parent[region + q] = pv;
        reinterpret_cast<float4*>(w4)[region + q] = wv;
      }
    }
    running = total;
  } else {
    const uint32_t n_words = nz_words(tiles);
    uint64_t* words = nz + (int64_t)pair * n_words;
    for (uint32_t w0 = 0; w0 < n_words; w0 += kWave) {
      const bool mine = w0 + lane < n_words;
      const uint64_t bits = mine ? words[w0 + lane] : 0ull;
      if (mine && bits != 0ull) words[w0 + lane] = 0ull;
      // the marked groups of these words in increasing order (all values wave-uniform); each
      // group's counts are requested before the previous group is compacted
      uint64_t lanes = ballot(bits != 0ull), bw = 0ull;
      uint32_t i = 0;
      auto next = [&]() -> uint32_t {  // the next marked group, or ~0u
        while (bw == 0ull) {
          if (lanes == 0ull) return 0xFFFFFFFFu;
          i = (uint32_t)__builtin_ctzll(lanes);
          lanes &= lanes - 1ull;
          bw = ((uint64_t)__builtin_amdgcn_readlane((uint32_t)(bits >> 32), i) << 32) |
               __builtin_amdgcn_readlane((uint32_t)bits, i);
        }
        const uint32_t j = (uint32_t)__builtin_ctzll(bw);
        bw &= bw - 1ull;
        return (w0 + i) * kWave + j;
      };
      uint32_t g = next();
      uint32_t c = g < n_groups ? load_count(g) : 0u;
      while (g != 0xFFFFFFFFu) {
        const uint32_t g2 = next();
        const uint32_t c2 = g2 < n_groups ? load_count(g2) : 0u;
        if (g < n_groups) group(g, c);
        g = g2;
        c = c2;
      }
    }
  }
  if (lane == 0) pair_count[pair] = running;
  return running;
}

// The call's last kernel: its flags (error bits in flags[0], largest pair count in flags[1],
// raised with device-scope atomics by the call's other kernels; zero when the call starts) go to
// its pinned host words and are cleared for the slot's next call.
__global__ void k_finalize(uint32_t* flags, uint32_t* host) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  const uint32_t e = __hip_atomic_load(flags, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t m = __hip_atomic_load(flags + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  host[0] = e;
  host[1] = m;
  __hip_atomic_store(flags, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(flags + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Each wave takes pairs pair = wave, wave + n_waves, ...: compacts them once every discover launch
// of the range has finished, and the workgroup's largest count is raised into *max_count with one
// atomic. A pair with skip[pair] set (its groups were left out of the launch: they keep nothing)
// gets a count of 0 without its tile counts being read.
constexpr int kCompactWaves = 4;

__global__ void __launch_bounds__(kCompactWaves * kWave)
    k_compact(const uint64_t* __restrict__ counts, uint32_t* __restrict__ parent,
              float* __restrict__ w4, int64_t* __restrict__ pair_count,
              uint32_t* __restrict__ max_count, uint64_t* __restrict__ nz,
              const uint8_t* __restrict__ skip, int64_t cap, uint32_t tile_lo, uint32_t tiles,
              uint32_t n_pairs, uint32_t head_slots) {
  __shared__ uint32_t wave_max[kCompactWaves];
  const uint32_t lane = lane_id();
  const uint32_t wv = threadIdx.x / kWave;
  const uint32_t n_waves = gridDim.x * kCompactWaves;
  uint32_t my_max = 0;
  for (uint32_t pair = __builtin_amdgcn_readfirstlane(blockIdx.x * kCompactWaves + wv);
       pair < n_pairs; pair += n_waves) {
    if (skip && skip[pair]) {
      if (lane == 0) pair_count[pair] = 0;
      continue;
    }
    my_max = max(my_max, compact_pair(counts, parent, w4, pair_count, nz, cap, tile_lo, tiles,
                                      pair, head_slots, lane));
  }
  if (lane == 0) wave_max[wv] = my_max;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t m = 0;
    for (int k = 0; k < kCompactWaves; ++k) m = max(m, wave_max[k]);
    raise_max(max_count, m);
  }
}

// The interpreting discover kernel: one launch covers every part of a call.
template <int MODE>
__global__ void __launch_bounds__(256)
    k_discover(const uint32_t* __restrict__ geo, const uint32_t* __restrict__ blob,
               const Group* __restrict__ groups,
               const float* __restrict__ bias_tab, uint64_t* __restrict__ status,
               uint32_t* __restrict__ err, uint32_t* __restrict__ parent, float* __restrict__ w4,
               int64_t* __restrict__ pair_count, float* __restrict__ raw, DiscoverScalars a) {
  discover_body<MODE, false>(geo, blob, groups, bias_tab, status, err, parent, w4, pair_count, raw,
                             a, 0ull);
}

// The tile geometry table of a depth: row T (T >= 1, a level-aligned tile of 256 positions) holds
// the corner term of its 16 x 16 block of cells (Eq. 1: (32 column + 1) 2^-level - 1, likewise for
// the row), the level's cell size 2^-level, and the grid index of its first position. Row 0 (the
// head tile, decoded lane by lane) and the rows from `tiles` to `rows` (padding) are zero.
__global__ void k_tile_geo(uint32_t* __restrict__ out, uint32_t tiles, uint32_t rows) {
  for (uint32_t T = blockIdx.x * blockDim.x + threadIdx.x; T < rows; T += gridDim.x * blockDim.x) {
    uint32_t r[4] = {0u, 0u, 0u, 0u};  // tile 0 (decoded per position) and the padding rows
    if (T > 0 && T < tiles) {
      TileGeo g;
      tile_geo_set(g, T);
      const float sc = pow2_neg((int)g.lvl);
      r[0] = __float_as_uint(__builtin_fmaf((float)(32u * g.cx + 1u), sc, -1.0f));
      r[1] = __float_as_uint(__builtin_fmaf((float)(32u * g.cy + 1u), sc, -1.0f));
      r[2] = __float_as_uint(sc);
      r[3] = (uint32_t)(level_offset(kFirstAlignedLevel) + (int64_t)(T - 1) * kTile);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) out[4 * (size_t)T + q] = r[q];
  }
}

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
           uint32_t n_desc, uint32_t n_sources, uint32_t blob_words, uint64_t bias_floats,
           uint64_t* __restrict__ nz, uint32_t nz_words) {
  __shared__ float U_all[kBindWaves][kMaxU];
  __shared__ uint32_t prog_all[kBindWaves][kBindProgWords];
  // the compaction's group marks start out clear (the discover kernel sets them)
  for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < nz_words; k += gridDim.x * blockDim.x)
    nz[k] = 0ull;
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

// ------------------------------------------------------------------------ allocation-free scratch
// The device memory of emr_eval_raw_noalloc: a fixed array in the library's code object, so the
// loader places one copy on every device the library runs on and nothing is allocated per call.
// Host code never passes this name to a kernel (on the host it is only a stand-in for the
// symbol); it passes the device address emr_noalloc_scratch looks up.
static __device__ __align__(256) uint8_t scratch[EMR_NOALLOC_SCRATCH_BYTES];

}  // namespace emr

// The current device's address of the allocation-free scratch (EMR_NOALLOC_SCRATCH_BYTES bytes),
// looked up with that device current on its first use and kept per device.
extern "C" hipError_t emr_noalloc_scratch(void** out) {
  static std::mutex mu;
  static void* addr[256] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 256) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(emr::scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255) != 0) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

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

extern "C" hipError_t emr_launch_tile_geo(uint32_t* out, uint32_t tiles, uint32_t rows,
                                          hipStream_t s) {
  if (rows == 0) return hipSuccess;
  uint32_t blocks = (rows + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(emr::k_tile_geo, dim3(blocks), dim3(256), 0, s, out, tiles, rows);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_bind(const emr::BindArgs* a, hipStream_t s) {
  if (a->n_members == 0) return hipSuccess;
  hipLaunchKernelGGL(emr::k_bind, dim3((a->n_members + emr::kBindWaves - 1) / emr::kBindWaves),
                     dim3(emr::kBindWaves * emr::kWave), 0, s, a->blob, a->desc,
                     a->members, a->src_xy, a->bias_tab, a->err, a->n_members, a->n_desc,
                     a->n_sources, a->blob_words, a->bias_floats, a->nz, a->nz_words);
  return hipGetLastError();
}

// The scalars and grid of one discover launch (either tier). per_cu: workgroups of the kernel
// that fit on one CU; cus: the device's CUs; blocks: the most workgroups to launch. *grid is 0
// when there is nothing to run.
extern "C" hipError_t emr_discover_setup(const emr::DiscoverArgs* a, uint32_t blocks, int per_cu,
                                         int cus, emr::DiscoverScalars* out, uint32_t* grid) {
  if (per_cu <= 0) per_cu = 1;
  if (cus <= 0) cus = 1;
  if (a->n_parts == 0 || a->n_parts > (uint32_t)emr::kMaxParts) return hipErrorInvalidValue;
  if (!a->geo || (uint64_t)a->tile_lo + a->tiles + emr::kGeoPadRows > a->geo_rows)
    return hipErrorInvalidValue;
  uint64_t groups = 0;
  for (uint32_t k = 0; k < a->n_parts; ++k) {
    const int S = (int)a->part_S[k], W = (int)a->part_W[k];
    if ((W != 4 && W != 8 && W != 16 && W != 32) || S < 1 || S > emr::max_group(W))
      return hipErrorInvalidValue;
    groups += a->part_groups[k];
  }
  // Chunk size: the largest of 16, 8 and 4 tiles that still gives every resident wave at least
  // four chunks (fewer, longer chunks spend less per-chunk work; enough of them keep the waves
  // balanced); else each chunk is one walk's worth of tiles, for parallelism.
  const uint64_t waves = 4ull * (uint64_t)per_cu * (uint64_t)cus;
  uint32_t target = 0;
  for (uint32_t c : {emr::kChunkTilesMax, 8u, 4u})
    if (target == 0 && groups * ((a->tiles + c - 1) / c) >= 4ull * waves) target = c;
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
    const uint32_t chunk = target > tpw ? target : tpw;  // at most kChunkTilesMax (tpw <= 4)
    const uint32_t cpg = (a->tiles + chunk - 1) / chunk;
    sc.part[k] = emr::DiscoverPart{(uint32_t)S, (uint32_t)W, a->part_group0[k],
                                   a->part_groups[k] * cpg, cpg, chunk};
    chunks += (uint64_t)a->part_groups[k] * cpg;
  }
  if (chunks > 0xFFFFFFFFull) return hipErrorInvalidValue;
  sc.n_chunks = (uint32_t)chunks;
  sc.depth = a->depth;
  sc.theta16 = 16.0f * a->theta;
  sc.code_bytes = 0;
  sc.nz = a->nz;
  sc.nz_words = emr::nz_words(a->tiles);
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
  *out = sc;
  *grid = blocks;
  return hipSuccess;
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
  // Workgroups of this kernel that fit on one CU (a property of the compiled kernel).
  static const int per_cu = [&] {
    int n = 0;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, 256, 0) == hipSuccess && n > 0
               ? n
               : 1;
  }();
  emr::DiscoverScalars sc{};
  uint32_t grid = 0;
  if ((e = emr_discover_setup(a, blocks, per_cu, cus, &sc, &grid)) != hipSuccess) return e;
  if (grid == 0) {
    // nothing to run: the events still bracket the (empty) launch position
    if (start && (e = hipEventRecord(start, s)) != hipSuccess) return e;
    if (stop && (e = hipEventRecord(stop, s)) != hipSuccess) return e;
    return hipSuccess;
  }
  const uint32_t* geo = a->geo;
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
    void* args[] = {&geo, &blob, &grp, &bias_tab, &status, &err, &parent, &w4, &pair_count, &raw,
                    &sc};
    e = hipLaunchCooperativeKernel((const void*)kern, dim3(grid), dim3(256), args, 0, s);
  } else {
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), 0, s, geo, blob, grp, bias_tab, status, err,
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
                                         int64_t* pair_count, uint32_t* max_count, uint64_t* nz,
                                         const uint8_t* skip, int64_t cap, uint32_t tile_lo,
                                         uint32_t tiles, uint32_t n_pairs, uint32_t head_slots,
                                         hipStream_t s) {
  if (n_pairs == 0) return hipSuccess;
  uint32_t blocks = (n_pairs + emr::kCompactWaves - 1) / emr::kCompactWaves;
  if (blocks > 8192) blocks = 8192;  // waves loop over pairs beyond this
  hipLaunchKernelGGL(emr::k_compact, dim3(blocks), dim3(emr::kCompactWaves * emr::kWave), 0, s,
                     counts, parent, w4, pair_count, max_count, nz, skip, cap, tile_lo, tiles,
                     n_pairs, head_slots);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_finalize(uint32_t* flags, uint32_t* host, hipStream_t s) {
  hipLaunchKernelGGL(emr::k_finalize, dim3(1), dim3(64), 0, s, flags, host);
  return hipGetLastError();
}
