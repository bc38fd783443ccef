// gfx950 kernels for eager multi-resolution substrate discovery.
//
//   k_grid      writes the cell centres of every queried position (Section 3.1, Eq. 1).
//   k_fill      clears the tile-group marks and per-pair totals of a workspace.
//   k_bind      evaluates the position-independent part of each (genome, source) CPPN once and
//               folds it into per-step biases (one wave per pair).
//   k_discover  the hot path: one lane per parent cell; each lane interprets the varying CPPN
//               program for S sources of one genome at the cell's four children at once
//               (Section 3.1, the batched query W), reduces the four siblings to their variance
//               in registers, applies var > theta (Section 3.2, Eq. 2), and writes the kept cells
//               to a record pool (one reservation per walk), each tile's pool offset and count to
//               its status word.
//   k_scan      one workgroup: the pairs' output offsets (exclusive scan of their totals), the
//               call's total and largest count, and the hand-over of the call's flags.
//   k_move      one wave per pair: gathers its records from the pool into its place in the
//               call's output (pairs back to back, CSR), in ascending parent order.
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
// After a record-mode discover launch every tile of the range has left its status word (pool
// offset << 8 | count) and every pair its total. k_scan turns the totals into output offsets
// (pairs back to back in pair order: CSR), k_move gathers each pair's records from the pool to its
// offset: tiles in increasing order, each tile's records in increasing lane (parent) order, so
// each pair's records come out in ascending parent order. Records whose pool or output index is
// beyond `cap`, or beyond their pair's count, are not moved (an overflowing call reports its
// total, which exceeds the capacity; a pair whose tiles were skipped after a table error gets no
// more than its count).

// The call's flag words go to its pinned host words and are cleared for the slot's next call.
__device__ __forceinline__ void hand_over_flags(uint32_t* flags, uint32_t* host) {
  uint32_t v[kFlagWords];
#pragma unroll
  for (int k = 0; k < kFlagWords; ++k)
    v[k] = __hip_atomic_load(flags + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  host[kFlagErr] = v[kFlagErr];
  host[kFlagMax] = v[kFlagMax];
  host[kFlagTotal] = v[kFlagTotal];
  host[kFlagTotal + 1] = v[kFlagTotal + 1];
#pragma unroll
  for (int k = 0; k < kFlagWords; ++k)
    __hip_atomic_store(flags + k, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The call's last kernel when k_scan does not hand over its flags (raw outputs, streamed calls).
__global__ void k_finalize(uint32_t* flags, uint32_t* host) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  hand_over_flags(flags, host);
}

constexpr int kScanThreads = 1024;
constexpr int kScanPer = 4;  // consecutive pairs per thread and round

// One workgroup: pairs in rounds of kScanThreads * kScanPer, thread t taking the kScanPer pairs
// from round + kScanPer t (their loads issued together). Writes pair_count, pair_offset
// (exclusive scan, pair_offset[n_pairs] = the total), clears the totals for the next launch,
// resets the pool counter, raises the largest count and stores the total in the flags, and, with
// A.host, hands the flags over. No other kernel writes the flag words while this one runs (the
// call's kernels are ordered on its stream and this is the only writer of the largest count), so
// thread 0 reads the words it needs together with the first round's totals and writes the final
// values without reading them again: the kernel waits for memory once before its stores.
__global__ void __launch_bounds__(kScanThreads) k_scan(ScanArgs A) {
  __shared__ uint64_t wsum[kScanThreads / kWave];
  __shared__ uint32_t wmax[kScanThreads / kWave];
  const uint32_t t = threadIdx.x, lane = t % kWave, wv = t / kWave;
  uint32_t f_err = 0, f_max = 0;
  if (t == 0) {
    f_err = __hip_atomic_load(A.flags + kFlagErr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    f_max = __hip_atomic_load(A.flags + kFlagMax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  uint64_t carry = 0;
  uint32_t mx = 0;
  for (uint32_t round = 0; round < A.n_pairs; round += kScanThreads * kScanPer) {
    const uint32_t i0 = round + t * kScanPer;
    uint32_t c[kScanPer];
#pragma unroll
    for (int k = 0; k < kScanPer; ++k) c[k] = i0 + k < A.n_pairs ? A.pair_total[i0 + k] : 0u;
    uint32_t mine = 0;
#pragma unroll
    for (int k = 0; k < kScanPer; ++k) {
      if (i0 + k < A.n_pairs) A.pair_total[i0 + k] = 0u;
      mine += c[k];
      mx = max(mx, c[k]);
    }
    uint64_t incl = mine;  // inclusive scan of the threads' sums within the wave
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const uint64_t v = __shfl_up(incl, off, kWave);
      if (lane >= (uint32_t)off) incl += v;
    }
    if (lane == kWave - 1) wsum[wv] = incl;
    __syncthreads();
    uint64_t before = 0, round_total = 0;
#pragma unroll
    for (int k = 0; k < kScanThreads / kWave; ++k) {
      if ((uint32_t)k < wv) before += wsum[k];
      round_total += wsum[k];
    }
    uint64_t at = carry + before + incl - mine;
#pragma unroll
    for (int k = 0; k < kScanPer; ++k)
      if (i0 + k < A.n_pairs) {
        A.pair_count[i0 + k] = c[k];
        if (A.host_counts) A.host_counts[i0 + k] = c[k];
        A.pair_offset[i0 + k] = (int64_t)at;
        at += c[k];
      }
    carry += round_total;
    __syncthreads();  // wsum is rewritten by the next round
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off, kWave));
  if (lane == 0) wmax[wv] = mx;
  __syncthreads();
  if (t == 0) {
    uint32_t m = f_max;
    for (int k = 0; k < kScanThreads / kWave; ++k) m = max(m, wmax[k]);
    A.pair_offset[A.n_pairs] = (int64_t)carry;
    if (A.host_counts) A.host_counts[A.n_pairs] = f_err;
    if (A.host) {
      // the call's last flag writes: its words go to the host and are cleared for the slot's
      // next call (the pool counter included: every record of the range is in the pool)
      A.host[kFlagErr] = f_err;
      A.host[kFlagMax] = m;
      A.host[kFlagTotal] = (uint32_t)carry;
      A.host[kFlagTotal + 1] = (uint32_t)(carry >> 32);
#pragma unroll
      for (int k = 0; k < kFlagWords; ++k)
        __hip_atomic_store(A.flags + k, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      __hip_atomic_store(A.flags + kFlagMax, m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store((uint64_t*)(A.flags + kFlagTotal), carry, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      // every record of the range is in the pool: a next range reserves from 0
      __hip_atomic_store((uint64_t*)(A.flags + kFlagPool), 0ull, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// A tile's count from its status word, at most the 64 parents a tile holds.
__device__ __forceinline__ uint32_t status_count(uint64_t w) {
  return min((uint32_t)(w & ((1u << kStatusCountBits) - 1u)), (uint32_t)(kTile / 4));
}

// Inclusive scan of a per-lane count c < 128 over the wave, bit-sliced: the counts of the lanes
// below are the sum over bits b of 2^b times the number of lanes below with bit b set (mbcnt).
__device__ __forceinline__ uint32_t wave_incl_scan7(uint32_t c) {
  uint32_t incl = c;
#pragma unroll
  for (int b = 0; b < 7; ++b) incl += mbcnt64(ballot((c >> b) & 1u)) << b;
  return incl;
}

// Moves the records of one group of up to 64 tiles (lane l holds tile l's status word w and count
// c, incl their inclusive scan): the group's rank q (the pair's rank at + q) goes from its tile's
// pool segment to base + at + q, in batches of 64 ranks, lane l moving the batch's l-th record.
__device__ __forceinline__ void move_group(const MoveArgs& A, uint64_t w, uint32_t c, uint32_t incl,
                                           int64_t base, uint32_t at, uint32_t count,
                                           uint32_t lane) {
  const uint32_t total = __builtin_amdgcn_readlane(incl, kWave - 1);
  const uint64_t has = ballot(c != 0u);
  for (uint32_t b = 0; b < total; b += kWave) {
    const uint32_t q = b + lane;
    uint64_t src = ~0ull;
    for (uint64_t m = has; m != 0ull; m &= m - 1ull) {
      const uint32_t i = (uint32_t)__builtin_ctzll(m);
      const uint32_t hi = __builtin_amdgcn_readlane(incl, i);
      const uint32_t lo = hi - __builtin_amdgcn_readlane(c, i);
      if (q >= lo && q < hi) {
        const uint64_t wi = read_lane64(w, i);
        src = (wi >> kStatusCountBits) + (q - lo);
      }
    }
    const int64_t dst = base + at + q;
    if (q < total && at + q < count && src < (uint64_t)A.cap && dst < A.cap) {
      A.parent[dst] = A.pool_parent[src];
      reinterpret_cast<float4*>(A.w4)[dst] = reinterpret_cast<const float4*>(A.pool_w4)[src];
    }
  }
}

// Visits the marked groups of a long range in increasing order, clearing the pair's marks: f(g) for
// each group g whose bit is set in the pair's nz words.
template <typename F>
__device__ __forceinline__ void for_marked_groups(const MoveArgs& A, uint32_t pair, uint32_t lane,
                                                  F&& f) {
  const uint32_t n_groups = (A.tiles + kWave - 1) / kWave;
  uint64_t* words = A.nz + (int64_t)pair * A.nz_words;
  for (uint32_t w0 = 0; w0 < A.nz_words; w0 += kWave) {
    const bool mine = w0 + lane < A.nz_words;
    const uint64_t bits = mine ? words[w0 + lane] : 0ull;
    if (mine && bits != 0ull) words[w0 + lane] = 0ull;
    for (uint64_t lanes = ballot(bits != 0ull); lanes != 0ull; lanes &= lanes - 1ull) {
      const uint32_t i = (uint32_t)__builtin_ctzll(lanes);
      uint64_t bw = read_lane64(bits, i);
      for (; bw != 0ull; bw &= bw - 1ull) {
        const uint32_t g = (w0 + i) * kWave + (uint32_t)__builtin_ctzll(bw);
        if (g < n_groups) f(g);
      }
    }
  }
}

// Each wave takes pairs wave, wave + n_waves, ...: the pair's count and offset from k_scan, then
// its tiles' records group by group (a range of at most two groups reads both groups' status
// words at once; a longer one visits only its marked groups).
constexpr int kMoveWaves = 4;

__global__ void __launch_bounds__(kMoveWaves * kWave) k_move(MoveArgs A) {
  const uint32_t lane = lane_id();
  const uint32_t n_waves = gridDim.x * kMoveWaves;
  const uint32_t n_groups = (A.tiles + kWave - 1) / kWave;
  const uint32_t first = __builtin_amdgcn_readfirstlane(blockIdx.x * kMoveWaves + threadIdx.x / kWave);
  // A pair's loads are issued together, before any of them is used: its skip mark (read from a
  // valid stand-in address when the call skips no pair), count and offset, and for a short range
  // its status words (read even when the pair has no records: they lie inside the status table).
  auto skipped = [&](uint32_t pair) -> const uint8_t* {
    return A.skip != nullptr ? A.skip + pair : (const uint8_t*)(A.pair_count + pair);
  };
  if (n_groups <= kNzMinGroups) {
    for (uint32_t pair = first; pair < A.n_pairs; pair += n_waves) {
      const uint64_t* row = A.status + (int64_t)pair * A.tiles;
      const uint8_t sv = *skipped(pair);
      const int64_t count64 = A.pair_count[pair];
      const int64_t base = A.pair_offset[pair];
      const uint64_t w0 = lane < A.tiles ? row[lane] : 0ull;
      const uint64_t w1 = n_groups > 1 && kWave + lane < A.tiles ? row[kWave + lane] : 0ull;
      const uint32_t count = (uint32_t)min(count64, (int64_t)0xFFFFFFFFll);
      if ((A.skip != nullptr && sv != 0) || count == 0u) continue;  // no records
      const uint32_t c0 = status_count(w0), c1 = status_count(w1);
      const uint32_t incl0 = wave_incl_scan7(c0), incl1 = wave_incl_scan7(c1);
      move_group(A, w0, c0, incl0, base, 0u, count, lane);
      if (n_groups > 1)
        move_group(A, w1, c1, incl1, base, __builtin_amdgcn_readlane(incl0, kWave - 1), count,
                   lane);
    }
    return;
  }
  for (uint32_t pair = first; pair < A.n_pairs; pair += n_waves) {
    const uint8_t sv = *skipped(pair);
    const int64_t count64 = A.pair_count[pair];
    const int64_t base = A.pair_offset[pair];
    // (the count and offset are used before the skip test, so that their loads go out with the
    // mark's instead of after the branch)
    asm volatile("" ::"v"(count64), "v"(base));
    if (A.skip != nullptr && sv != 0) continue;  // no records, no marks
    const uint32_t count = (uint32_t)min(count64, (int64_t)0xFFFFFFFFll);
    const uint64_t* row = A.status + (int64_t)pair * A.tiles;
    uint32_t at = 0;
    for_marked_groups(A, pair, lane, [&](uint32_t g) {
      if (count == 0u) return;
      const uint32_t t = g * kWave + lane;
      const uint64_t w = t < A.tiles ? row[t] : 0ull;
      const uint32_t c = status_count(w);
      const uint32_t incl = wave_incl_scan7(c);
      move_group(A, w, c, incl, base, at, count, lane);
      at += __builtin_amdgcn_readlane(incl, kWave - 1);
    });
  }
}

// The interpreting discover kernel: one launch covers every part of a call.
template <int MODE>
__global__ void __launch_bounds__(kDiscoverThreads)
    k_discover(const uint32_t* __restrict__ geo, const uint32_t* __restrict__ blob,
               const Group* __restrict__ groups,
               const float* __restrict__ bias_tab, uint64_t* __restrict__ status,
               uint32_t* __restrict__ err, float* __restrict__ raw, DiscoverScalars a) {
  discover_body<MODE, false>(geo, blob, groups, bias_tab, status, err, raw, a, 0ull);
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
                     a->n_sources, a->blob_words, a->bias_floats);
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
  const uint64_t waves = (uint64_t)emr::kDiscoverWaves * (uint64_t)per_cu * (uint64_t)cus;
  uint32_t target = 0;
  for (uint32_t c : {emr::kChunkTilesMax, 8u, 4u})
    if (target == 0 && groups * ((a->tiles + c - 1) / c) >= 4ull * waves) target = c;
  emr::DiscoverScalars sc{};
  sc.cap = a->cap;
  sc.n_pos = a->n_pos;
  sc.tile_lo = a->tile_lo;
  sc.tiles = a->tiles;
  sc.n_parts = a->n_parts;
  uint64_t chunks = 0;
  for (uint32_t k = 0; k < a->n_parts; ++k) {
    const int S = (int)a->part_S[k], W = (int)a->part_W[k];
    const uint32_t tpw = (uint32_t)emr::positions_per_lane(S, W) / emr::kTileIters;
    uint32_t chunk = target > tpw ? target : tpw;  // at most kChunkTilesMax (tpw <= 4)
    if (a->part_chunk[k] != 0u) {
      chunk = a->part_chunk[k];
      if (chunk < tpw || chunk > emr::kChunkTilesMax || (chunk & (chunk - 1u)) != 0u)
        return hipErrorInvalidValue;
    }
    const uint32_t cpg = (a->tiles + chunk - 1) / chunk;
    // (a part's chunk index fits a list entry's index field)
    if ((uint64_t)a->part_groups[k] * cpg >= (1ull << emr::kEntryPartShift))
      return hipErrorInvalidValue;
    sc.part[k] = emr::DiscoverPart{(uint32_t)S, (uint32_t)W, a->part_group0[k],
                                   a->part_groups[k] * cpg, cpg, chunk};
    chunks += (uint64_t)a->part_groups[k] * cpg;
  }
  // (a workgroup's chunk index then stays below 2^32 when it steps past its last chunk)
  if (chunks > 0x7FFFFFFFull) return hipErrorInvalidValue;
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
  sc.pool_ctr = (uint64_t*)(a->err + emr::kFlagPool);
  sc.pool_parent = a->pool_parent;
  sc.pool_w4 = a->pool_w4;
  sc.pair_total = a->pair_total;
  // Clamp the grid to what can be resident at once (the waves take their chunks; none waits for
  // another), and to one workgroup per chunk (few chunks: spread over as many CUs).
  const uint32_t resident = (uint32_t)per_cu * (uint32_t)cus;
  if (blocks > chunks) blocks = (uint32_t)chunks;
  if (blocks > resident) blocks = resident;
  // A schedule is made for one grid: it must be this launch's. (Only the compiled tier's
  // kernels read it; the interpreter's launcher refuses one.)
  if (a->sched != nullptr) {
    if (a->sched_lists != blocks || a->sched_stride == 0u || a->sched_stride % emr::kWave != 0u ||
        a->sched_stride > emr::kListLds)
      return hipErrorInvalidValue;
    sc.sched = a->sched;
    sc.sched_stride = a->sched_stride;
    sc.sched_lists = a->sched_lists;
  }
  *out = sc;
  *grid = blocks;
  return hipSuccess;
}

// Workgroups of the interpreter's discover kernel (mode 0 raw, 1 records) that fit on one CU.
extern "C" int emr_discover_per_cu(int mode) {
  auto occ = [](auto kern) {
    int n = 0;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, emr::kDiscoverThreads, 0) ==
                   hipSuccess &&
               n > 0
               ? n
               : 1;
  };
  static const int per_cu[2] = {occ(emr::k_discover<emr::kModeRaw>),
                                occ(emr::k_discover<emr::kModeRecords>)};
  return per_cu[mode == emr::kModeRecords ? 1 : 0];
}

template <int MODE>
static hipError_t launch_discover_t(const emr::DiscoverArgs* a, uint32_t blocks, hipStream_t s,
                                    hipEvent_t start, hipEvent_t stop) {
  auto kern = emr::k_discover<MODE>;
  if (a->sched != nullptr) return hipErrorInvalidValue;  // the interpreter runs round-robin
  int dev = 0, cus = 0;
  hipError_t e;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
    return e;
  const int per_cu = emr_discover_per_cu(MODE);
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
  float* raw = a->raw;
  if (start && (e = hipEventRecord(start, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(emr::kDiscoverThreads), 0, s, geo, blob, grp, bias_tab, status, err, raw,
                     sc);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return stop ? hipEventRecord(stop, s) : hipSuccess;
}

// One launch for all the parts (sources per walk and register window) listed in *a. blocks: the
// most 256-thread workgroups (4 waves each) to launch; the launch uses at most one wave per chunk
// of tiles and no more workgroups than can be resident at once; every wave walks its share of the
// chunks. start, stop: events recorded on s around the launch, or NULL.
// mode: 0 raw outputs, 1 records to the pool (then emr_launch_compact).
extern "C" hipError_t emr_launch_discover(const emr::DiscoverArgs* a, int mode, uint32_t blocks,
                                          hipStream_t s, hipEvent_t start, hipEvent_t stop) {
  switch (mode) {
    case emr::kModeRaw: return launch_discover_t<emr::kModeRaw>(a, blocks, s, start, stop);
    case emr::kModeRecords: return launch_discover_t<emr::kModeRecords>(a, blocks, s, start, stop);
    default: return hipErrorInvalidValue;
  }
}

// Offsets of a CSR output from per-pair (or per-genome) totals, one workgroup.
extern "C" hipError_t emr_launch_scan(const emr::ScanArgs* S, hipStream_t s) {
  hipLaunchKernelGGL(emr::k_scan, dim3(1), dim3(emr::kScanThreads), 0, s, *S);
  return hipGetLastError();
}

// The compaction of one record-mode range (after its discover launch, on the same stream): the
// pairs' offsets, then the records' move.
extern "C" hipError_t emr_launch_compact(const emr::ScanArgs* S, const emr::MoveArgs* M,
                                         hipStream_t s) {
  if (S->n_pairs == 0) return hipSuccess;
  hipLaunchKernelGGL(emr::k_scan, dim3(1), dim3(emr::kScanThreads), 0, s, *S);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  uint32_t blocks = (M->n_pairs + emr::kMoveWaves - 1) / emr::kMoveWaves;
  if (blocks > 8192) blocks = 8192;  // waves loop over pairs beyond this
  hipLaunchKernelGGL(emr::k_move, dim3(blocks), dim3(emr::kMoveWaves * emr::kWave), 0, s, *M);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_finalize(uint32_t* flags, uint32_t* host, hipStream_t s) {
  hipLaunchKernelGGL(emr::k_finalize, dim3(1), dim3(64), 0, s, flags, host);
  return hipGetLastError();
}
