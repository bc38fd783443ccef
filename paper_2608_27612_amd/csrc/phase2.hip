// gfx950 kernels that work on the CSR output of a discover call.
//
//   hidden nodes (Section 2, Phase 1 feeding Phase 2): per genome, the children of the kept cells of
//     its outgoing pairs as a bitmap over grid positions (a parent's four children are one aligned
//     nibble), counted, offset by k_scan and emitted in ascending heap order as outgoing sources at
//     their cell centres (Eq. 1);
//   connections (Section 4's types, Section 3.3's weight filter): each child of a kept parent as a
//     connection, kept by its type and weight magnitude;
//   Eq. 2 read literally: a record stays when every ancestor of its cell is a record of the pair;
//   the band filter: the connections whose band value (band.hip) exceeds a threshold.
// Each output is CSR (k_scan in kernels.hip turns per-pair or per-genome totals into offsets).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/emr.h"
#include "band.h"
#include "discover.h"
#include "emr_internal.h"

namespace emr {

// Centre of grid position p (heap cell p + 1), Eq. 1: level l, Morton index within the level.
__device__ __forceinline__ void cell_centre(uint32_t p, float* x, float* y) {
  const int l = level_of(p);
  const uint32_t m = p - (uint32_t)level_offset(l);
  const float sc = pow2_neg(l);
  *x = __builtin_fmaf((float)(2u * compact_even(m) + 1u), sc, -1.0f);
  *y = __builtin_fmaf((float)(2u * compact_even(m >> 1) + 1u), sc, -1.0f);
}

// Each wave takes pairs wave, wave + n_waves, ...
#define FOR_EACH_PAIR_WAVE(pair, n)                                                              \
  for (uint32_t pair = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / kWave) +        \
                                                      threadIdx.x / kWave);                      \
       pair < (n); pair += gridDim.x * (blockDim.x / kWave))

// The pair's records [lo, hi) within the buffers' capacity.
__device__ __forceinline__ void pair_range(const RecordsIn& R, uint32_t pair, int64_t* lo,
                                           int64_t* hi) {
  const int64_t off = R.offset[pair], cnt = R.count[pair];
  *lo = off < 0 ? 0 : (off > R.cap ? R.cap : off);
  const int64_t end = off + (cnt < 0 ? 0 : cnt);
  *hi = end > R.cap ? R.cap : (end < *lo ? *lo : end);
}

// ------------------------------------------------------------------------ hidden nodes
// The call's records in parallel (a pair's records can number from none to hundreds of
// thousands, so they are spread by record, not by pair): wave w takes the records
// [w kMarkSpan, (w + 1) kMarkSpan) and lane l the records w kMarkSpan + l, + 64, ...; a record's
// pair is the last pair whose offset is at most the record's index (a binary search for the
// lane's first record, then a gallop forward from the pair before, the indices only growing).
// A record outside the range of the pair found (offsets out of order) marks nothing.
constexpr uint32_t kMarkSpan = 16 * kWave;

// The last q in [lo, hi) with off[q] <= r, given off[lo] <= r and (hi = n or off[hi] > r).
__device__ __forceinline__ uint32_t last_at_most(const int64_t* off, uint32_t lo, uint32_t hi,
                                                 int64_t r) {
  while (hi - lo > 1u) {
    const uint32_t mid = lo + (hi - lo) / 2u;
    if (off[mid] <= r)
      lo = mid;
    else
      hi = mid;
  }
  return lo;
}

__global__ void __launch_bounds__(256) k_hidden_mark(HiddenArgs A) {
  const uint32_t lane = lane_id();
  const int64_t Q = n_parents(A.rec.depth);
  const uint32_t np = A.rec.n_pairs;
  if (np == 0u) return;
  const int64_t* off = A.rec.offset;
  const int64_t total = min(max(off[np], (int64_t)0), A.rec.cap);  // the call's records held
  if (off[0] > 0) return;                                           // not a CSR offset table
  const int64_t n_waves = (int64_t)gridDim.x * (blockDim.x / kWave);
  for (int64_t base = (int64_t)(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave) * kMarkSpan;
       base < total; base += n_waves * kMarkSpan) {
    uint32_t p = 0u;
    bool first = true;
    for (uint32_t j = 0; j < kMarkSpan / kWave; ++j) {
      const int64_t r = base + (int64_t)j * kWave + lane;
      if (r >= total) break;
      if (first) {
        p = last_at_most(off, 0u, np, r);
        first = false;
      } else {
        // off[p] <= an earlier index < r: widen [p, hi) until off[hi] > r, then search it
        uint32_t lo = p, step = 1u, hi = p + 1u;
        while (hi < np && off[hi] <= r) {
          lo = hi;
          step = step < (1u << 30) ? 2u * step : step;
          hi = np - lo > step ? lo + step : np;
        }
        p = last_at_most(off, lo, hi, r);
      }
      int64_t lo_r, hi_r;
      pair_range(A.rec, p, &lo_r, &hi_r);
      if (r < lo_r || r >= hi_r) continue;
      const uint32_t info = A.rec.pair_info[2 * p];
      const uint32_t g = info >> 1;
      if ((info & 1u) != 0u || g >= A.n_genomes) continue;  // incoming pairs add no hidden node
      const uint32_t P = A.rec.parent[r];
      if ((int64_t)P >= Q) continue;
      // grid positions 4P .. 4P+3; the many pairs of one genome mostly mark cells already marked,
      // so a plain read first keeps them from queueing atomics on the same words
      uint32_t* bits = A.fresh + (int64_t)g * A.words;
      const uint32_t m = 0xFu << (4u * (P % 8u));
      if ((__hip_atomic_load(bits + P / 8u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & m) != m)
        atomicOr(bits + P / 8u, m);
    }
  }
}

// One workgroup per genome: its new cells (found now, not known before).
__global__ void __launch_bounds__(256) k_hidden_count(HiddenArgs A) {
  __shared__ uint32_t part[256 / kWave];
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const uint32_t* f = A.fresh + (int64_t)g * A.words;
    const uint32_t* k = A.known ? A.known + (int64_t)g * A.words : nullptr;
    uint32_t c = 0;
    for (int64_t w = threadIdx.x; w < A.words; w += blockDim.x)
      c += __builtin_popcount(f[w] & (k ? ~k[w] : ~0u));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) c += (uint32_t)__shfl_xor((int)c, off, kWave);
    if (lane_id() == 0) part[threadIdx.x / kWave] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t t = 0;
      for (int i = 0; i < 256 / kWave; ++i) t += part[i];
      A.totals[g] = t;
    }
    __syncthreads();
  }
}

// One workgroup per genome: thread t owns a contiguous run of bitmap words, so the genome's new
// cells come out in ascending order at offsets[g] + (cells of the runs before) + rank in the run;
// then the genome's known bits take the new cells.
__global__ void __launch_bounds__(256) k_hidden_emit(HiddenArgs A) {
  __shared__ uint32_t part[256];
  const int64_t n_pos = n_positions(A.rec.depth);
  const int64_t per = (A.words + 255) / 256;
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const uint32_t* f = A.fresh + (int64_t)g * A.words;
    uint32_t* k = A.known ? A.known + (int64_t)g * A.words : nullptr;
    const int64_t w0 = (int64_t)threadIdx.x * per;
    const int64_t w1 = w0 + per < A.words ? w0 + per : A.words;
    uint32_t c = 0;
    for (int64_t w = w0; w < w1; ++w) c += __builtin_popcount(f[w] & (k ? ~k[w] : ~0u));
    part[threadIdx.x] = c;
    __syncthreads();
    if (threadIdx.x == 0) {  // exclusive scan of the 256 runs
      uint32_t run = 0;
      for (int i = 0; i < 256; ++i) {
        const uint32_t v = part[i];
        part[i] = run;
        run += v;
      }
    }
    __syncthreads();
    int64_t at = A.offsets[g] + part[threadIdx.x];
    for (int64_t w = w0; w < w1; ++w) {
      const uint32_t kw = k ? k[w] : 0u;
      for (uint32_t b = f[w] & ~kw; b != 0u; b &= b - 1u) {
        const int64_t p = w * 32 + __builtin_ctz(b);
        if (p < n_pos && at < A.cap) {
          float x, y;
          cell_centre((uint32_t)p, &x, &y);
          A.out_src[3 * at] = __float_as_uint(x);
          A.out_src[3 * at + 1] = __float_as_uint(y);
          A.out_src[3 * at + 2] = (uint32_t)EMR_DIR_OUT;
          if (A.out_cell) A.out_cell[at] = (uint32_t)(p + 1);
        }
        ++at;
      }
      if (k) k[w] = kw | f[w];
    }
    __syncthreads();  // part is rewritten for the next genome
  }
}

// ------------------------------------------------------------------------ connections
// Type of a connection from (ax, ay) to (bx, by) (Section 4).
__device__ __forceinline__ uint32_t conn_type(float ax, float ay, float bx, float by) {
  if (ax == bx && ay == by) return EMR_CONN_SELF;
  if (ay < by) return EMR_CONN_FORWARD;
  if (ay > by) return EMR_CONN_BACKWARD;
  return EMR_CONN_LATERAL;
}

// Bit k of the result: child k of record i is an expressed connection of its pair.
__device__ __forceinline__ uint32_t expressed(const ExpressArgs& A, int64_t i, float sx, float sy,
                                              bool incoming) {
  const uint32_t P = A.rec.parent[i];
  if ((int64_t)P >= n_parents(A.rec.depth)) return 0u;
  const float4 w = reinterpret_cast<const float4*>(A.rec.w4)[i];
  const float wk[4] = {w.x, w.y, w.z, w.w};
  uint32_t m = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float cx, cy;
    cell_centre(4u * P + (uint32_t)k, &cx, &cy);
    const uint32_t t = incoming ? conn_type(cx, cy, sx, sy) : conn_type(sx, sy, cx, cy);
    if ((t & A.type_mask) != 0u && __builtin_fabsf(wk[k]) > A.w_min) m |= 1u << k;
  }
  return m;
}

// Sum over the wave of a per-lane count c < 8 (bit-sliced ballots).
__device__ __forceinline__ uint32_t wave_sum3(uint32_t c) {
  uint32_t t = 0;
#pragma unroll
  for (int b = 0; b < 3; ++b) t += popc64(ballot((c >> b) & 1u)) << b;
  return t;
}
__device__ __forceinline__ uint32_t wave_excl3(uint32_t c) {
  uint32_t t = 0;
#pragma unroll
  for (int b = 0; b < 3; ++b) t += mbcnt64(ballot((c >> b) & 1u)) << b;
  return t;
}

template <bool EMIT>
__global__ void __launch_bounds__(256) k_express(ExpressArgs A) {
  const uint32_t lane = lane_id();
  FOR_EACH_PAIR_WAVE(pair, A.rec.n_pairs) {
    const uint32_t info = A.rec.pair_info[2 * pair], j = A.rec.pair_info[2 * pair + 1];
    const float sx = A.rec.src_xy[2 * j], sy = A.rec.src_xy[2 * j + 1];
    int64_t lo, hi;
    pair_range(A.rec, pair, &lo, &hi);
    uint32_t total = 0;
    const int64_t base = EMIT ? A.out_offset[pair] : 0;
    for (int64_t b = lo; b < hi; b += kWave) {
      const int64_t i = b + lane;
      const uint32_t m = i < hi ? expressed(A, i, sx, sy, (info & 1u) != 0u) : 0u;
      const uint32_t c = (uint32_t)__builtin_popcount(m);
      if constexpr (EMIT) {
        int64_t at = base + total + wave_excl3(c);
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if ((m >> k) & 1u) {
            if (at < A.cap) {
              A.out_cell[at] = 4u * A.rec.parent[i] + 1u + (uint32_t)k;
              A.out_w[at] = A.rec.w4[4 * i + k];
            }
            ++at;
          }
      }
      total += wave_sum3(c);
    }
    if (!EMIT && lane == 0) A.totals[pair] = total;
  }
}

// ------------------------------------------------------------------------ band filter
// Per pair (one wave): the connections with band > theta_band (strict; a NaN band never passes),
// counted, then emitted in order at the pair's offset.
template <bool EMIT>
__global__ void __launch_bounds__(256) k_band_select(BandSelectArgs A) {
  const uint32_t lane = lane_id();
  FOR_EACH_PAIR_WAVE(pair, A.n_pairs) {
    int64_t lo = A.in_offset[pair], hi = A.in_offset[pair + 1];
    lo = lo < 0 ? 0 : (lo > A.in_cap ? A.in_cap : lo);
    hi = hi > A.in_cap ? A.in_cap : (hi < lo ? lo : hi);
    uint32_t total = 0;
    const int64_t base = EMIT ? A.out_offset[pair] : 0;
    for (int64_t b = lo; b < hi; b += kWave) {
      const int64_t i = b + lane;
      const bool keep = i < hi && A.band[i] > A.theta_band;
      const uint64_t m = ballot(keep);
      if constexpr (EMIT) {
        const int64_t at = base + total + mbcnt64(m);
        if (keep && at < A.out_cap) {
          A.out_cell[at] = A.in_cell[i];
          A.out_w[at] = A.in_w[i];
        }
      }
      total += popc64(m);
    }
    if (!EMIT && lane == 0) A.totals[pair] = total;
  }
}

// ------------------------------------------------------------------------ Eq. 2 chain rule
__global__ void __launch_bounds__(256) k_chain_mark(ChainArgs A) {
  const uint32_t lane = lane_id();
  const int64_t Q = n_parents(A.rec.depth);
  FOR_EACH_PAIR_WAVE(pair, A.rec.n_pairs) {
    int64_t lo, hi;
    pair_range(A.rec, pair, &lo, &hi);
    uint32_t* bits = A.member + (int64_t)pair * A.qwords;
    for (int64_t i = lo + lane; i < hi; i += kWave) {
      const uint32_t P = A.rec.parent[i];
      if ((int64_t)P < Q) atomicOr(bits + P / 32u, 1u << (P % 32u));
    }
  }
}

// Record i of a pair (member: the pair's bitmap) passes when every ancestor of its cell is a
// record of the pair (the root is its own ancestor line's start).
__device__ __forceinline__ bool chain_kept(const ChainArgs& A, const uint32_t* member, int64_t i) {
  uint32_t P = A.rec.parent[i];
  if ((int64_t)P >= n_parents(A.rec.depth)) return false;
  bool ok = true;
  while (P > 0u) {
    P = (P - 1u) / 4u;
    ok = ok && ((member[P / 32u] >> (P % 32u)) & 1u) != 0u;
  }
  return ok;
}

template <bool EMIT>
__global__ void __launch_bounds__(256) k_chain(ChainArgs A) {
  const uint32_t lane = lane_id();
  FOR_EACH_PAIR_WAVE(pair, A.rec.n_pairs) {
    int64_t lo, hi;
    pair_range(A.rec, pair, &lo, &hi);
    const uint32_t* member = A.member + (int64_t)pair * A.qwords;
    uint32_t total = 0;
    const int64_t base = EMIT ? A.out_offset[pair] : 0;
    for (int64_t b = lo; b < hi; b += kWave) {
      const int64_t i = b + lane;
      const bool keep = i < hi && chain_kept(A, member, i);
      const uint64_t kb = ballot(keep);
      if constexpr (EMIT) {
        const int64_t at = base + total + mbcnt64(kb);
        if (keep && at < A.cap) {
          A.out_parent[at] = A.rec.parent[i];
          reinterpret_cast<float4*>(A.out_w4)[at] = reinterpret_cast<const float4*>(A.rec.w4)[i];
        }
      }
      total += popc64(kb);
    }
    if (!EMIT && lane == 0) A.totals[pair] = total;
  }
}

}  // namespace emr

// ------------------------------------------------------------------------ launchers
static uint32_t wave_blocks(uint32_t n) {  // workgroups of 4 waves, one wave per item (capped)
  uint32_t b = (n + 3) / 4;
  return b == 0 ? 1 : (b > 8192 ? 8192 : b);
}

extern "C" hipError_t emr_launch_hidden(const emr::HiddenArgs* A, int step, hipStream_t s) {
  const uint32_t gb = A->n_genomes == 0 ? 1 : (A->n_genomes > 65535 ? 65535 : A->n_genomes);
  switch (step) {
    case 0: {
      // waves of kMarkSpan records over the records the buffers can hold (the waves loop when
      // there are more)
      const int64_t spans = (A->rec.cap + emr::kMarkSpan - 1) / emr::kMarkSpan;
      const uint32_t blocks = (uint32_t)std::min<int64_t>(std::max<int64_t>((spans + 3) / 4, 1), 2048);
      hipLaunchKernelGGL(emr::k_hidden_mark, dim3(blocks), dim3(256), 0, s, *A);
      break;
    }
    case 1: hipLaunchKernelGGL(emr::k_hidden_count, dim3(gb), dim3(256), 0, s, *A); break;
    case 2: hipLaunchKernelGGL(emr::k_hidden_emit, dim3(gb), dim3(256), 0, s, *A); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_express(const emr::ExpressArgs* A, int emit, hipStream_t s) {
  if (emit)
    hipLaunchKernelGGL(emr::k_express<true>, dim3(wave_blocks(A->rec.n_pairs)), dim3(256), 0, s, *A);
  else
    hipLaunchKernelGGL(emr::k_express<false>, dim3(wave_blocks(A->rec.n_pairs)), dim3(256), 0, s, *A);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_band_select(const emr::BandSelectArgs* A, int emit,
                                              hipStream_t s) {
  if (emit)
    hipLaunchKernelGGL(emr::k_band_select<true>, dim3(wave_blocks(A->n_pairs)), dim3(256), 0, s, *A);
  else
    hipLaunchKernelGGL(emr::k_band_select<false>, dim3(wave_blocks(A->n_pairs)), dim3(256), 0, s, *A);
  return hipGetLastError();
}

extern "C" hipError_t emr_launch_chain(const emr::ChainArgs* A, int step, hipStream_t s) {
  const dim3 grid(wave_blocks(A->rec.n_pairs));
  switch (step) {
    case 0: hipLaunchKernelGGL(emr::k_chain_mark, grid, dim3(256), 0, s, *A); break;
    case 1: hipLaunchKernelGGL(emr::k_chain<false>, grid, dim3(256), 0, s, *A); break;
    case 2: hipLaunchKernelGGL(emr::k_chain<true>, grid, dim3(256), 0, s, *A); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
