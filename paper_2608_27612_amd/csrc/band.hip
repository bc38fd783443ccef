// gfx950 kernel of ES-HyperNEAT's band values of expressed connections (the band threshold that
// Theorem 1 names beside the variance threshold; ES-HyperNEAT's pruning step defines it): for
// connection (pair, cell C, weight w), the pair's CPPN at the four same-level neighbour centres
// of C, one cell side d away along x and y, and band = max(min(|w - left|, |w - right|),
// min(|w - down|, |w - up|)). One wave per pair: its program runs through the interpreter's record
// step (one source per walk), each lane holding P / 4 connections and their 4 neighbours each.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/emr.h"
#include "band.h"
#include "discover.h"
#include "emr_internal.h"

namespace emr {

// The walks of one pair over its connections [lo, hi): connection i = b + 64 k + lane holds
// instances 4k .. 4k + 3 (left, right, down, up).
template <int W>
__device__ __forceinline__ void band_walks(const BandArgs& A, const BandPair& bp, int64_t lo,
                                           int64_t hi, uint32_t lane) {
  constexpr int P = positions_per_lane(1, W);
  constexpr int C = P / 4;
  const int64_t n_pos = n_positions(A.depth);
  for (int64_t b = lo; b < hi; b += (int64_t)kWave * C) {
    float px[P], py[P], wc[C];
    bool live[C];
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int64_t i = b + (int64_t)k * kWave + lane;
      live[k] = i < hi;
      uint32_t F = live[k] ? A.conn_cell[i] : 1u;
      wc[k] = live[k] ? A.conn_w[i] : 0.0f;
      if (F == 0u || (int64_t)F > n_pos) {  // not a cell of this grid
        if (live[k]) atomicOr(A.err, kErrTable);
        live[k] = false;
        F = 1u;
      }
      // Eq. 1: the centre of grid position F - 1 (level l, Morton index m), side d = 2^(1-l)
      const uint32_t p = F - 1u;
      const int l = level_of(p);
      const uint32_t m = p - (uint32_t)level_offset(l);
      const float sc = pow2_neg(l);
      const float x = __builtin_fmaf((float)(2u * compact_even(m) + 1u), sc, -1.0f);
      const float y = __builtin_fmaf((float)(2u * compact_even(m >> 1) + 1u), sc, -1.0f);
      const float d = 2.0f * sc;
      px[4 * k + 0] = x - d;
      py[4 * k + 0] = y;
      px[4 * k + 1] = x + d;
      py[4 * k + 1] = y;
      px[4 * k + 2] = x;
      py[4 * k + 2] = y - d;
      px[4 * k + 3] = x;
      py[4 * k + 3] = y + d;
    }
    Walker<1, P, W> R;
    R.def();
    R.walk((uint64_t)(A.blob + bp.var_off), (uint64_t)(A.bias + bp.bias_base), bp.n_rec, px, py);
#pragma unroll
    for (int k = 0; k < C; ++k) {
      if (!live[k]) continue;
      const float* a = R.acc + 4 * k;
      const float dl = __builtin_fabsf(wc[k] - a[0]), dr = __builtin_fabsf(wc[k] - a[1]);
      const float dd = __builtin_fabsf(wc[k] - a[2]), du = __builtin_fabsf(wc[k] - a[3]);
      A.band[b + (int64_t)k * kWave + lane] =
          __builtin_fmaxf(__builtin_fminf(dl, dr), __builtin_fminf(dd, du));
    }
  }
}

__global__ void __launch_bounds__(256) k_band(BandArgs A) {
  const uint32_t lane = lane_id();
  for (uint32_t pair = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / kWave) +
                                                      threadIdx.x / kWave);
       pair < A.n_pairs; pair += gridDim.x * (blockDim.x / kWave)) {
    const BandPair bp = A.pairs[pair];
    // The pair's records, rows and window must lie inside their tables (the walk reads one record
    // and one row past the last, and a row as four floats).
    const uint32_t rec_words = kRecWords * (bp.n_rec + 1), row_floats = 4u * (bp.n_rec + 2);
    const bool ok = bp.n_rec <= kMaxRecords && (bp.var_off & (kRecWords - 1)) == 0 &&
                    rec_words <= A.blob_words && bp.var_off <= A.blob_words - rec_words &&
                    row_floats <= A.bias_floats && bp.bias_base <= A.bias_floats - row_floats &&
                    (bp.window == 4u || bp.window == 8u || bp.window == 16u || bp.window == 32u);
    if (!ok) {
      if (lane == 0) atomicOr(A.err, kErrTable);
      continue;
    }
    int64_t lo = A.conn_offset[pair], hi = A.conn_offset[pair + 1];
    lo = lo < 0 ? 0 : (lo > A.cap ? A.cap : lo);
    hi = hi > A.cap ? A.cap : (hi < lo ? lo : hi);
    switch (bp.window) {
      case 4u: band_walks<4>(A, bp, lo, hi, lane); break;
      case 8u: band_walks<8>(A, bp, lo, hi, lane); break;
      case 16u: band_walks<16>(A, bp, lo, hi, lane); break;
      default: band_walks<32>(A, bp, lo, hi, lane); break;
    }
  }
}

}  // namespace emr

extern "C" hipError_t emr_launch_band(const emr::BandArgs* A, hipStream_t s) {
  uint32_t b = (A->n_pairs + 3) / 4;
  b = b == 0 ? 1 : (b > 8192 ? 8192 : b);
  hipLaunchKernelGGL(emr::k_band, dim3(b), dim3(256), 0, s, *A);
  return hipGetLastError();
}
