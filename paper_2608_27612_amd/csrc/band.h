// Arguments of the band kernels (band.hip: the band values; phase2.hip: the band filter), shared
// with their host side (runtime.cpp).
#pragma once
#include <stdint.h>

namespace emr {

// One pair's program as the band kernel walks it (16 bytes per pair, built by the host from the
// plan's groups): the varying program's records, its register window, and the pair's bias rows
// (the group's rows shifted to the pair's slot, so that slot 0 of each row is the pair's).
struct BandPair {
  uint32_t var_off;    // word offset of the record stream in the population's program words
  uint32_t n_rec;      // records (0: the output does not depend on the position: row 0 holds it)
  uint32_t window;     // register window (4, 8, 16, 32); 0: no group holds the pair (error)
  uint32_t bias_base;  // float offset of the pair's row 0 in the bias table
};

struct BandArgs {
  const uint32_t* blob;        // the population's program words
  const float* bias;           // the plan's bias rows
  const BandPair* pairs;       // [n_pairs]
  const int64_t* conn_offset;  // [n_pairs + 1]
  const uint32_t* conn_cell;   // heap cells
  const float* conn_w;
  float* band;                 // [connections]
  uint32_t* err;               // error word of the call's flag slot
  int64_t cap;                 // connections the buffers hold
  uint32_t n_pairs;
  int32_t depth;
  uint32_t blob_words;
  uint32_t bias_floats;        // floats of the bias table, padding included
};

struct BandSelectArgs {
  const int64_t* in_offset;  // [n_pairs + 1]
  const uint32_t* in_cell;
  const float* in_w;
  const float* band;
  int64_t in_cap;
  float theta_band;
  uint32_t* totals;           // [n_pairs]
  const int64_t* out_offset;  // [n_pairs + 1] from k_scan
  uint32_t* out_cell;
  float* out_w;
  int64_t out_cap;
  uint32_t n_pairs;
};

}  // namespace emr
