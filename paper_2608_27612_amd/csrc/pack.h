// Host-side genome packer (see pack.cpp).
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/emr.h"
#include "emr_internal.h"

namespace emr {

// What the packer learned about one (genome, direction) program.
struct GenomeInfo {
  int n_steps = 0;       // varying nodes evaluated per query
  int fma_xy = 0;        // edges from the position's x / y
  int fma_node = 0;      // edges between varying nodes
  int act_count[6] = {0, 0, 0, 0, 0, 0};  // varying nodes per activation id
  // The part of the above in nodes whose value does not depend on the source (kRecShared)
  int shared_edges = 0;  // their edges from x / y and from varying nodes
  int shared_act_count[6] = {0, 0, 0, 0, 0, 0};
  int window = 0;        // register slots needed
  int n_unodes = 0;      // uniform computed nodes
  int n_rec = 0;         // program records
  bool out_varying = false;
};

// Validates genome g and appends its two direction programs to `blob`. On failure returns false
// with *st / *msg set and leaves `blob` partially written (the caller discards it).
bool pack_genome(const emr_genome& g, std::vector<uint32_t>& blob, ProgDesc desc[2],
                 GenomeInfo info[2], emr_status* st, std::string* msg);

}  // namespace emr
