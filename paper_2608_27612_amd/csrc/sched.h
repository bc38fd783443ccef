// Static balancing of a discover launch's chunks over its waves (sched.cpp).
#pragma once
#include <stdint.h>

#include <vector>

namespace emr {

// Longest-processing-time-first list scheduling of n chunks of estimated cost cost[c] over
// `waves` waves, in two levels when domains > 1:
//  - the waves form `domains` domains: wave w belongs to domain (w / domain_waves) % domains;
//  - chunks with the same key[c] (< n_keys) all go to one domain: keys in order of decreasing
//    total cost (equal totals by key), each to the domain with the least load per wave so far
//    (equal: the lowest domain); when a key holds more than a tenth of a domain's mean load (few
//    keys), the domains could not be balanced and all waves form one domain instead;
//  - within a domain (or over all waves when domains <= 1), chunks in order of decreasing cost
//    (equal costs by index), each to the wave with the least load so far (equal: the lowest wave).
// The result is a table of `waves` rows of *stride entries (stride a multiple of 64, at least 64):
// row w lists wave w's chunks in the order they were assigned (costliest first), then kNoChunk.
// Every chunk appears exactly once. Within a domain the greedy rule keeps every wave's load within
// the domain's mean load per wave plus its largest chunk.
// Returns false (and leaves *table empty) for waves == 0, a negative or non-finite cost, a key
// >= n_keys, domains > 1 without keys, or more domains than waves / domain_waves can fill.
bool lpt_schedule(const float* cost, const uint32_t* key, uint32_t n_keys, uint32_t n,
                  uint32_t waves, uint32_t domain_waves, uint32_t domains,
                  std::vector<uint32_t>* table, uint32_t* stride);

}  // namespace emr

// The same through a C ABI, for host tests: writes the table when table_cap (entries) holds it.
// Returns 0 on success, 1 when the table does not fit (*stride still set), -1 on invalid input.
extern "C" int emr_lpt_schedule(const float* cost, const uint32_t* key, uint32_t n_keys,
                                uint32_t n, uint32_t waves, uint32_t domain_waves,
                                uint32_t domains, uint32_t* table, uint64_t table_cap,
                                uint32_t* stride);
