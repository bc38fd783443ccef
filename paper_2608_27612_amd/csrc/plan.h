// The host side of discovery (plan.cpp): a population's packed tables, a call's plan (groups of
// sources, buckets, the launch's parts, the table image the kernels read, the workspace layout)
// and a check of every offset the kernels take from those tables. Host only (no HIP): the test
// shim compiles it too.
#pragma once
#include <stdint.h>

#include <functional>
#include <string>
#include <vector>

#include "../../include/emr.h"
#include "emr_internal.h"
#include "pack.h"

namespace emr {

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Algorithmic VALU slots per query of one (genome, direction) program evaluated for S sources at
// once: one per position-dependent edge, the activation costs (transcendental instructions
// weighted by rT), and 2.5 for the variance and threshold share of a query; the nodes whose value
// does not depend on the source are evaluated once for the S sources, so each query counts 1 / S
// of their edges and activations.
// The cost is base + rT * trans: query_base() is the part without transcendentals, query_trans()
// their count per query. A program whose output does not depend on the position costs nothing
// per query: its output is the source's constant (folded once by the bind kernel, like every
// position-independent node) and the variance of a constant is exactly zero, so the kernels
// evaluate and test nothing for it.
double query_base(const GenomeInfo& inf, int S = 1);
double query_trans(const GenomeInfo& inf, int S = 1);
double query_slots(const GenomeInfo& inf, double rT, int S = 1);
// Useful floating-point operations per query: a multiply-add per position-dependent edge counts
// 2, every other activation operation and each transcendental 1, the variance 2.5 (shared nodes
// counted as above).
double query_flops(const GenomeInfo& inf, int S = 1);

// The register window bucket (4, 8, 16, 32) holding `window` live values, or -1.
int window_bucket(int window);

// Packs genomes 0 .. n - 1 as n_parts contiguous ranges, each into its own word vector (run(n_parts,
// f) calls f(t) for every part t, possibly in parallel), then concatenates the vectors (each
// padded to a record boundary) and moves each range's descriptors by its vector's base, with 16
// words of padding at the end (the kernels may read a few words past a program's end). On failure
// returns the lowest failing genome's status in *bad / *msg.
emr_status pack_genomes(int32_t n, const std::function<emr_genome(int32_t)>& genome_at,
                        int n_parts, const std::function<void(int, const std::function<void(int)>&)>& run,
                        std::vector<ProgDesc>* desc, std::vector<GenomeInfo>* info,
                        std::vector<uint32_t>* words, int32_t* bad, std::string* msg);

// The tables of one discover / raw-eval call, built on the host.
struct PlanTables {
  int depth = 0;
  int64_t n_pairs = 0;
  int64_t tiles = 0;
  int32_t n_genomes = 0;
  int32_t n_sources = 0;
  struct Bucket {
    int S, window;
    uint32_t first, count;
    double cost;  // summed per-query cost of its groups' programs (launch order)
    uint32_t varying;  // its first `varying` groups have a position-dependent output (the rest,
                       // the cheapest, do not)
  };
  // The discover launch of a call: its buckets (one per sources per walk and register window),
  // costliest first.
  struct Launch {
    int n_parts;
    int part[kMaxBuckets];  // bucket indices
    double cost;
    // per position of the range, over all the launch's queries: cost-model slots without
    // transcendentals, transcendental instructions, and queries (sources)
    double slots_base, slots_trans, sources;
  };
  std::vector<Group> groups;
  std::vector<Bucket> buckets;
  std::vector<Launch> launches;  // one (none without groups)
  std::vector<Member> members;
  std::vector<uint32_t> group_member0;  // index of each group's first member
  std::vector<float> src_xy;
  uint64_t bias_floats = 0;
  // Per group: cost-model slots of one query of one of its sources (the launch schedules' chunk
  // costs).
  std::vector<float> group_cost;
  // The tables' host image (groups at t_groups, members at t_members, source coordinates at
  // t_srcxy, one byte per pair at t_uniform: 1 when the pair's output does not depend on the
  // position; per pair at t_pairinfo: genome << 1 | dir, then the source index).
  std::vector<char> img;
  size_t t_groups = 0, t_members = 0, t_srcxy = 0, t_uniform = 0, t_pairinfo = 0;
  // What the plan was built for (exact copies, compared on reuse).
  std::vector<emr_source> key_sources;
  std::vector<int32_t> key_offs;
  bool key_has_offs = false;
  int32_t key_n_shared = 0;
  // Workspace layout (bytes from the workspace start): tile status words, the compaction's group
  // marks and per-pair record totals (cleared before each record call: clear_words words from
  // off_nz); then (total onwards) the record pool of a call's capacity.
  size_t off_status = 0;
  size_t total = 0;
  size_t status_bytes = 0;
  size_t off_nz = 0, nz_bytes = 0;
  size_t off_ptotal = 0;
  int64_t clear_words = 0;
  // Floats of a bias table: the groups' rows plus 16 floats of padding (the compiled tier loads a
  // group's rows 1 .. 4 at once).
  size_t bias_table_floats() const { return (size_t)bias_floats + 16; }
};

// Builds the tables of a call over a population's descriptors (desc/info: 2 per genome) for the
// sources (shared by every genome when offs is NULL, else genome g owns sources offs[g] ..
// offs[g + 1] - 1) at the given depth. EMR_E_INVAL / EMR_E_LIMIT with *msg on bad arguments or
// sizes beyond the tables' index ranges.
emr_status build_plan_tables(const ProgDesc* desc, const GenomeInfo* info, int32_t n_genomes,
                             const emr_source* sources, int32_t n_sources, const int32_t* offs,
                             int32_t n_shared, int32_t depth, PlanTables* P, std::string* msg);

// Every offset, count and index the kernels take from the tables of P (groups, members, pair
// records, the uniform marks, the bias rows, the population's descriptors and program words of
// blob_words words) lies inside its table, every pair is one group member's, and the workspace
// regions follow each other without overlap. False with *msg naming the first violation.
bool check_plan_tables(const PlanTables& P, const ProgDesc* desc, uint64_t blob_words,
                       std::string* msg);

}  // namespace emr
