// Arguments of the network kernels (network.hip), shared with their host driver (networks.cpp).
//
// Numbering. Before pruning, genome g has raw nodes 0 .. n_sub - 1 (its substrate sources, in
// substrate order) and n_sub + i for the i-th set bit of its hidden-cell bitmap (ascending grid
// position); raw node j of genome g is entry raw_node[g] + j of the per-node arrays. Its raw edges
// (one per expressed connection of every phase, genome by genome, each genome's phases in order,
// each phase's pairs in order, each pair's connections in cell order) are entries
// raw_edge[g] .. raw_edge[g + 1] - 1 of eu/ev/ew, holding global raw node numbers raw_node[g] + j
// (kNoNode: the grid end is not a hidden node, the edge is dropped). After pruning, the kept nodes
// of genome g are renumbered in raw order (substrate nodes first, all kept) as entries
// node_offset[g] + k of the network arrays, and the kept edges are grouped by destination (CSR,
// in_offset), each group in raw order.
#pragma once
#include <stdint.h>

namespace emr {

constexpr uint32_t kNoNode = 0xFFFFFFFFu;
constexpr int kNetThreads = 256;

// Error bits of the network kernels.
constexpr uint32_t kNetErrIndex = 1u;   // an index outside its table (a host bug; never expected)

struct NetRankArgs {
  const uint32_t* known;  // [n_genomes * words] hidden-cell bitmaps
  uint32_t* rank;         // [n_genomes * words] set bits of the genome's earlier words
  uint32_t* hidden;       // [n_genomes] set bits per genome
  int64_t words;
  uint32_t n_genomes;
};

struct NetEdgeArgs {
  // one phase's expressed connections (CSR over its pairs)
  const int64_t* conn_offset;  // [n_pairs + 1]
  const uint32_t* conn_cell;
  const float* conn_w;
  int64_t n_pairs;
  int64_t total;               // conn_offset[n_pairs]
  // the phase's pairs: shared substrate sources (src_offsets == NULL: pair = g * n_sub + j) or
  // per-genome hidden sources (pair = source index, genome g owns src_offsets[g] .. [g + 1] - 1,
  // source r sits at heap cell src_cell[r])
  const int64_t* src_offsets;  // [n_genomes + 1] or NULL
  const uint32_t* src_cell;    // [n_sources] or NULL
  const uint8_t* sub_dir;      // [n_sub] 0: input (outgoing queries), 1: output (incoming)
  uint32_t n_sub;
  uint32_t n_genomes;
  const uint32_t* known;
  const uint32_t* rank;
  int64_t words;
  const int64_t* seg;          // [n_genomes] raw edge index of genome g's first edge of this phase
  const int64_t* raw_edge;     // [n_genomes + 1]
  const int64_t* raw_node;     // [n_genomes + 1]
  uint32_t* eu;                // [raw edges] global raw node numbers (raw_node[g] + local)
  uint32_t* ev;
  float* ew;
  uint32_t* err;
};

// Pruning. Flags per raw node (global numbering): reachable from an input (fwd), reaches an
// output (bwd); kept edges counted into their destination's in-degree.
struct NetFlagArgs {
  const uint8_t* sub_dir;
  const int64_t* raw_node;  // [n_genomes + 1]
  uint8_t* fwd;             // [raw nodes]
  uint8_t* bwd;             // [raw nodes]
  uint32_t* in_deg;         // [raw nodes] kept edges into the node
  uint32_t* kept_nodes;     // [n_genomes] kept hidden nodes (k_net_kept)
  uint32_t* kept_edges;     // [n_genomes] kept edges (k_net_kept)
  uint32_t n_sub;
  uint32_t n_genomes;
};

struct NetReachArgs {
  const uint32_t* eu;       // [raw edges] global raw node numbers, kNoNode: dropped
  const uint32_t* ev;
  uint8_t* fwd;
  uint8_t* bwd;
  uint32_t* in_deg;         // k_net_degree only
  uint32_t* changed;        // set to 1 by a pass that changed a flag (k_net_reach only)
  int64_t edges;            // raw edges
  int64_t nodes;            // raw nodes
};

struct NetNodeArgs {
  const uint32_t* known;
  const uint32_t* rank;
  int64_t words;
  const int64_t* raw_node;
  const uint8_t* fwd;
  const uint8_t* bwd;
  const uint32_t* in_deg;
  const int32_t* in_slot;      // [n_sub] input number of a substrate node, or -1
  const int64_t* node_offset;  // [n_genomes + 1] kept nodes
  const int64_t* edge_offset;  // [n_genomes + 1] kept edges
  uint32_t* gid;               // [raw nodes] kept node number (global), or kNoNode
  uint32_t* node_cell;         // [nodes] heap cell, kNoNode for substrate nodes
  int32_t* node_in;            // [nodes] input number of a substrate input node, else -1
  int64_t* in_offset;          // [nodes + 1]
  uint32_t* err;
  uint32_t n_sub;
  uint32_t n_genomes;
};

// The kept edges grouped by destination, each group in raw order: a stable sort of the raw edges
// by their destination's kept number (dropped edges get the key `sentinel` = nodes and sort
// last), then a gather of the sorted edges' sources and weights.
struct NetKeyArgs {
  const uint32_t* eu;
  const uint32_t* ev;
  const uint8_t* fwd;
  const uint8_t* bwd;
  const uint32_t* gid;
  uint32_t* key;            // [raw edges]
  uint32_t* val;            // [raw edges] the raw edge index
  int64_t edges;            // raw edges
  int64_t nodes;            // raw nodes
  uint32_t sentinel;        // kept nodes in all
  uint32_t* err;
};

struct NetGatherArgs {
  const uint32_t* key;      // sorted
  const uint32_t* val;      // sorted raw edge indices
  const uint32_t* eu;
  const float* ew;
  const uint32_t* gid;
  const int64_t* in_offset; // [nodes + 1]
  uint32_t* in_src;         // [edges] global node number of the source
  float* in_w;              // [edges]
  int64_t edges;            // kept edges
  int64_t raw_edges;
  int64_t raw_nodes;
  int64_t nodes;
  uint32_t* err;
};

// Synchronous activation over pattern blocks of 4 (one pattern per float4 component); state
// buffers [pblocks][nodes] of float4, swapped after each step.
struct NetStateArgs {
  const int32_t* node_in;   // [nodes]
  const float* patterns;    // [n_patterns * n_inputs]
  float* state;             // [pblocks * nodes * 4]
  int64_t nodes;
  uint32_t n_inputs;
  uint32_t n_patterns;
  uint32_t pblocks;
};

struct NetStepArgs {
  const int32_t* node_in;
  const int64_t* in_offset;
  const uint32_t* in_src;
  const float* in_w;
  const float* cur;
  float* nxt;
  int64_t nodes;
  uint32_t pblocks;
};

struct NetOutArgs {
  const int64_t* node_offset;  // [n_genomes + 1]
  const int32_t* out_node;     // [n_outputs] substrate index of output o
  const float* state;          // the final state
  const float* targets;        // [n_patterns] or NULL (fitness: one output, 4 patterns)
  float* outputs;              // [n_genomes * n_patterns * n_outputs] or NULL
  float* fitness;              // [n_genomes] or NULL
  int64_t nodes;
  uint32_t n_genomes;
  uint32_t n_outputs;
  uint32_t n_patterns;
  uint32_t pblocks;
};

}  // namespace emr
