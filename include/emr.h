/*
 * emr.h - C ABI of the MI355X (gfx950) eager multi-resolution substrate discovery library.
 *
 * The method (EMR-HyperNEAT, Phase 1): build the multiresolution grid of cell centres for every
 * level (Section 3.1, Eq. 1), query every (genome, source node, position) with the genome's CPPN in
 * one batched pass over a population (Section 3.1, the batched query W), then keep the four
 * children of every cell whose children's variance exceeds theta (Section 3.2, Eq. 2, and the
 * proof of the Superset Discovery theorem), compacting the survivors.
 *
 * General rules
 *   - Every call returns emr_status; nothing throws across the ABI. On failure a message is
 *     available from emr_last_error() (thread-local, owned by the library, valid until the calling
 *     thread's next call).
 *   - "host" pointers are ordinary CPU memory owned by the caller and only read during the call.
 *     "device" pointers are gfx950 global memory owned by the caller.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream). Device work is
 *     enqueued on it asynchronously unless the call says it synchronizes.
 *   - Argument and genome validation happens on the host before anything is enqueued; on such an
 *     error nothing is written.
 *
 * Depth convention: depth D counts levels below the root cell [-1,1]^2. Level l (1..D) has 4^l cells
 * of width 2/2^l centred at ((2i+1)/2^l - 1, (2j+1)/2^l - 1). The paper's depth d_p (Eq. 1 starts
 * with 4 cells at d = 0) is D - 1 here. The root is never queried; it is the parent of level 1.
 *
 * Cell numbering (heap order): the root is 0; the children of cell F are 4F+1 .. 4F+4; child k
 * (k = 0..3) lies on the +x side if bit 0 of k is set and on the +y side if bit 1 is set. Queried
 * positions are cells F = 1 .. N(D), stored at grid index p = F - 1. Parents are F = 0 .. Q(D)-1.
 *   N(D) = (4^(D+1) - 4) / 3 positions,  Q(D) = (4^D - 1) / 3 parents.
 */
#ifndef EMR_H
#define EMR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EMR_OK = 0,
  EMR_E_INVAL = -1,    /* bad argument */
  EMR_E_CYCLE = -2,    /* a genome's enabled edges contain a cycle */
  EMR_E_LIMIT = -3,    /* a genome or call exceeds a documented limit */
  EMR_E_NOMEM = -4,    /* host or device allocation failed */
  EMR_E_CAPACITY = -5, /* some pair found more records than the output region holds */
  EMR_E_DEVICE = -6,   /* a HIP runtime call failed, or no gfx950 device */
  EMR_E_ABORTED = -7,  /* a streaming sink asked to stop */
  EMR_E_IO = -8        /* a file could not be read or written */
} emr_status;

/* Message for the calling thread's last failed call ("" if none). */
const char* emr_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int32_t emr_version(void);

/* ------------------------------------------------------------------ genomes (Section 2) */

/* Activation ids. linear z; sigmoid 1/(1+e^-z); tanh z; gaussian e^(-z^2); sine sin z; abs |z|. */
enum { EMR_ACT_LINEAR = 0, EMR_ACT_SIGMOID = 1, EMR_ACT_TANH = 2, EMR_ACT_GAUSS = 3,
       EMR_ACT_SINE = 4, EMR_ACT_ABS = 5 };

/* Node kinds. The five input roles feed the CPPN tuple (x1, y1, x2, y2, 1) of Section 2. */
enum { EMR_IN_X1 = 0, EMR_IN_Y1 = 1, EMR_IN_X2 = 2, EMR_IN_Y2 = 3, EMR_IN_BIAS = 4,
       EMR_NODE_HIDDEN = 5, EMR_NODE_OUTPUT = 6 };

/* Query direction of a source node s at grid position p: outgoing evaluates CPPN(s, p), i.e.
 * (x1, y1) = s and (x2, y2) = p; incoming evaluates CPPN(p, s). */
enum { EMR_DIR_OUT = 0, EMR_DIR_IN = 1 };

/* One NEAT CPPN genome (host memory, caller-owned, read only during emr_pack_population).
 * A non-input node computes act(bias + sum of w * v_src over its enabled incoming edges).
 * Rules: exactly one output node; each input role at most once (a missing role contributes
 * nothing); edge endpoints in range; no edge into an input node; the enabled edges form a DAG. */
typedef struct {
  int32_t n_nodes, n_edges;
  const uint8_t* kind;    /* [n_nodes] EMR_IN_* / EMR_NODE_* */
  const uint8_t* act;     /* [n_nodes] EMR_ACT_*; ignored for input nodes */
  const float* bias;      /* [n_nodes] or NULL (all zero) */
  const int32_t* src;     /* [n_edges] node ids */
  const int32_t* dst;     /* [n_edges] node ids */
  const float* w;         /* [n_edges] */
  const uint8_t* enabled; /* [n_edges] or NULL (all enabled) */
} emr_genome;

/* A substrate source node (host memory). */
typedef struct {
  float x, y;
  int32_t dir; /* EMR_DIR_OUT or EMR_DIR_IN */
} emr_source;

/* ------------------------------------------------------------------ grid (Section 3.1, Eq. 1) */

/* N(D) positions and Q(D) parents for depth D (0 <= D <= EMR_MAX_DEPTH). Host only. */
#define EMR_MAX_DEPTH 15
emr_status emr_grid_count(int32_t depth, int64_t* n_positions, int64_t* n_parents);

/* Writes the centre of every queried position in heap order: xy_dev[2p], xy_dev[2p+1] for
 * p = 0 .. N(D)-1 (device, caller-owned, 2*N(D) floats). Coordinates are exact in fp32. */
emr_status emr_build_grids(int32_t depth, float* xy_dev, void* stream);

/* ------------------------------------------------------------------ packing (Section 3.1) */

/* Opaque, library-owned packed population: per genome, one program per query direction holding
 * only the nodes whose value varies with the grid position, in topological order, with register
 * slots assigned by liveness; plus the position-independent part, evaluated once per
 * (genome, source). Immutable after packing; may be used from several streams at once. */
typedef struct emr_population emr_population;

/* Limits of one genome after dead-node pruning. */
#define EMR_MAX_NODES 256   /* nodes in the genome as given */
#define EMR_MAX_EDGES 4096  /* edges in the genome as given */
#define EMR_MAX_LIVE 32     /* position-dependent values alive at once */

/* Validates and packs n genomes, then copies the tables to the current device (synchronously).
 * On a validation failure returns EMR_E_INVAL / EMR_E_CYCLE / EMR_E_LIMIT and sets *bad_index to
 * the first failing genome (else -1); *out is set only on success. */
emr_status emr_pack_population(const emr_genome* genomes, int32_t n, emr_population** out,
                               int32_t* bad_index);

/* The same for genomes given as concatenated arrays (host, caller-owned, read only during the
 * call): genome g has nodes node_off[g] .. node_off[g+1]-1 of kind/act/bias and edges
 * edge_off[g] .. edge_off[g+1]-1 of src/dst/w/enabled, node ids counted from the genome's first
 * node. node_off and edge_off have n+1 ascending entries starting at 0; bias and enabled may be
 * NULL (all 0, all enabled). Per-genome rules and errors as emr_pack_population. */
emr_status emr_pack_population_flat(int32_t n, const int64_t* node_off, const uint8_t* kind,
                                    const uint8_t* act, const float* bias, const int64_t* edge_off,
                                    const int32_t* src, const int32_t* dst, const float* w,
                                    const uint8_t* enabled, emr_population** out,
                                    int32_t* bad_index);
void emr_free_population(emr_population* pop);

/* Per-genome facts of a packed population (host arrays of n_genomes, any may be NULL):
 * varying steps and position-dependent edges per direction (index [2g + dir]) and the register
 * window the kernel needs. */
emr_status emr_population_info(const emr_population* pop, int32_t* n_genomes, int32_t* steps2,
                               int32_t* var_edges2, int32_t* window);

/* ------------------------------------------------------------------ discovery (Section 3.2) */

/* Pairs. With src_offsets == NULL every genome uses the same n_shared sources and
 * pair = g * n_shared + j. Otherwise src_offsets (host, [n_genomes+1], ascending, starting at 0)
 * gives genome g the sources src_offsets[g] .. src_offsets[g+1]-1 and pair = that source index. */

/* Output of emr_discover (device buffers, caller-owned): the kept cells of every pair, pairs back
 * to back in pair order (CSR). Record i of pair r, i < pair_count[r], is
 * parent[pair_offset[r] + i] (the heap index of a kept cell) and w4[4 * (pair_offset[r] + i) + k]
 * (the CPPN output at its child k), each pair's records in ascending parent order;
 * pair_offset[n_pairs] is the call's total. Counts and offsets are always exact; a total above
 * `capacity` is an overflow (reported by emr_result_check with the total, so a retry can size the
 * buffers), and then the records are not complete. Memory follows the kept cells: capacity is
 * the caller's choice (n_pairs * Q(D) can never overflow). */
typedef struct {
  uint32_t* parent;      /* [capacity] */
  float* w4;             /* [capacity * 4] */
  int64_t capacity;      /* records the buffers hold, 0 .. 2^32 - 1 */
  int64_t* pair_count;   /* [n_pairs] */
  int64_t* pair_offset;  /* [n_pairs + 1] */
  void* workspace;       /* device scratch, >= emr_workspace_bytes(..., capacity) bytes, aligned to
                            256 bytes */
  int64_t workspace_bytes;
} emr_result;

/* Device scratch (bytes) needed by an emr_discover call of this capacity (0 for emr_eval_raw) for
 * this population, these sources (host) and this depth: per-tile status words, the compaction's
 * tile-group marks and per-pair record totals, the folded per-(genome, source) biases, and a
 * record pool of `capacity` records (20 bytes each) that the discover kernel fills in any order
 * and the compaction gathers from. A call's error flags, largest count and total live in a
 * library-owned slot (see emr_result_check). A record call leaves the workspace's counters cleared,
 * and the next record call with the same workspace, plan (population, sources, depth), capacity
 * and stream does not clear them again: do not write into a workspace between calls (any other
 * call with it, or a change of any of those, makes the next call clear it first). EMR_E_INVAL for
 * a capacity outside [0, 2^32 - 1]. Host only. (The grouping
 * tables of a call live with the population: it keeps those of its last sources and depth on the
 * device, and a call with different ones replaces them.) */
emr_status emr_workspace_bytes(const emr_population* pop, const emr_source* sources,
                               int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                               int32_t depth, int64_t capacity, int64_t* bytes);

/*
 * Eager discovery: for every pair (genome g, source s) and every parent cell P (levels 0..D-1),
 * queries the CPPN of g at the four children of P, computes their population variance
 *   mu = ((w0+w1)+(w2+w3)) / 4,  var = ((d0^2+d1^2)+(d2^2+d3^2)) / 4,  d_k = w_k - mu,
 * and keeps P when var > theta (strict; NaN never kept). fp32 throughout.
 * `sources` is host memory (n_sources entries, n_sources = n_shared or src_offsets[n_genomes]).
 * Enqueued on `stream`; the host returns after staging small per-call tables.
 * The workspace must not be shared by calls that overlap in time. Calls with distinct workspaces
 * and outputs are independent (each takes its own flag slot; the population's tables and compiled
 * code are only read): several may be in flight at once, on one stream or on several, and a
 * caller can enqueue the next calls before checking the earlier ones with emr_result_check.
 */
emr_status emr_discover(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                        const int32_t* src_offsets, int32_t n_shared, int32_t depth, float theta,
                        const emr_result* out, void* stream);

/* Waits for the latest discover (or raw-output) call made with out's workspace on the current
 * device, then reports EMR_E_DEVICE if a kernel flagged an internal error, or EMR_E_CAPACITY if
 * the call found more records than out->capacity. *total (may be NULL) receives the records
 * found, *max_count (may be NULL) the largest pair count. `stream` is not used (the call's own
 * completion is waited for, not the stream's later work). A call's flags live in a library-owned
 * ring of 256 slots per device, written by the call's last kernel straight to pinned memory: a
 * result is checked before 255 further calls on its device, and EMR_E_INVAL reports a workspace
 * with no call to check. */
emr_status emr_result_check(const emr_result* out, int64_t* total, int64_t* max_count,
                            void* stream);

/* Waits for the latest call that wrote a CSR output through `workspace` on the current device
 * (emr_discover, emr_hidden_sources, emr_express, emr_chain_filter, emr_band_values,
 * emr_band_filter) and reports it like
 * emr_result_check: EMR_E_DEVICE for a kernel error, EMR_E_CAPACITY when it found more than
 * `capacity` entries; *total and *max_count (largest per pair or per genome; either may be NULL).
 * emr_result_check(out, ...) is emr_call_check(out->workspace, out->capacity, ...). */
emr_status emr_call_check(const void* workspace, int64_t capacity, int64_t* total,
                          int64_t* max_count, void* stream);

/* ------------------------------------------------------------------ after discovery
 * Operations on the checked CSR output `rec` of an emr_discover call, given the same population,
 * sources and depth as that call. Each writes a CSR output of its own through a workspace and is
 * checked with emr_call_check. */

/* Words of a per-genome cell bitmap at this depth: bit p of word p / 32 stands for grid position p
 * (heap cell p + 1), p < N(D). Host only. */
emr_status emr_cell_words(int32_t depth, int64_t* words);

/* Output of emr_hidden_sources (device buffers, caller-owned). */
typedef struct {
  emr_source* sources;  /* [capacity] outgoing sources at the hidden cells' centres, per genome in
                           ascending heap order */
  uint32_t* cell;       /* [capacity] their heap indices, or NULL */
  int64_t capacity;
  int64_t* offsets;     /* [n_genomes + 1]: genome g's are offsets[g] .. offsets[g+1]-1 */
  uint32_t* known;      /* [n_genomes * emr_cell_words(depth)] or NULL: cells already hidden nodes
                           (excluded from the output), or-ed with the output's cells by the call */
  void* workspace;      /* >= emr_hidden_workspace_bytes(...), 256-byte aligned */
  int64_t workspace_bytes;
} emr_hidden;

emr_status emr_hidden_workspace_bytes(int32_t n_genomes, int32_t depth, int64_t* bytes);

/*
 * The hidden nodes of a discovery (Section 2: Phase 1's discovered positions become the sources of
 * Phase 2, the hidden-to-hidden query; Section 4's recurrent substrates): per genome, the heap
 * cells 4P+1 .. 4P+4 of every kept parent P of its outgoing pairs, deduplicated, in ascending
 * order, minus the cells set in `known`; each is returned as an outgoing source at its cell centre
 * (Eq. 1, exact in fp32). Passing a phase's new nodes as the next emr_discover call's per-genome
 * sources (src_offsets from `offsets`), and `known` again to the next emr_hidden_sources call,
 * iterates Phase 2 until no genome finds a new node. Check with emr_call_check(workspace,
 * capacity): *total = the nodes found, *max_count = the most of one genome.
 */
emr_status emr_hidden_sources(const emr_population* pop, const emr_source* sources,
                              int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                              int32_t depth, const emr_result* rec, const emr_hidden* out,
                              void* stream);

/* Connection types (Section 4): forward y_s < y_t, backward y_s > y_t, lateral y_s = y_t, self
 * s = t (same position), for a connection from node s to node t. */
enum { EMR_CONN_FORWARD = 1, EMR_CONN_BACKWARD = 2, EMR_CONN_LATERAL = 4, EMR_CONN_SELF = 8,
       EMR_CONN_ALL = 15 };

/* Output of emr_express (device buffers, caller-owned): pair r's connections are entries
 * pair_offset[r] .. + pair_count[r] - 1, in ascending cell order. */
typedef struct {
  uint32_t* cell;       /* [capacity] heap index of the grid end of the connection */
  float* w;             /* [capacity] its weight (the CPPN output at that cell) */
  int64_t capacity;
  int64_t* pair_count;  /* [n_pairs] */
  int64_t* pair_offset; /* [n_pairs + 1] */
  void* workspace;      /* >= emr_express_workspace_bytes(n_pairs), 256-byte aligned */
  int64_t workspace_bytes;
} emr_connections;

emr_status emr_express_workspace_bytes(int64_t n_pairs, int64_t* bytes);

/*
 * The connections a discovery expresses: each child C of a kept parent of pair (g, s) is a
 * connection s -> C for an outgoing source and C -> s for an incoming one, weighted by the CPPN
 * output at C; it is kept when its type (Section 4) is in type_mask and |w| > w_min (Section 3.3:
 * the weight magnitude filter that replaces ES-HyperNEAT's band threshold, 0.1 in the paper).
 * fp32 comparisons. Check with emr_call_check(workspace, capacity).
 */
emr_status emr_express(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                       const int32_t* src_offsets, int32_t n_shared, int32_t depth,
                       const emr_result* rec, int32_t type_mask, float w_min,
                       const emr_connections* out, void* stream);

/* Workspace of emr_band_values: a 16-byte program entry per pair. Host only. */
emr_status emr_band_workspace_bytes(int64_t n_pairs, int64_t* bytes);

/*
 * ES-HyperNEAT's band values of expressed connections (Theorem 1 names a band threshold beside the
 * variance threshold and leaves it to ES-HyperNEAT, whose pruning step keeps a point whose weight
 * stands out from its neighbours' on both sides along x or along y). For connection i of `conn`
 * (the CSR output of emr_express for the same population, sources and depth: pair r, heap cell C
 * with centre (x, y) at level l, weight w): the pair's CPPN at the same-level neighbour centres
 * (x - d, y), (x + d, y), (x, y - d), (x, y + d), d = 2^(1-l) (exact in fp32), and
 *   band[i] = max(min(|w - left|, |w - right|), min(|w - down|, |w - up|))
 * in fp32 (fminf / fmaxf: a NaN operand is ignored). band: device, caller-owned, [conn->capacity]
 * (entries past the connections are not written). conn->pair_count and conn->workspace are not
 * used. `workspace` (device, >= emr_band_workspace_bytes(n_pairs), 256-byte aligned) holds the
 * pairs' program entries. Enqueued on `stream`; check with emr_call_check(workspace, 0):
 * EMR_E_DEVICE when a connection names no cell of the grid (its band is not written).
 */
emr_status emr_band_values(const emr_population* pop, const emr_source* sources,
                           int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                           int32_t depth, const emr_connections* conn, float* band,
                           void* workspace, int64_t workspace_bytes, void* stream);

/*
 * The band filter: the connections of `in` (n_pairs pairs, the layout of emr_express) whose band
 * value (emr_band_values, device [in->capacity]) exceeds theta_band (strict; a NaN band never
 * does), in their order, to `out` (its workspace at least emr_express_workspace_bytes(n_pairs)).
 * theta_band < 0 keeps every connection with a band value that is not NaN. EMR_E_INVAL for a NaN
 * theta_band. Check with emr_call_check(out->workspace, out->capacity).
 */
emr_status emr_band_filter(const emr_connections* in, const float* band, int64_t n_pairs,
                           float theta_band, const emr_connections* out, void* stream);

emr_status emr_chain_workspace_bytes(int64_t n_pairs, int32_t depth, int64_t* bytes);

/*
 * Eq. 2 read literally: keeps a record only when every ancestor of its cell is a record of the
 * same pair too (the active mask propagated from the root), which is ES-HyperNEAT's division
 * (the Superset Discovery theorem's lazy set). `out` receives those records in CSR form (its
 * workspace at least emr_chain_workspace_bytes); n_pairs is the discover call's. Check with
 * emr_result_check(out).
 */
emr_status emr_chain_filter(const emr_result* rec, int64_t n_pairs, int32_t depth,
                            const emr_result* out, void* stream);

/* ------------------------------------------------------------------ streaming
 * Deep runs stream their output between device and host memory (Section 5.2: the depth-7 note of
 * the per-generation timing table and the depth 8..13 runs of the total-runtime figure; Section 6
 * on depth 13). Here the stream carries only the compacted records, chunk by chunk. */

/* Receives the records of one pair for one chunk: n_records (> 0) kept parent cells in ascending
 * order, parent[i] their heap indices and w4[4 i + k] the CPPN outputs at their children. The
 * pointers are host memory owned by the library (pinned staging) and valid only during the call.
 * Return 0 to continue; any other value stops the run before these records count as delivered. */
typedef int32_t (*emr_sink)(int64_t pair, int64_t chunk, const uint32_t* parent, const float* w4,
                            int64_t n_records, void* user);

/* Number of chunks a streamed call at this depth and chunk size has. A chunk is a run of
 * chunk_positions / 256 tiles of every pair; a tile is 256 grid positions of one level, except
 * the first tile, which holds levels 1..3 (84 positions). chunk_positions must be a positive
 * multiple of 256. Host only. */
emr_status emr_stream_chunks(int32_t depth, int64_t chunk_positions, int64_t* n_chunks);

/*
 * Eager discovery in chunks, for depths whose output does not fit one device buffer: for chunk
 * c = 0, 1, ... (see emr_stream_chunks) every pair's kept parents whose children lie in the chunk
 * are found exactly as by emr_discover, then passed to `sink` once per (chunk, pair) with records,
 * chunk after chunk and pair after pair, each pair's records in ascending parent order. So the
 * concatenation over chunks of a pair's records equals its emr_discover output.
 * Work and delivery overlap: the GPU computes chunk c + 1 on `stream` while the records of chunk c
 * are copied to pinned host memory on a library side stream and delivered.
 * Cursor: deliveries are numbered k = chunk * n_pairs + pair. The run starts at cursor `start`
 * (0 for a full run; deliveries below it are skipped), and *next (may be NULL) receives the
 * cursor to resume from: n_chunks * n_pairs after a complete run, or, when the sink returns
 * nonzero, the cursor of the delivery it refused (status EMR_E_ABORTED). Returns when done.
 * Device memory: the library needs a workspace whose record pool, and two chunk outputs, hold
 * n_pairs * min(64 chunk_positions / 256, Q(D)) records each (20 bytes a record), plus pinned
 * staging, a side stream and events; it keeps them after the call for the next streamed call on
 * the device (grown when a call needs more, held until the process ends); EMR_E_LIMIT if the
 * record buffers would exceed 48 GiB or 2^32 records (use smaller chunks).
 * Errors: EMR_E_INVAL for bad arguments (checked before any GPU work), EMR_E_NOMEM, EMR_E_DEVICE
 * (also when a kernel flagged an internal error: checked before each chunk is delivered, so no
 * record of a chunk computed after such an error reaches the sink; *next then holds the cursor of
 * that chunk's first delivery), EMR_E_ABORTED.
 */
emr_status emr_discover_stream(const emr_population* pop, const emr_source* sources,
                               int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                               int32_t depth, float theta, int64_t chunk_positions, int64_t start,
                               emr_sink sink, void* user, int64_t* next, void* stream);

/* ------------------------------------------------------------------ record files
 * A sink that writes a streamed run to a file, so the output of a deep run is bounded by the disk
 * rather than by host memory (Section 6: the depth-13 substrates streamed from disk), and a run
 * that stopped resumes where the file ends. Host only; one handle serves one run at a time.
 *
 * File layout (little-endian): a 32-byte header {char magic[8] = "EMRRECv1", int64 n_pairs,
 * int64 0, int64 0}; then one block per delivery, in increasing cursor order:
 * {int64 pair, int64 chunk, int64 n (>= 1)}, uint32 parent[n], float w4[4 n] (as delivered). */
typedef struct emr_record_file emr_record_file;

/* Opens `path` for a run over n_pairs pairs (the streamed call's: genomes x shared sources, or
 * the total of the per-genome sources). resume = 0 creates or truncates the file. resume = 1 keeps
 * an existing file's whole deliveries (a trailing partial block, left by a run that died while
 * writing, is cut off) and sets *cursor (may be NULL) to the cursor after the last one: pass it
 * as emr_discover_stream's `start`; a missing file is created (*cursor = 0). buffer_bytes is the
 * host write buffer (0: 8 MiB; at most 2^30). *out receives the handle.
 * EMR_E_INVAL (bad arguments, not a record file, another n_pairs, malformed blocks), EMR_E_IO. */
emr_status emr_record_file_open(const char* path, int64_t n_pairs, int32_t resume,
                                int64_t buffer_bytes, emr_record_file** out, int64_t* cursor);

/* The emr_sink that appends a delivery to the file; `user` is the handle. Refuses (returns 1) a
 * delivery whose cursor precedes the file's end, a malformed delivery, and every delivery after a
 * failed write or a refusal; the reason is reported by emr_record_file_close. */
int32_t emr_record_file_sink(int64_t pair, int64_t chunk, const uint32_t* parent, const float* w4,
                             int64_t n_records, void* user);

/* Flushes, syncs and closes the file and frees the handle (always). *records and *next (either
 * may be NULL) receive the records in the file and the cursor after its last delivery.
 * EMR_E_IO when a write failed, EMR_E_INVAL when a delivery was refused, else EMR_OK. */
emr_status emr_record_file_close(emr_record_file* file, int64_t* records, int64_t* next);

/* ------------------------------------------------------------------ networks
 * The networks the experiments evaluate (Section 5: XOR over its four input patterns), built from
 * each genome's discovered substrate, and their activation. The paper names the parts (Phase 1,
 * the hidden-to-hidden phase of Section 2 and the connection types of Section 4's configurations)
 * without spelling out the assembly; the library builds it as ES-HyperNEAT does:
 *   - phase 0 is emr_discover on the substrate sources; its hidden nodes are the children of the
 *     kept parents of the outgoing pairs (emr_hidden_sources);
 *   - each further phase (at most `iterations`) queries, per genome, the hidden nodes the previous
 *     phase found and no earlier phase had, as outgoing sources at their cell centres, and adds the
 *     children of its kept parents that are new; it stops early when no genome finds one;
 *   - every phase's connections are expressed with type_mask and w_min (emr_express); each is an
 *     edge between the source's node and the grid cell's node, in the connection's direction; a
 *     connection to a cell that is not a hidden node (an incoming source's cell that no outgoing
 *     query reached) is dropped;
 *   - a hidden node is kept when an input reaches it and it reaches an output; an edge u -> v when
 *     an input reaches u and v reaches an output. Substrate nodes are always kept.
 * Node numbers per genome: the substrate sources in substrate order (inputs are the outgoing
 * sources, outputs the incoming ones), then the kept hidden nodes in ascending heap cell order.
 * A node's incoming edges are listed in the order phase, pair, cell.
 * Activation is synchronous: input nodes hold the pattern's values, every other node starts at 0
 * and at each step takes sigmoid(sum of w * the source node's previous value) = 1/(1+e^-z) over
 * its incoming edges, in fp32: edge k of the node's list goes to partial sum k mod 64 (an fmaf
 * chain in list order), and the 64 partial sums are added in a fixed butterfly, so every run
 * gives the same bits. Each step is one launch on the stream. */
typedef struct emr_networks emr_networks;

#define EMR_SUBSTRATE_NODE 0xFFFFFFFFu /* node_cell of a substrate node */

/* Builds the networks of every genome of `pop` for the substrate (host, n_substrate sources with
 * at least one input and one output) at this depth and theta; type_mask (EMR_CONN_*, 1..15) and
 * w_min filter the connections; iterations (0..64) bounds the hidden-to-hidden phases (0: the
 * feedforward configuration without them). Runs on `stream` and synchronizes with it; *out
 * receives a handle owning every device buffer below (free with emr_free_networks). The
 * population's grouping tables are replaced by those of the last phase (emr_discover's rule).
 * EMR_E_INVAL, EMR_E_LIMIT (more than 2^32 - 2 nodes), EMR_E_NOMEM, EMR_E_DEVICE, or any status of
 * the discovery calls it makes. */
emr_status emr_build_networks(const emr_population* pop, const emr_source* substrate,
                              int32_t n_substrate, int32_t depth, float theta, int32_t type_mask,
                              float w_min, int32_t iterations, emr_networks** out, void* stream);

/* The networks (device pointers owned by the handle, valid until emr_free_networks). Genome g's
 * nodes are node_offset[g] .. node_offset[g+1] - 1; node i's incoming edges are
 * in_offset[i] .. in_offset[i+1] - 1, with in_src the source's node index (counted over all
 * genomes) and in_w the weight. known: the hidden cells of every phase before pruning, a
 * bitmap of known_words words per genome (bit p stands for heap cell p + 1). */
typedef struct {
  int32_t n_genomes, n_substrate, n_inputs, n_outputs, depth, phases;
  int64_t nodes, edges;
  const int64_t* node_offset; /* [n_genomes + 1] */
  const uint32_t* node_cell;  /* [nodes]: heap cell, EMR_SUBSTRATE_NODE for substrate nodes */
  const int64_t* in_offset;   /* [nodes + 1] */
  const uint32_t* in_src;     /* [edges] */
  const float* in_w;          /* [edges] */
  const uint32_t* known;      /* [n_genomes * known_words] */
  int64_t known_words;
} emr_network_info;
emr_status emr_networks_info(const emr_networks* net, emr_network_info* info);

/* One phase of a build (0 .. phases - 1), for inspection: its sources (host, owned by the handle:
 * the substrate for phase 0, else per genome the queried hidden nodes at src_offsets, with their
 * heap cells in src_cell on the device), its checked discovery (CSR over n_pairs pairs: parent,
 * w4, pair_offset, `records` in all) and its expressed connections (conn_cell, conn_w,
 * conn_offset, `connections` in all). Device pointers owned by the handle. */
typedef struct {
  const emr_source* sources;
  int32_t n_sources;
  const int32_t* src_offsets; /* NULL for phase 0 */
  const uint32_t* src_cell;   /* NULL for phase 0 */
  int64_t n_pairs;
  const uint32_t* parent;
  const float* w4;
  const int64_t* pair_offset;
  int64_t records;
  const uint32_t* conn_cell;
  const float* conn_w;
  const int64_t* conn_offset;
  int64_t connections;
} emr_network_phase;
emr_status emr_networks_phase(const emr_networks* net, int32_t phase, emr_network_phase* out);

/* Activates every network for n_patterns (1..65536) input patterns (host, [n_patterns][n_inputs]
 * in input order, read during the call) for `steps` (0..2^20) synchronous steps and writes the
 * outputs (device, caller-owned, [n_genomes][n_patterns][n_outputs]). Enqueued on `stream` (the
 * device the networks were built on must be current). The handle's state buffers serve one call at
 * a time: calls on one handle must be ordered on one stream. */
emr_status emr_activate(const emr_networks* net, const float* inputs, int32_t n_patterns,
                        int32_t steps, float* outputs, void* stream);

/* XOR fitness of every network (device, caller-owned, [n_genomes]): 1 - the mean squared error of
 * the single output over (a, b) = (0,0), (0,1), (1,0), (1,1) with targets 0, 1, 1, 0, after
 * `steps` steps; a and b are the first and second input other than bias_input, the input held at
 * 1 (-1: none). Needs one output and two inputs besides the bias. Enqueued like emr_activate. */
emr_status emr_xor_fitness(const emr_networks* net, int32_t bias_input, int32_t steps,
                           float* fitness, void* stream);

void emr_free_networks(emr_networks* net);

/* Copies `bytes` of device memory (such as the buffers the info calls above point to) to host
 * memory after the work already on `stream`; returns when the copy is done. */
emr_status emr_copy_to_host(void* host, const void* device, int64_t bytes, void* stream);

/*
 * Raw CPPN outputs (debug and parity): out_dev[r * N(D) + p] = CPPN output of pair r at grid
 * position p (device, caller-owned, n_pairs * N(D) floats). Same arithmetic as emr_discover.
 */
emr_status emr_eval_raw(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                        const int32_t* src_offsets, int32_t n_shared, int32_t depth, float* out_dev,
                        void* workspace, int64_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ allocation-free raw outputs
 * For callers that cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation. */

/* Size of the library's allocation-free scratch: a static array in the library's code object, one
 * copy per device the library runs on, held until the process ends. */
#define EMR_NOALLOC_SCRATCH_BYTES (32 << 20)

/*
 * emr_eval_raw without allocating: the same outputs (out_dev[r * N(D) + p], device, caller-owned,
 * n_pairs * N(D) floats), computed by the interpreter (the compiled tier loads a module, so it is
 * never used here), with every device buffer besides out_dev and err_dev in the scratch: the
 * call's tables, the depth's tile geometry and the workspace. The call makes no device, pinned or
 * host-registered allocation and loads no module; the only host memory it keeps is its plan,
 * held by the population (one per distinct sources and depth used this way).
 * err_dev: device, caller-owned, one word; the call's first kernel clears it and its kernels raise
 * error bits into it (2: a table entry out of range, the affected outputs left unwritten), to be
 * read after the stream's work completes.
 * Errors: EMR_E_INVAL for bad arguments; EMR_E_LIMIT when the call's tables, tile geometry and
 * workspace exceed EMR_NOALLOC_SCRATCH_BYTES (checked before anything is enqueued); EMR_E_DEVICE.
 * Every call on a device shares that device's scratch and leaves its last contents there: calls
 * that overlap in time on one device (other streams, other threads) race and must not be made.
 */
emr_status emr_eval_raw_noalloc(const emr_population* pop, const emr_source* sources,
                                int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                                int32_t depth, float* out_dev, uint32_t* err_dev, void* stream);

/* Algorithmic VALU work of one emr_discover call under the cost model documented with the
 * benchmark: total lane-operation slots (*slots) and number of queries (*queries). Per query of a
 * (genome, direction) program: one slot per position-dependent edge, the activations' slots
 * (transcendental instructions weighted by transcendental_slots) and 2.5 for the variance, where
 * a node whose value does not depend on the source counts once for the S sources walked together
 * (1 / S of it per query: the compiled tier evaluates it once per position); a
 * program whose output does not depend on the position costs 0 (its outputs are per-source
 * constants and their variance is exactly zero). *evaluated: the queries of the pairs whose output
 * depends on the position (the others are answered by their per-source constant); *flops: useful
 * floating-point operations, 2 per position-dependent edge (a multiply-add), 1 per other
 * activation operation and per transcendental, 2.5 per query for the variance. Any output pointer
 * may be NULL. Host only. */
emr_status emr_discover_cost(const emr_population* pop, const emr_source* sources,
                             int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                             int32_t depth, double transcendental_slots, double* slots,
                             double* queries, double* evaluated, double* flops);

/* ------------------------------------------------------------------ compiled tier */

/* The discover kernel runs a call's varying CPPN programs either through the interpreter (the
 * record step walks each packed program record by record) or as machine code compiled for the
 * population: each (genome, direction) program is translated on the host into gfx950 instructions
 * with its weights as literal operands, written into the code area of a copy of a template code
 * object, and loaded as a module (Sections 3.1-3.2 compute the same thing either way; the compiled
 * program performs the interpreter's arithmetic instruction for instruction, so both produce the
 * same bits). Compilation costs host time (translation, about 1 ms per MB of code to load) and
 * pays off for repeated or large calls. Policies:
 *   EMR_JIT_OFF     always interpret;
 *   EMR_JIT_AUTO    compile a plan (a population with the same sources and depth) when it is run
 *                   a second time, or at once when the call is large; a failed compilation leaves
 *                   the plan interpreted (see emr_jit_info);
 *   EMR_JIT_ALWAYS  compile on the first call; a failed compilation fails the call. */
enum { EMR_JIT_OFF = 0, EMR_JIT_AUTO = 1, EMR_JIT_ALWAYS = 2 };

/* Sets the process-wide policy (default EMR_JIT_AUTO) for later calls. EMR_E_INVAL otherwise. */
emr_status emr_set_jit(int32_t policy);

/* The compiled tier of the population's current plan (the plan of its last call): *state 0 not
 * compiled, 1 compiled, -1 compilation failed (emr_last_error then holds the reason); *programs the
 * distinct programs compiled, *code_bytes their machine code, *compile_ms the host translation time
 * and *load_ms the module load. Any output pointer may be NULL. Host only. */
emr_status emr_jit_info(const emr_population* pop, int32_t* state, int64_t* programs,
                        int64_t* code_bytes, double* compile_ms, double* load_ms);

/* ------------------------------------------------------------------ profiling */

/* One discover-kernel launch of a profiled emr_discover / emr_eval_raw call on this thread (a call
 * makes one launch for every tile range it covers: one for emr_discover, one per chunk when
 * streamed): the variant of its costliest part (sources per walk S, register window W, positions
 * per lane P), its tiles, queries and algorithmic VALU slots over all its parts under the cost
 * model of emr_discover_cost, and its duration from a HIP event pair recorded on the call's stream
 * around the launch. */
typedef struct {
  int32_t group_size, window, positions;
  int32_t call;  /* profiled call the launch belongs to, counted from 0 */
  int64_t tiles, queries;
  double slots;
  float ms;
  int32_t compiled; /* 1: the launch ran compiled programs, 0: the interpreter */
  int32_t listed;   /* 1: its workgroups took their chunks from the plan's balanced lists (a
                       compiled plan's later calls), 0: from round-robin shares */
  int32_t parts;    /* runs of groups with one chunk size the launch was split into */
} emr_launch_profile;

/* Sets per-launch event timing for the calling thread's later calls and drops the records held:
 * on = 0 off, 1 every discover launch, 2 only the first discover launch of a call; `every` >= 1:
 * only one call in `every` is timed (the first, then every `every`-th), which keeps the events'
 * own cost off the other calls. transcendental_slots is the cost-model weight used for `slots`.
 * EMR_E_INVAL for another `on` or `every` < 1. */
emr_status emr_profile_enable(int32_t on, int32_t every, double transcendental_slots);

/* *n receives the number of launch records held (the timed launches of the profiled calls since
 * the last enable or read). With out != NULL, synchronizes on their events, writes up to `cap` of
 * them to `out` (host) and drops them. Records are in launch order. */
emr_status emr_profile_read(emr_launch_profile* out, int32_t cap, int32_t* n);

#ifdef __cplusplus
}
#endif

#endif /* EMR_H */
