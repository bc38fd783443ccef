// gfx950 kernels that turn the discovered substrate into networks and run them (the networks the
// experiments evaluate, Section 5): the hidden-cell bitmap's rank (node numbers), the expressed
// connections as edges between node numbers, pruning to the nodes on an input-to-output path, the
// kept nodes' numbering and their incoming edges grouped by destination, and synchronous
// activation over a batch of input patterns with an optional XOR fitness.
//
// Work over edges runs one thread per edge across the whole population, and activation one wave
// per (node, pattern block): genomes are very unequal (a genome with a high-frequency CPPN can
// hold a large share of the population's edges), so no step may give one genome to one
// workgroup when its cost grows with the genome's edges. Only steps whose cost follows a
// genome's node count (its bitmap, its node numbering) run one workgroup per genome. Numbering
// and layouts: network.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "emr_internal.h"
#include "network.h"

namespace emr {
namespace {

// Exclusive prefix sum over the workgroup's kNetThreads threads (every thread must call it);
// *total receives the sum. `part` holds one word per wave.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* part, uint32_t* total) {
  const uint32_t lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)x, (unsigned)o, kWave);
    if (lane >= (uint32_t)o) x += y;
  }
  if (lane == kWave - 1) part[wv] = x;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kNetThreads / kWave; ++i) {
    const uint32_t p = part[i];
    before += (i < (int)wv) ? p : 0u;
    tot += p;
  }
  __syncthreads();  // `part` is free again
  *total = tot;
  return before + x - v;
}

// The r with off[r] <= i < off[r + 1], for off[0] <= i < off[n] (empty segments skipped).
__device__ __forceinline__ int64_t find_segment(const int64_t* off, int64_t n, int64_t i) {
  int64_t lo = 0, hi = n;
  while (hi - lo > 1) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (off[mid] <= i) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Raw node number of heap cell `cell` in genome g (n_sub + its rank among the genome's hidden
// cells), or kNoNode when the cell is not a hidden node.
__device__ __forceinline__ uint32_t node_of(const uint32_t* known, const uint32_t* rank,
                                            int64_t words, uint32_t g, uint32_t n_sub,
                                            uint32_t cell) {
  if (cell == 0u) return kNoNode;
  const uint32_t p = cell - 1u;  // grid position
  const int64_t w = (int64_t)(p >> 5);
  if (w >= words) return kNoNode;
  const uint32_t word = known[(int64_t)g * words + w];
  const uint32_t b = p & 31u;
  if (((word >> b) & 1u) == 0u) return kNoNode;
  return n_sub + rank[(int64_t)g * words + w] + (uint32_t)__builtin_popcount(word & ((1u << b) - 1u));
}

__device__ __forceinline__ float sigmoid_f(float z) { return 1.0f / (1.0f + expf(-z)); }

__device__ __forceinline__ float comp(const float4& v, uint32_t c) {
  return c == 0u ? v.x : (c == 1u ? v.y : (c == 2u ? v.z : v.w));
}

__device__ __forceinline__ int64_t grid_thread() {
  return (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
}
__device__ __forceinline__ int64_t grid_threads() { return (int64_t)gridDim.x * blockDim.x; }

}  // namespace

// ------------------------------------------------------------------------ node numbers
__global__ void __launch_bounds__(kNetThreads) k_net_rank(NetRankArgs A) {
  __shared__ uint32_t part[kNetThreads / kWave];
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const uint32_t* k = A.known + (int64_t)g * A.words;
    uint32_t* r = A.rank + (int64_t)g * A.words;
    uint32_t run = 0;
    for (int64_t base = 0; base < A.words; base += 4 * kNetThreads) {
      const int64_t w0 = base + 4 * (int64_t)threadIdx.x;
      uint32_t c[4], s = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = w0 + q < A.words ? (uint32_t)__builtin_popcount(k[w0 + q]) : 0u;
        s += c[q];
      }
      uint32_t total;
      uint32_t acc = run + block_excl_scan(s, part, &total);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (w0 + q < A.words) r[w0 + q] = acc;
        acc += c[q];
      }
      run += total;
    }
    if (threadIdx.x == 0) A.hidden[g] = run;
  }
}

// ------------------------------------------------------------------------ raw edges
// One thread per expressed connection of one phase.
__global__ void __launch_bounds__(kNetThreads) k_net_edges(NetEdgeArgs A) {
  for (int64_t i = grid_thread(); i < A.total; i += grid_threads()) {
    const int64_t r = find_segment(A.conn_offset, A.n_pairs, i);
    uint32_t g, sn, dir;
    int64_t first;
    if (A.src_offsets == nullptr) {
      g = (uint32_t)(r / A.n_sub);
      const uint32_t j = (uint32_t)(r % A.n_sub);
      sn = j;
      dir = A.sub_dir[j];
      first = (int64_t)g * A.n_sub;
    } else {
      g = (uint32_t)find_segment(A.src_offsets, A.n_genomes, r);
      first = A.src_offsets[g];
      sn = g < A.n_genomes ? node_of(A.known, A.rank, A.words, g, A.n_sub, A.src_cell[r]) : kNoNode;
      dir = 0u;
    }
    if (g >= A.n_genomes || sn == kNoNode) {
      atomicOr(A.err, kNetErrIndex);
      continue;
    }
    const int64_t o = A.seg[g] + (i - A.conn_offset[first]);
    if (o < A.raw_edge[g] || o >= A.raw_edge[g + 1]) {
      atomicOr(A.err, kNetErrIndex);
      continue;
    }
    const uint32_t cn = node_of(A.known, A.rank, A.words, g, A.n_sub, A.conn_cell[i]);
    const int64_t nb = A.raw_node[g], n = A.raw_node[g + 1] - nb;
    uint32_t u = dir == 0u ? sn : cn, v = dir == 0u ? cn : sn;
    if (cn == kNoNode) {
      u = v = kNoNode;  // the grid end is not a hidden node: dropped
    } else if ((int64_t)u >= n || (int64_t)v >= n) {
      atomicOr(A.err, kNetErrIndex);
      u = v = kNoNode;
    } else {
      u += (uint32_t)nb;  // (the host bounds the raw nodes below kNoNode)
      v += (uint32_t)nb;
    }
    A.eu[o] = u;
    A.ev[o] = v;
    A.ew[o] = A.conn_w[i];
  }
}

// ------------------------------------------------------------------------ pruning
// Flags of every raw node before the passes: substrate inputs reach themselves, substrate
// outputs reach an output; no kept edge yet. One workgroup per genome (its nodes).
__global__ void __launch_bounds__(kNetThreads) k_net_flags(NetFlagArgs A) {
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const int64_t nb = A.raw_node[g], n = A.raw_node[g + 1] - nb;
    for (int64_t j = threadIdx.x; j < n; j += blockDim.x) {
      const bool sub = j < (int64_t)A.n_sub;
      A.fwd[nb + j] = (uint8_t)(sub && A.sub_dir[j] == 0u);
      A.bwd[nb + j] = (uint8_t)(sub && A.sub_dir[j] != 0u);
      A.in_deg[nb + j] = 0u;
    }
  }
}

// One pass over every raw edge of the population: u -> v carries reachability from an input
// forward (fwd[u] -> fwd[v]) and reachability of an output backward (bwd[v] -> bwd[u]). Flags only
// go from 0 to 1, so a thread reading a flag another thread is setting sees either value; a pass
// that changes nothing saw only values fixed since the launch began (every write of the previous
// pass is visible at launch), which is the fixed point. The host repeats passes until one
// reports no change.
__global__ void __launch_bounds__(kNetThreads) k_net_reach(NetReachArgs A) {
  bool ch = false;
  for (int64_t e = grid_thread(); e < A.edges; e += grid_threads()) {
    const uint32_t u = A.eu[e], v = A.ev[e];
    if ((int64_t)u >= A.nodes || (int64_t)v >= A.nodes) continue;  // dropped edge
    if (A.fwd[u] && !A.fwd[v]) {
      A.fwd[v] = 1;
      ch = true;
    }
    if (A.bwd[v] && !A.bwd[u]) {
      A.bwd[u] = 1;
      ch = true;
    }
  }
  if (__ballot(ch) != 0ull && (threadIdx.x % kWave) == 0) *A.changed = 1u;
}

// An edge u -> v is kept when an input reaches u and v reaches an output (then both ends are
// kept nodes); each kept edge counts into its destination's in-degree.
__global__ void __launch_bounds__(kNetThreads) k_net_degree(NetReachArgs A) {
  for (int64_t e = grid_thread(); e < A.edges; e += grid_threads()) {
    const uint32_t u = A.eu[e], v = A.ev[e];
    if ((int64_t)u >= A.nodes || (int64_t)v >= A.nodes) continue;
    if (A.fwd[u] && A.bwd[v]) atomicAdd(A.in_deg + v, 1u);
  }
}

// Per genome: kept hidden nodes (reached from an input and reaching an output) and kept edges
// (the sum of the in-degrees). One workgroup per genome (its nodes).
__global__ void __launch_bounds__(kNetThreads) k_net_kept(NetFlagArgs A) {
  __shared__ uint32_t part[kNetThreads / kWave];
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const int64_t nb = A.raw_node[g], n = A.raw_node[g + 1] - nb;
    uint32_t kn = 0u, ke = 0u;
    for (int64_t j = threadIdx.x; j < n; j += blockDim.x) {
      if (j >= (int64_t)A.n_sub && A.fwd[nb + j] && A.bwd[nb + j]) ++kn;
      ke += A.in_deg[nb + j];
    }
    uint32_t tn, te;
    block_excl_scan(kn, part, &tn);
    block_excl_scan(ke, part, &te);
    if (threadIdx.x == 0) {
      A.kept_nodes[g] = tn;
      A.kept_edges[g] = te;
    }
  }
}

// ------------------------------------------------------------------------ kept nodes
// One workgroup per genome: kept numbers in raw order, the kept nodes' first incoming edge and
// input numbers, then the kept hidden nodes' heap cells.
__global__ void __launch_bounds__(kNetThreads) k_net_nodes(NetNodeArgs A) {
  __shared__ uint32_t part[kNetThreads / kWave];
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const int64_t nb = A.raw_node[g], n = A.raw_node[g + 1] - nb;
    const int64_t NB = A.node_offset[g], NE = A.node_offset[g + 1];
    const int64_t EB = A.edge_offset[g];
    uint32_t run_id = 0u, run_deg = 0u;
    for (int64_t base = 0; base < n; base += kNetThreads) {
      const int64_t j = base + threadIdx.x;
      uint32_t keep = 0u, deg = 0u;
      if (j < n) {
        keep = (j < (int64_t)A.n_sub || (A.fwd[nb + j] && A.bwd[nb + j])) ? 1u : 0u;
        deg = keep ? A.in_deg[nb + j] : 0u;
      }
      uint32_t tk, td;
      const uint32_t ek = block_excl_scan(keep, part, &tk);
      const uint32_t ed = block_excl_scan(deg, part, &td);
      if (j < n) {
        const uint32_t id = run_id + ek;
        uint32_t gl = kNoNode;
        if (keep) {
          if (NB + id >= NE) {
            atomicOr(A.err, kNetErrIndex);
          } else {
            gl = (uint32_t)(NB + id);  // (the host bounds the kept nodes below kNoNode)
            A.in_offset[NB + id] = EB + run_deg + ed;
            const bool sub = j < (int64_t)A.n_sub;
            A.node_in[NB + id] = sub ? A.in_slot[j] : -1;
            if (sub) A.node_cell[NB + id] = kNoNode;
          }
        }
        A.gid[nb + j] = gl;
      }
      run_id += tk;
      run_deg += td;
    }
    if (threadIdx.x == 0) {
      if (NB + run_id != NE || EB + run_deg != A.edge_offset[g + 1]) atomicOr(A.err, kNetErrIndex);
      if (g == A.n_genomes - 1) A.in_offset[NE] = A.edge_offset[g + 1];
    }
    __syncthreads();  // gid of the whole genome before the cell pass
    const uint32_t* kw = A.known + (int64_t)g * A.words;
    const uint32_t* rk = A.rank + (int64_t)g * A.words;
    for (int64_t w = threadIdx.x; w < A.words; w += blockDim.x) {
      uint32_t word = kw[w];
      uint32_t raw = A.n_sub + rk[w];
      while (word != 0u) {
        const uint32_t b = (uint32_t)__builtin_ctz(word);
        word &= word - 1u;
        if ((int64_t)raw >= n) {
          atomicOr(A.err, kNetErrIndex);
          break;
        }
        const uint32_t id = A.gid[nb + raw];
        if (id != kNoNode && (int64_t)id >= NB && (int64_t)id < NE)
          A.node_cell[id] = 32u * (uint32_t)w + b + 1u;
        ++raw;
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------------ incoming edges
// Sort keys of the raw edges: a kept edge's destination's kept number (sentinel: dropped).
__global__ void __launch_bounds__(kNetThreads) k_net_keys(NetKeyArgs A) {
  for (int64_t e = grid_thread(); e < A.edges; e += grid_threads()) {
    const uint32_t u = A.eu[e], v = A.ev[e];
    uint32_t key = A.sentinel;
    if ((int64_t)u < A.nodes && (int64_t)v < A.nodes && A.fwd[u] && A.bwd[v]) {
      const uint32_t gu = A.gid[u], gv = A.gid[v];
      if (gu >= A.sentinel || gv >= A.sentinel) atomicOr(A.err, kNetErrIndex);
      else key = gv;
    }
    A.key[e] = key;
    A.val[e] = (uint32_t)e;  // (the host bounds the raw edges below 2^32)
  }
}

// The sorted kept edges (the first `edges` entries) to their CSR slots: entry i holds the edge
// at slot i, whose destination's range must contain i.
__global__ void __launch_bounds__(kNetThreads) k_net_gather(NetGatherArgs A) {
  for (int64_t i = grid_thread(); i < A.edges; i += grid_threads()) {
    const uint32_t k = A.key[i], e = A.val[i];
    if ((int64_t)k >= A.nodes || (int64_t)e >= A.raw_edges || i < A.in_offset[k] ||
        i >= A.in_offset[k + 1]) {
      atomicOr(A.err, kNetErrIndex);
      continue;
    }
    const uint32_t u = A.eu[e];
    const uint32_t gu = (int64_t)u < A.raw_nodes ? A.gid[u] : kNoNode;
    if ((int64_t)gu >= A.nodes) {
      atomicOr(A.err, kNetErrIndex);
      continue;
    }
    A.in_src[i] = gu;
    A.in_w[i] = A.ew[e];
  }
}

// ------------------------------------------------------------------------ activation
// Initial state: input nodes hold their pattern values, every other node 0.
__global__ void __launch_bounds__(kNetThreads) k_net_state(NetStateArgs A) {
  const int64_t total = (int64_t)A.pblocks * A.nodes;
  float4* st = reinterpret_cast<float4*>(A.state);
  for (int64_t t = grid_thread(); t < total; t += grid_threads()) {
    const uint32_t pb = (uint32_t)(t / A.nodes);
    const int64_t i = t - (int64_t)pb * A.nodes;
    const int32_t slot = A.node_in[i];
    float c[4] = {0.f, 0.f, 0.f, 0.f};
    if (slot >= 0 && (uint32_t)slot < A.n_inputs) {
#pragma unroll
      for (uint32_t q = 0; q < 4; ++q) {
        const uint32_t p = 4u * pb + q;
        c[q] = p < A.n_patterns ? A.patterns[(int64_t)p * A.n_inputs + (uint32_t)slot] : 0.0f;
      }
    }
    st[t] = make_float4(c[0], c[1], c[2], c[3]);
  }
}

// One synchronous step: one wave per (node, pattern block). An input node keeps its values; every
// other node takes sigmoid of the sum of w * (the source's previous state) over its incoming
// edges: lane k sums edges k, k + 64, ... of the node's list as an fmaf chain in list order, then
// the 64 partial sums are added in a fixed butterfly (the same bits on every run).
__global__ void __launch_bounds__(kNetThreads) k_net_step(NetStepArgs A) {
  const int64_t item = (int64_t)blockIdx.x * (kNetThreads / kWave) + threadIdx.x / kWave;
  const int64_t total = (int64_t)A.pblocks * A.nodes;
  if (item >= total) return;
  const uint32_t lane = threadIdx.x % kWave;
  const uint32_t pb = (uint32_t)(item / A.nodes);
  const int64_t i = item - (int64_t)pb * A.nodes;
  const float4* cur = reinterpret_cast<const float4*>(A.cur) + (int64_t)pb * A.nodes;
  float4* nxt = reinterpret_cast<float4*>(A.nxt) + (int64_t)pb * A.nodes;
  if (A.node_in[i] >= 0) {
    if (lane == 0) nxt[i] = cur[i];
    return;
  }
  float zx = 0.f, zy = 0.f, zz = 0.f, zw = 0.f;
  const int64_t e1 = A.in_offset[i + 1];
  for (int64_t e = A.in_offset[i] + lane; e < e1; e += kWave) {
    const uint32_t s = A.in_src[e];
    if ((int64_t)s >= A.nodes) continue;  // (gather checked every source)
    const float w = A.in_w[e];
    const float4 x = cur[s];
    zx = fmaf(w, x.x, zx);
    zy = fmaf(w, x.y, zy);
    zz = fmaf(w, x.z, zz);
    zw = fmaf(w, x.w, zw);
  }
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) {
    zx += __shfl_xor(zx, o, kWave);
    zy += __shfl_xor(zy, o, kWave);
    zz += __shfl_xor(zz, o, kWave);
    zw += __shfl_xor(zw, o, kWave);
  }
  if (lane == 0) nxt[i] = make_float4(sigmoid_f(zx), sigmoid_f(zy), sigmoid_f(zz), sigmoid_f(zw));
}

// Outputs of every (genome, pattern, output), and the XOR fitness of every genome (one output,
// four patterns: 1 - the mean squared error against the targets).
__global__ void __launch_bounds__(kNetThreads) k_net_out(NetOutArgs A) {
  const float4* st = reinterpret_cast<const float4*>(A.state);
  const int64_t per_g = (int64_t)A.n_patterns * A.n_outputs;
  if (A.outputs) {
    for (int64_t t = grid_thread(); t < (int64_t)A.n_genomes * per_g; t += grid_threads()) {
      const uint32_t g = (uint32_t)(t / per_g);
      const int64_t r = t - (int64_t)g * per_g;
      const uint32_t p = (uint32_t)(r / A.n_outputs), o = (uint32_t)(r % A.n_outputs);
      const int64_t node = A.node_offset[g] + A.out_node[o];
      if (node >= A.node_offset[g + 1] || node >= A.nodes) continue;  // (host-checked)
      A.outputs[t] = comp(st[(int64_t)(p / 4u) * A.nodes + node], p % 4u);
    }
  }
  if (A.fitness) {
    for (int64_t g = grid_thread(); g < (int64_t)A.n_genomes; g += grid_threads()) {
      const int64_t node = A.node_offset[g] + A.out_node[0];
      if (node >= A.node_offset[g + 1] || node >= A.nodes) continue;
      const float4 v = st[node];
      float se = 0.0f;
      for (uint32_t q = 0; q < A.n_patterns && q < 4u; ++q) {
        const float d = comp(v, q) - A.targets[q];
        se = fmaf(d, d, se);
      }
      A.fitness[g] = 1.0f - se / (float)A.n_patterns;
    }
  }
}

}  // namespace emr

namespace {
uint32_t genome_blocks(uint32_t n) { return n == 0 ? 1u : (n > 65535u ? 65535u : n); }
// Workgroups for a grid-stride loop over n items (at least one, at most 16384).
uint32_t stride_blocks(int64_t n) {
  int64_t b = (n + emr::kNetThreads - 1) / emr::kNetThreads;
  return (uint32_t)(b < 1 ? 1 : (b > 16384 ? 16384 : b));
}
}  // namespace

// Steps: 0 rank, 1 edges, 2 flags, 3 reach pass, 4 degrees, 5 kept counts, 6 nodes, 7 keys,
// 8 gather, 9 initial state, 10 one activation step, 11 outputs / fitness.
extern "C" hipError_t emr_launch_net(int step, const void* args, int64_t work, hipStream_t s) {
  using namespace emr;
  (void)work;
  const dim3 blk(kNetThreads);
  switch (step) {
    case 0: {
      const auto& A = *static_cast<const NetRankArgs*>(args);
      hipLaunchKernelGGL(k_net_rank, dim3(genome_blocks(A.n_genomes)), blk, 0, s, A);
      break;
    }
    case 1: {
      const auto& A = *static_cast<const NetEdgeArgs*>(args);
      if (A.total <= 0) return hipSuccess;
      hipLaunchKernelGGL(k_net_edges, dim3(stride_blocks(A.total)), blk, 0, s, A);
      break;
    }
    case 2: {
      const auto& A = *static_cast<const NetFlagArgs*>(args);
      hipLaunchKernelGGL(k_net_flags, dim3(genome_blocks(A.n_genomes)), blk, 0, s, A);
      break;
    }
    case 3: {
      const auto& A = *static_cast<const NetReachArgs*>(args);
      hipLaunchKernelGGL(k_net_reach, dim3(stride_blocks(A.edges)), blk, 0, s, A);
      break;
    }
    case 4: {
      const auto& A = *static_cast<const NetReachArgs*>(args);
      hipLaunchKernelGGL(k_net_degree, dim3(stride_blocks(A.edges)), blk, 0, s, A);
      break;
    }
    case 5: {
      const auto& A = *static_cast<const NetFlagArgs*>(args);
      hipLaunchKernelGGL(k_net_kept, dim3(genome_blocks(A.n_genomes)), blk, 0, s, A);
      break;
    }
    case 6: {
      const auto& A = *static_cast<const NetNodeArgs*>(args);
      hipLaunchKernelGGL(k_net_nodes, dim3(genome_blocks(A.n_genomes)), blk, 0, s, A);
      break;
    }
    case 7: {
      const auto& A = *static_cast<const NetKeyArgs*>(args);
      hipLaunchKernelGGL(k_net_keys, dim3(stride_blocks(A.edges)), blk, 0, s, A);
      break;
    }
    case 8: {
      const auto& A = *static_cast<const NetGatherArgs*>(args);
      if (A.edges <= 0) return hipSuccess;
      hipLaunchKernelGGL(k_net_gather, dim3(stride_blocks(A.edges)), blk, 0, s, A);
      break;
    }
    case 9: {
      const auto& A = *static_cast<const NetStateArgs*>(args);
      hipLaunchKernelGGL(k_net_state, dim3(stride_blocks((int64_t)A.pblocks * A.nodes)), blk, 0, s,
                         A);
      break;
    }
    case 10: {
      const auto& A = *static_cast<const NetStepArgs*>(args);
      const int64_t waves = (int64_t)A.pblocks * A.nodes;
      const int64_t b = (waves + kNetThreads / kWave - 1) / (kNetThreads / kWave);
      if (b <= 0) return hipSuccess;
      if (b > 0x7FFFFFFF) return hipErrorInvalidValue;
      hipLaunchKernelGGL(k_net_step, dim3((uint32_t)b), blk, 0, s, A);
      break;
    }
    case 11: {
      const auto& A = *static_cast<const NetOutArgs*>(args);
      const int64_t items = A.outputs ? (int64_t)A.n_genomes * A.n_patterns * A.n_outputs
                                      : (int64_t)A.n_genomes;
      hipLaunchKernelGGL(k_net_out, dim3(stride_blocks(items)), blk, 0, s, A);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
