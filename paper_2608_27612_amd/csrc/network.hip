// gfx950 kernels that turn the discovered substrate into networks and run them (the networks the
// experiments evaluate, Section 5): the hidden-cell bitmap's rank (node numbers), the expressed
// connections as edges between node numbers, pruning to the nodes on an input-to-output path, the
// kept nodes' numbering and their incoming edges grouped by destination, and synchronous
// activation over a batch of input patterns with an optional XOR fitness. One workgroup per genome
// for the per-genome steps: a genome's network is small next to the chip, and a workgroup's
// barriers order its passes. Numbering and layouts: network.h.
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
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < A.total; i += stride) {
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
    uint32_t u = dir == 0u ? sn : cn, v = dir == 0u ? cn : sn;
    if (cn == kNoNode) u = v = kNoNode;  // the grid end is not a hidden node: dropped
    A.eu[o] = u;
    A.ev[o] = v;
    A.ew[o] = A.conn_w[i];
  }
}

// ------------------------------------------------------------------------ pruning
// One workgroup per genome: reachability from the inputs (fwd) and to the outputs (bwd) by passes
// over the genome's edges until a pass changes nothing. Flags only ever go from 0 to 1, so a pass
// that reads a flag another thread is setting sees either value and the fixed point is the same;
// at most 2 n + 1 passes change something.
__global__ void __launch_bounds__(kNetThreads) k_net_prune(NetPruneArgs A) {
  __shared__ uint32_t changed;
  __shared__ uint32_t part[kNetThreads / kWave];
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const int64_t nb = A.raw_node[g], n = A.raw_node[g + 1] - nb;
    const int64_t eb = A.raw_edge[g], ee = A.raw_edge[g + 1];
    uint8_t* fwd = A.fwd + nb;
    uint8_t* bwd = A.bwd + nb;
    for (int64_t j = threadIdx.x; j < n; j += blockDim.x) {
      const bool sub = j < (int64_t)A.n_sub;
      fwd[j] = (uint8_t)(sub && A.sub_dir[j] == 0u);
      bwd[j] = (uint8_t)(sub && A.sub_dir[j] != 0u);
      A.in_deg[nb + j] = 0u;
    }
    __syncthreads();
    const int64_t max_pass = 2 * n + 2;
    for (int64_t pass = 0;; ++pass) {
      if (threadIdx.x == 0) changed = 0u;
      __syncthreads();
      uint32_t ch = 0u;
      for (int64_t e = eb + threadIdx.x; e < ee; e += blockDim.x) {
        const uint32_t u = A.eu[e], v = A.ev[e];
        if ((int64_t)u >= n || (int64_t)v >= n) continue;  // dropped edge
        if (fwd[u] && !fwd[v]) {
          fwd[v] = 1;
          ch = 1u;
        }
        if (bwd[v] && !bwd[u]) {
          bwd[u] = 1;
          ch = 1u;
        }
      }
      if (ch) changed = 1u;
      __syncthreads();
      const uint32_t c = changed;
      __syncthreads();  // every thread has read it before the next pass clears it
      if (c == 0u) break;
      if (pass >= max_pass) {
        if (threadIdx.x == 0) atomicOr(A.err, kNetErrPasses);
        break;
      }
    }
    uint32_t kn = 0u, ke = 0u;
    for (int64_t j = (int64_t)A.n_sub + threadIdx.x; j < n; j += blockDim.x)
      kn += (fwd[j] && bwd[j]) ? 1u : 0u;
    for (int64_t e = eb + threadIdx.x; e < ee; e += blockDim.x) {
      const uint32_t u = A.eu[e], v = A.ev[e];
      if ((int64_t)u >= n || (int64_t)v >= n) continue;
      if (fwd[u] && bwd[v]) {
        ++ke;
        atomicAdd(A.in_deg + nb + v, 1u);
      }
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
// One workgroup per genome: kept numbers in raw order, the kept nodes' first incoming edge, then
// the kept hidden nodes' heap cells.
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
        A.new_id[nb + j] = keep ? id : kNoNode;
        if (keep) {
          if (NB + id >= NE) {
            atomicOr(A.err, kNetErrIndex);
          } else {
            A.in_offset[NB + id] = EB + run_deg + ed;
            if (j < (int64_t)A.n_sub) A.node_cell[NB + id] = kNoNode;
          }
        }
      }
      run_id += tk;
      run_deg += td;
    }
    if (threadIdx.x == 0) {
      if (NB + run_id != NE || EB + run_deg != A.edge_offset[g + 1]) atomicOr(A.err, kNetErrIndex);
      if (g == A.n_genomes - 1) A.in_offset[NE] = A.edge_offset[g + 1];
    }
    __syncthreads();  // new_id of the whole genome before the cell pass
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
        const uint32_t id = A.new_id[nb + raw];
        if (id != kNoNode && NB + id < NE) A.node_cell[NB + id] = 32u * (uint32_t)w + b + 1u;
        ++raw;
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------------ incoming edges
// One workgroup per genome, its raw edges in tiles of kNetThreads in raw order: each kept edge
// goes to its destination's next free slot, its rank among the tile's earlier edges with the same
// destination deciding the order within the tile, so every destination's edges stay in raw order.
__global__ void __launch_bounds__(kNetThreads) k_net_place(NetPlaceArgs A) {
  __shared__ uint32_t keys[kNetThreads];
  for (uint32_t g = blockIdx.x; g < A.n_genomes; g += gridDim.x) {
    const int64_t nb = A.raw_node[g], n = A.raw_node[g + 1] - nb;
    const int64_t eb = A.raw_edge[g], ee = A.raw_edge[g + 1];
    const int64_t NB = A.node_offset[g], NE = A.node_offset[g + 1];
    for (int64_t base = eb; base < ee; base += kNetThreads) {
      const int64_t e = base + threadIdx.x;
      uint32_t key = kNoNode, src = 0u;
      float w = 0.0f;
      if (e < ee) {
        const uint32_t u = A.eu[e], v = A.ev[e];
        if ((int64_t)u < n && (int64_t)v < n && A.fwd[nb + u] && A.bwd[nb + v]) {
          const uint32_t nu = A.new_id[nb + u], nv = A.new_id[nb + v];
          if (nu == kNoNode || nv == kNoNode || NB + nv >= NE || NB + nu >= NE) {
            atomicOr(A.err, kNetErrIndex);
          } else {
            key = nv;
            src = nu;
            w = A.ew[e];
          }
        }
      }
      keys[threadIdx.x] = key;
      __syncthreads();
      uint32_t rank = 0u;
      bool last = true;
      if (key != kNoNode) {
        for (uint32_t t = 0; t < kNetThreads; ++t) {
          if (keys[t] != key) continue;
          if (t < threadIdx.x) ++rank;
          else if (t > threadIdx.x) last = false;
        }
        const int64_t slot = A.in_offset[NB + key] + A.cursor[NB + key] + rank;
        if (slot < A.in_offset[NB + key] || slot >= A.in_offset[NB + key + 1] || slot >= A.edges) {
          atomicOr(A.err, kNetErrIndex);
        } else {
          A.in_src[slot] = (uint32_t)(NB + src);
          A.in_w[slot] = w;
        }
      }
      __syncthreads();  // every cursor read of this tile precedes the updates
      if (key != kNoNode && last) A.cursor[NB + key] += rank + 1u;
      __syncthreads();  // updates and `keys` before the next tile
    }
  }
}

// ------------------------------------------------------------------------ activation
// One workgroup per (genome, block of 4 patterns); node states as float4 (one pattern per
// component) in two global buffers, swapped after each synchronous step. Input nodes hold their
// pattern values; every other node takes sigmoid(sum of w * source state) over its incoming
// edges in CSR order (fmaf chain).
__global__ void __launch_bounds__(kNetThreads) k_net_forward(NetForwardArgs A) {
  const uint32_t g = blockIdx.x / A.pblocks, pb = blockIdx.x % A.pblocks;
  if (g >= A.n_genomes) return;
  const int64_t NB = A.node_offset[g], n = A.node_offset[g + 1] - NB;
  float4* cur = reinterpret_cast<float4*>(A.state) + (int64_t)pb * A.nodes;
  float4* nxt = reinterpret_cast<float4*>(A.state) + ((int64_t)A.pblocks + pb) * A.nodes;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < (int64_t)A.n_sub && A.in_slot[i] >= 0) {
      float c[4];
#pragma unroll
      for (uint32_t q = 0; q < 4; ++q) {
        const uint32_t p = 4u * pb + q;
        c[q] = p < A.n_patterns ? A.patterns[(int64_t)p * A.n_inputs + A.in_slot[i]] : 0.0f;
      }
      v = make_float4(c[0], c[1], c[2], c[3]);
    }
    cur[NB + i] = v;
  }
  __syncthreads();
  for (uint32_t t = 0; t < A.steps; ++t) {
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
      float4 v;
      if (i < (int64_t)A.n_sub && A.in_slot[i] >= 0) {
        v = cur[NB + i];
      } else {
        float zx = 0.f, zy = 0.f, zz = 0.f, zw = 0.f;
        const int64_t e1 = A.in_offset[NB + i + 1];
        for (int64_t e = A.in_offset[NB + i]; e < e1; ++e) {
          const uint32_t s = A.in_src[e];
          if ((int64_t)s >= A.nodes) continue;
          const float w = A.in_w[e];
          const float4 x = cur[s];
          zx = fmaf(w, x.x, zx);
          zy = fmaf(w, x.y, zy);
          zz = fmaf(w, x.z, zz);
          zw = fmaf(w, x.w, zw);
        }
        v = make_float4(sigmoid_f(zx), sigmoid_f(zy), sigmoid_f(zz), sigmoid_f(zw));
      }
      nxt[NB + i] = v;
    }
    __syncthreads();
    float4* tmp = cur;
    cur = nxt;
    nxt = tmp;
  }
  for (int64_t i = threadIdx.x; i < (int64_t)A.n_sub && i < n; i += blockDim.x) {
    const int32_t o = A.out_slot[i];
    if (o < 0) continue;
    const float4 v = cur[NB + i];
    for (uint32_t q = 0; q < 4; ++q) {
      const uint32_t p = 4u * pb + q;
      if (p < A.n_patterns && A.outputs)
        A.outputs[((int64_t)g * A.n_patterns + p) * A.n_outputs + (uint32_t)o] = comp(v, q);
    }
    if (A.fitness && o == 0) {
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
}  // namespace

extern "C" hipError_t emr_launch_net(int step, const void* args, int64_t work, hipStream_t s) {
  using namespace emr;
  switch (step) {
    case 0: {
      const auto& A = *static_cast<const NetRankArgs*>(args);
      hipLaunchKernelGGL(k_net_rank, dim3(genome_blocks(A.n_genomes)), dim3(kNetThreads), 0, s, A);
      break;
    }
    case 1: {
      const auto& A = *static_cast<const NetEdgeArgs*>(args);
      if (A.total <= 0) return hipSuccess;
      int64_t b = (A.total + kNetThreads - 1) / kNetThreads;
      if (b > 16384) b = 16384;
      hipLaunchKernelGGL(k_net_edges, dim3((uint32_t)b), dim3(kNetThreads), 0, s, A);
      break;
    }
    case 2: {
      const auto& A = *static_cast<const NetPruneArgs*>(args);
      hipLaunchKernelGGL(k_net_prune, dim3(genome_blocks(A.n_genomes)), dim3(kNetThreads), 0, s, A);
      break;
    }
    case 3: {
      const auto& A = *static_cast<const NetNodeArgs*>(args);
      hipLaunchKernelGGL(k_net_nodes, dim3(genome_blocks(A.n_genomes)), dim3(kNetThreads), 0, s, A);
      break;
    }
    case 4: {
      const auto& A = *static_cast<const NetPlaceArgs*>(args);
      hipLaunchKernelGGL(k_net_place, dim3(genome_blocks(A.n_genomes)), dim3(kNetThreads), 0, s, A);
      break;
    }
    case 5: {
      const auto& A = *static_cast<const NetForwardArgs*>(args);
      if (work <= 0 || work > 0x7FFFFFFF) return hipErrorInvalidValue;  // workgroups
      hipLaunchKernelGGL(k_net_forward, dim3((uint32_t)work), dim3(kNetThreads), 0, s, A);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
