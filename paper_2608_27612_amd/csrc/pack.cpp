// Host-side packing of NEAT CPPN genomes into the kernels' program format.
//
// A genome's CPPN (Section 2: inputs x1, y1, x2, y2 and a constant 1) is evaluated by the GPU once
// per (source, grid position) (Section 3.1, the batched query W). For a fixed query direction only
// two inputs change from one grid position to the next, so each live node is classified as
// position-dependent ("varying") or constant per (genome, source) ("uniform"). The packer emits,
// per direction, the varying nodes as a straight program for the lane interpreter and the uniform
// nodes as a small program the bind kernel evaluates once per source, folding every uniform
// contribution into a per-step bias.
#include "pack.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <queue>
#include <utility>

namespace emr {

// Input scale of each activation for varying nodes: the packer multiplies every weight and bias
// that feeds a varying node by it, so the kernel's activation code starts from c z (see the record
// tails of the discover kernel): sigmoid and tanh need -log2 e and -2 log2 e (for 2^x), the
// gaussian sqrt(log2 e) (2^-(c z)^2 = e^-z^2), the sine 1 / (2 pi) (the hardware sine takes
// revolutions). Each scaled value is the product of the float weight and the exact constant,
// rounded once.
static double act_input_scale(int act) {
  const double log2e = 1.4426950408889634074;
  const double inv_2pi = 0.15915494309189533577;
  switch (act) {
    case EMR_ACT_SIGMOID: return -log2e;
    case EMR_ACT_TANH: return -2.0 * log2e;
    case EMR_ACT_GAUSS: return 1.2011224087864497555;  // sqrt(log2 e)
    case EMR_ACT_SINE: return inv_2pi;
    default: return 1.0;
  }
}
static float scaled(float w, double c) { return (float)((double)w * c); }

namespace {

struct Err {
  emr_status st;
  std::string msg;
};

bool fail(Err* e, emr_status st, const char* fmt, int a = 0, int b = 0) {
  char buf[256];
  std::snprintf(buf, sizeof buf, fmt, a, b);
  e->st = st;
  e->msg = buf;
  return false;
}

inline uint32_t fbits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return u;
}

struct Edge {
  int src, dst;
  float w;
};

// Validation of the raw genome against the rules stated with emr_genome.
bool validate(const emr_genome& g, Err* e) {
  if (g.n_nodes < 1 || g.n_nodes > EMR_MAX_NODES)
    return fail(e, EMR_E_LIMIT, "n_nodes=%d outside [1, %d]", g.n_nodes, EMR_MAX_NODES);
  if (g.n_edges < 0 || g.n_edges > EMR_MAX_EDGES)
    return fail(e, EMR_E_LIMIT, "n_edges=%d outside [0, %d]", g.n_edges, EMR_MAX_EDGES);
  if (!g.kind || !g.act) return fail(e, EMR_E_INVAL, "kind/act pointer is NULL");
  if (g.n_edges > 0 && (!g.src || !g.dst || !g.w))
    return fail(e, EMR_E_INVAL, "edge arrays are NULL with n_edges=%d", g.n_edges);
  int n_out = 0, role_seen[5] = {0, 0, 0, 0, 0};
  for (int v = 0; v < g.n_nodes; ++v) {
    int k = g.kind[v];
    if (k > EMR_NODE_OUTPUT) return fail(e, EMR_E_INVAL, "node %d has kind %d", v, k);
    if (k <= EMR_IN_BIAS) {
      if (role_seen[k]++) return fail(e, EMR_E_INVAL, "input role %d appears twice (node %d)", k, v);
    } else {
      if (g.act[v] > EMR_ACT_ABS) return fail(e, EMR_E_INVAL, "node %d has activation %d", v, g.act[v]);
      if (k == EMR_NODE_OUTPUT) n_out++;
    }
  }
  if (n_out != 1) return fail(e, EMR_E_INVAL, "%d output nodes (need exactly 1)", n_out);
  for (int i = 0; i < g.n_edges; ++i) {
    if (g.src[i] < 0 || g.src[i] >= g.n_nodes || g.dst[i] < 0 || g.dst[i] >= g.n_nodes)
      return fail(e, EMR_E_INVAL, "edge %d has an endpoint out of range", i);
    if (g.kind[g.dst[i]] <= EMR_IN_BIAS)
      return fail(e, EMR_E_INVAL, "edge %d enters input node %d", i, g.dst[i]);
  }
  return true;
}

}  // namespace

bool pack_genome(const emr_genome& g, std::vector<uint32_t>& blob, ProgDesc desc[2],
                 GenomeInfo info[2], emr_status* st, std::string* msg) {
  Err err{EMR_OK, ""};
  if (!validate(g, &err)) {
    *st = err.st;
    *msg = err.msg;
    return false;
  }
  const int n = g.n_nodes;
  std::vector<Edge> edges;  // enabled edges, in edge-list order
  edges.reserve(g.n_edges);
  for (int i = 0; i < g.n_edges; ++i)
    if (!g.enabled || g.enabled[i]) edges.push_back({g.src[i], g.dst[i], g.w[i]});

  // Kahn's algorithm; among ready nodes the lowest id goes first.
  std::vector<int> indeg(n, 0), order;
  std::vector<std::vector<int>> out_edges(n), in_edges(n);
  for (int i = 0; i < (int)edges.size(); ++i) {
    indeg[edges[i].dst]++;
    out_edges[edges[i].src].push_back(i);
    in_edges[edges[i].dst].push_back(i);
  }
  std::priority_queue<int, std::vector<int>, std::greater<int>> ready;
  for (int v = 0; v < n; ++v)
    if (indeg[v] == 0) ready.push(v);
  while (!ready.empty()) {
    int u = ready.top();
    ready.pop();
    order.push_back(u);
    for (int ei : out_edges[u])
      if (--indeg[edges[ei].dst] == 0) ready.push(edges[ei].dst);
  }
  if ((int)order.size() != n) {
    *st = EMR_E_CYCLE;
    *msg = "enabled edges contain a cycle";
    return false;
  }

  int out_node = -1;
  int role_node[5] = {-1, -1, -1, -1, -1};
  for (int v = 0; v < n; ++v) {
    if (g.kind[v] == EMR_NODE_OUTPUT) out_node = v;
    if (g.kind[v] <= EMR_IN_BIAS) role_node[g.kind[v]] = v;
  }
  // Live nodes: those with an enabled path to the output.
  std::vector<char> live(n, 0);
  {
    std::vector<int> stack{out_node};
    live[out_node] = 1;
    while (!stack.empty()) {
      int v = stack.back();
      stack.pop_back();
      for (int ei : in_edges[v]) {
        int s = edges[ei].src;
        if (!live[s]) {
          live[s] = 1;
          stack.push_back(s);
        }
      }
    }
  }

  for (int dir = 0; dir < 2; ++dir) {
    // Roles that vary with the grid position: (x2, y2) for outgoing queries, (x1, y1) incoming.
    const int vx_role = dir == EMR_DIR_OUT ? EMR_IN_X2 : EMR_IN_X1;
    const int vy_role = dir == EMR_DIR_OUT ? EMR_IN_Y2 : EMR_IN_Y1;
    std::vector<char> varying(n, 0);
    for (int v : order) {
      if (!live[v]) continue;
      int k = g.kind[v];
      if (k <= EMR_IN_BIAS) {
        varying[v] = (k == vx_role || k == vy_role);
        continue;
      }
      for (int ei : in_edges[v])
        if (live[edges[ei].src] && varying[edges[ei].src]) varying[v] = 1;
    }
    // Uniform value indices: U[0..4] = input roles, U[5 + k] = k-th uniform computed node.
    std::vector<int> uidx(n, -1);
    std::vector<int> unodes, vsteps;
    for (int v : order) {
      if (!live[v]) continue;
      if (g.kind[v] <= EMR_IN_BIAS) {
        if (!varying[v]) uidx[v] = g.kind[v];
        continue;
      }
      if (varying[v]) {
        vsteps.push_back(v);
      } else {
        uidx[v] = 5 + (int)unodes.size();
        unodes.push_back(v);
      }
    }
    const bool out_varying = varying[out_node] != 0;
    // Nodes reached from the source's coordinates: (x1, y1) for outgoing queries, (x2, y2)
    // incoming. Any other node takes the same value for every source at a position.
    const int sx_role = dir == EMR_DIR_OUT ? EMR_IN_X1 : EMR_IN_X2;
    const int sy_role = dir == EMR_DIR_OUT ? EMR_IN_Y1 : EMR_IN_Y2;
    std::vector<char> from_source(n, 0);
    for (int v : order) {
      if (!live[v]) continue;
      const int k = g.kind[v];
      if (k <= EMR_IN_BIAS) {
        from_source[v] = (k == sx_role || k == sy_role);
        continue;
      }
      for (int ei : in_edges[v])
        if (live[edges[ei].src] && from_source[edges[ei].src]) from_source[v] = 1;
    }

    // Register slots for varying computed nodes by liveness: a slot is freed after the last step
    // that reads it, before that step's own result is assigned.
    std::vector<int> step_of(n, -1), last_use(n, -1), slot(n, -1), assigned(n, -1);
    for (int t = 0; t < (int)vsteps.size(); ++t) step_of[vsteps[t]] = t;
    for (int t = 0; t < (int)vsteps.size(); ++t)
      for (int ei : in_edges[vsteps[t]]) {
        int s = edges[ei].src;
        if (live[s] && varying[s] && g.kind[s] > EMR_IN_BIAS) last_use[s] = t;
      }
    std::vector<int> free_slots;  // kept sorted descending so back() is the lowest
    int window = 0, next_slot = 0;
    for (int t = 0; t < (int)vsteps.size(); ++t) {
      int v = vsteps[t];
      for (int ei : in_edges[v]) {
        int s = edges[ei].src;
        if (slot[s] >= 0 && last_use[s] == t) {
          free_slots.push_back(slot[s]);
          slot[s] = -2;  // released (an edge list may name the same source twice)
        }
      }
      std::sort(free_slots.rbegin(), free_slots.rend());
      const bool is_output_step = out_varying && v == out_node;
      if (is_output_step) continue;  // the output stays in the accumulators
      int sl;
      if (!free_slots.empty()) {
        sl = free_slots.back();
        free_slots.pop_back();
      } else {
        sl = next_slot++;
      }
      slot[v] = sl;
      assigned[v] = sl;
      window = std::max(window, sl + 1);
    }
    // the declared limit is the kernels' widest register window (5-bit slot indices)
    static_assert(EMR_MAX_LIVE == kMaxWindow && kMaxWindow <= (1 << kSlotBits), "window limit");
    if (window > EMR_MAX_LIVE) {
      *st = EMR_E_LIMIT;
      char buf[128];
      std::snprintf(buf, sizeof buf, "needs %d live position-dependent values (limit %d)", window,
                    EMR_MAX_LIVE);
      *msg = buf;
      return false;
    }

    // ---- varying program: 16-word records (layout in emr_internal.h)
    ProgDesc& d = desc[dir];
    GenomeInfo& inf = info[dir];
    inf = GenomeInfo{};
    while (blob.size() % kRecWords) blob.push_back(0u);
    d.var_off = (uint32_t)blob.size();
    d.n_steps = (uint32_t)vsteps.size();
    d.flags = (out_varying ? 1u : 0u) | ((uint32_t)window << 8);
    d.pad[0] = d.pad[1] = 0;
    uint32_t n_rec = 0;
    std::vector<uint32_t> first_rec(vsteps.size(), 0);  // record index of each node's first record
    for (int t = 0; t < (int)vsteps.size(); ++t) {
      const int v = vsteps[t];
      first_rec[t] = n_rec;
      float ax = 0.0f, ay = 0.0f;
      int ax_edges = 0, ay_edges = 0;
      std::vector<std::pair<uint32_t, float>> node_edges;  // (source slot, w) in edge-list order
      for (int ei : in_edges[v]) {
        const Edge& E = edges[ei];
        if (!live[E.src] || !varying[E.src]) continue;  // uniform: folded by the bind kernel
        const int k = g.kind[E.src];
        if (k == vx_role) {
          ax += E.w;  // parallel edges from x add their weights
          inf.fma_xy++;
          ax_edges++;
        } else if (k == vy_role) {
          ay += E.w;
          inf.fma_xy++;
          ay_edges++;
        } else {
          node_edges.push_back({(uint32_t)assigned[E.src], E.w});
          inf.fma_node++;
        }
      }
      const bool is_out = out_varying && v == out_node;
      const bool shared = !is_out && !from_source[v];
      const uint32_t dst = is_out ? 0u : (uint32_t)assigned[v];
      const double c_act = act_input_scale(g.act[v]);
      const size_t ne = node_edges.size();
      const size_t n_chunks = ne == 0 ? 1 : (ne + kRecEdges - 1) / kRecEdges;
      for (size_t c = 0; c < n_chunks; ++c) {
        const size_t r = blob.size();
        blob.resize(r + kRecWords, 0u);
        const size_t k0 = c * kRecEdges, k1 = std::min(ne, k0 + kRecEdges);
        uint32_t meta = ((uint32_t)(k1 - k0) << kRecEdgeShift) | (dst << kRecDstShift);
        if (c == 0) {
          meta |= kRecFirst | (shared ? kRecShared : 0u);
          blob[r + 1] = fbits(scaled(ax, c_act));
          blob[r + 2] = fbits(scaled(ay, c_act));
        }
        if (c + 1 == n_chunks) meta |= (is_out ? kRecTailOutput : kRecTailStore) + g.act[v];
        blob[r] = meta;
        // The kernel runs a record's edges from position n - 1 down to 0, so the node's edges
        // go in reverse positions and are accumulated in edge-list order.
        for (size_t k = k0; k < k1; ++k) {
          const size_t e = k1 - 1 - k;
          blob[r + 3 + e / 6] |= node_edges[k].first << (kSlotBits * (e % 6));
          blob[r + 5 + e] = fbits(scaled(node_edges[k].second, c_act));
        }
        n_rec++;
      }
      inf.act_count[g.act[v]]++;
      if (shared) {
        inf.shared_edges += (ax_edges + ay_edges) + (int)ne;
        inf.shared_act_count[g.act[v]]++;
      }
    }
    d.n_rec = n_rec;
    inf.n_steps = (int)vsteps.size();
    inf.window = window;
    inf.out_varying = out_varying;

    // ---- uniform program
    d.uni_off = (uint32_t)blob.size();
    size_t ub = blob.size();
    blob.resize(ub + 4 + 4 * unodes.size() + 4 * vsteps.size(), 0u);
    blob[ub + 0] = (uint32_t)unodes.size();
    blob[ub + 1] = out_varying ? kNone : (uint32_t)uidx[out_node];
    blob[ub + 2] = (uint32_t)vsteps.size();
    for (int k = 0; k < (int)unodes.size(); ++k) {
      int v = unodes[k];
      uint32_t first = (uint32_t)blob.size(), cnt = 0;
      for (int ei : in_edges[v]) {
        const Edge& E = edges[ei];
        if (!live[E.src]) continue;
        blob.push_back((uint32_t)uidx[E.src]);
        blob.push_back(fbits(E.w));
        cnt++;
      }
      uint32_t* r = &blob[ub + 4 + 4 * k];
      r[0] = g.act[v];
      r[1] = cnt;
      r[2] = first - (uint32_t)ub;
      r[3] = fbits(g.bias ? g.bias[v] : 0.0f);
    }
    for (int t = 0; t < (int)vsteps.size(); ++t) {
      int v = vsteps[t];
      const double c_act = act_input_scale(g.act[v]);  // the fold feeds the scaled accumulator
      uint32_t first = (uint32_t)blob.size(), cnt = 0;
      for (int ei : in_edges[v]) {
        const Edge& E = edges[ei];
        if (!live[E.src] || varying[E.src]) continue;
        blob.push_back((uint32_t)uidx[E.src]);
        blob.push_back(fbits(scaled(E.w, c_act)));
        cnt++;
      }
      uint32_t* r = &blob[ub + 4 + 4 * unodes.size() + 4 * t];
      r[0] = cnt;
      r[1] = first - (uint32_t)ub;
      r[2] = fbits(scaled(g.bias ? g.bias[v] : 0.0f, c_act));
      r[3] = first_rec[t];
    }
    d.uni_end = (uint32_t)blob.size();
    inf.n_unodes = (int)unodes.size();
    inf.n_rec = (int)n_rec;
  }
  (void)role_node;
  return true;
}

}  // namespace emr
