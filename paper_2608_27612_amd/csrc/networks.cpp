// Networks built from a population's discovered substrates, and their activation (the networks the
// experiments evaluate, Section 5: XOR over its four patterns, with the hidden-to-hidden
// connection type of Section 4's configurations).
//
// The host drives the phases through the library's own entry points: Phase 1 on the substrate
// sources (emr_discover), its hidden nodes (emr_hidden_sources, which also records every hidden
// cell in a per-genome bitmap) and expressed connections (emr_express); then each hidden-to-hidden
// phase queries the previous phase's new hidden nodes, up to the requested number of phases or
// until no genome finds a new one. The network kernels (network.hip) then number the nodes, map
// every expressed connection to an edge, prune to the input-to-output paths (passes over every
// edge of the population until one changes nothing) and group each kept node's incoming edges (a
// stable sort of the edges by destination). Every step synchronizes with the host where it needs
// a count.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/emr.h"
#include "network.h"

namespace emr {
emr_status set_error(emr_status st, const std::string& msg);
}
extern "C" hipError_t emr_launch_net(int step, const void* args, int64_t work, hipStream_t s);
extern "C" hipError_t emr_net_sort(void* tmp, size_t* bytes, const uint32_t* kin, uint32_t* kout,
                                   const uint32_t* vin, uint32_t* vout, uint32_t n, int bits,
                                   hipStream_t s);

namespace {

emr_status failf(emr_status st, const char* fmt, ...) {
  char b[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(b, sizeof b, fmt, ap);
  va_end(ap);
  return emr::set_error(st, b);
}

#define NET_HIP(call)                                                                          \
  do {                                                                                         \
    hipError_t e_ = (call);                                                                    \
    if (e_ != hipSuccess) return failf(EMR_E_DEVICE, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)
#define NET_TRY(call)              \
  do {                             \
    emr_status s_ = (call);        \
    if (s_ != EMR_OK) return s_;   \
  } while (0)

// Device memory of the network builds, kept for reuse: a build allocates and frees dozens of
// buffers whose sizes change little from one generation to the next, and a hipMalloc / hipFree
// pair costs about 0.1 ms. A freed buffer enters its device's cache with an event recorded on the
// stream that used it (no event when the caller has already waited for that work) and is handed
// out again once that event has completed, to a request of at most its size and more than half
// of it. At most kCacheBytes stay cached per device; a buffer beyond that is freed. Cached memory
// is held until the process ends.
constexpr size_t kCacheBytes = size_t(8) << 30;

struct CacheEntry {
  void* p;
  hipEvent_t ev;  // nullptr: idle
};
struct DevCache {
  std::mutex mu;
  std::map<int, std::multimap<size_t, CacheEntry>> blocks;
  std::map<int, size_t> held;
  std::vector<hipEvent_t> spare;
};
DevCache& dev_cache() {
  static DevCache* c = new DevCache;  // (never destroyed: cached buffers live as long as the process)
  return *c;
}

// A cached buffer of at least `bytes` on device `dev` whose last use has completed, or nullptr.
void* cache_take(int dev, size_t bytes, size_t* cap) {
  DevCache& C = dev_cache();
  std::lock_guard<std::mutex> lk(C.mu);
  auto& m = C.blocks[dev];
  for (auto it = m.lower_bound(bytes); it != m.end() && it->first / 2 < bytes; ++it) {
    if (it->second.ev) {
      const hipError_t q = hipEventQuery(it->second.ev);
      if (q != hipSuccess) {
        (void)hipGetLastError();  // (not ready is no error of the caller's)
        continue;
      }
      C.spare.push_back(it->second.ev);
    }
    void* p = it->second.p;
    *cap = it->first;
    C.held[dev] -= it->first;
    m.erase(it);
    return p;
  }
  return nullptr;
}

// Frees every cached buffer of `dev` (waiting for the last use of each).
void cache_flush(int dev) {
  DevCache& C = dev_cache();
  std::lock_guard<std::mutex> lk(C.mu);
  auto& m = C.blocks[dev];
  for (auto& kv : m) {
    if (kv.second.ev) {
      (void)hipEventSynchronize(kv.second.ev);
      C.spare.push_back(kv.second.ev);
    }
    (void)hipFree(kv.second.p);
  }
  m.clear();
  C.held[dev] = 0;
}

// Returns a buffer to the cache; `s` is the stream of its last use, or nullptr with `idle` when
// that use is known to have completed.
void cache_give(int dev, void* p, size_t cap, hipStream_t s, bool idle) {
  DevCache& C = dev_cache();
  std::unique_lock<std::mutex> lk(C.mu);
  if (C.held[dev] + cap > kCacheBytes) {
    lk.unlock();
    (void)hipFree(p);  // (waits for the device's outstanding work)
    return;
  }
  hipEvent_t ev = nullptr;
  if (!idle) {
    if (!C.spare.empty()) {
      ev = C.spare.back();
      C.spare.pop_back();
    } else if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      lk.unlock();
      (void)hipFree(p);
      return;
    }
    if (hipEventRecord(ev, s) != hipSuccess) {
      (void)hipGetLastError();
      C.spare.push_back(ev);
      lk.unlock();
      (void)hipFree(p);
      return;
    }
  }
  C.blocks[dev].emplace(cap, CacheEntry{p, ev});
  C.held[dev] += cap;
}

// A device allocation of a build or of the networks handle, from the cache.
struct Dev {
  void* p = nullptr;
  size_t bytes = 0;   // asked for
  size_t cap = 0;     // the buffer's size
  int dev = 0;
  hipStream_t s = nullptr;  // the stream its users run on
  Dev() = default;
  Dev(const Dev&) = delete;
  Dev& operator=(const Dev&) = delete;
  ~Dev() { reset(); }
  // Back to the cache, usable once the work queued on `s` so far has completed.
  void reset() { release(false); }
  // Back to the cache when the caller has waited for every use of the buffer.
  void reset_idle() { release(true); }
  void take(Dev& o) {
    reset();
    p = o.p;
    bytes = o.bytes;
    cap = o.cap;
    dev = o.dev;
    s = o.s;
    o.p = nullptr;
    o.bytes = o.cap = 0;
  }
  template <class T>
  T* as() const {
    return static_cast<T*>(p);
  }

 private:
  void release(bool idle) {
    if (p) cache_give(dev, p, cap, s, idle);
    p = nullptr;
    bytes = cap = 0;
  }
};

emr_status alloc(Dev& d, size_t bytes, const char* what, hipStream_t s) {
  d.reset();
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return failf(EMR_E_DEVICE, "networks: no current device");
  }
  const size_t want = bytes ? (bytes + 255) & ~size_t(255) : 256;
  size_t cap = 0;
  void* p = cache_take(dev, want, &cap);
  if (!p) {
    cap = want;
    if (hipMalloc(&p, want) != hipSuccess) {
      (void)hipGetLastError();
      cache_flush(dev);
      if (hipMalloc(&p, want) != hipSuccess) {
        (void)hipGetLastError();
        return failf(EMR_E_NOMEM, "networks: cannot allocate %zu bytes for %s", bytes, what);
      }
    }
  }
  d.p = p;
  d.bytes = bytes;
  d.cap = cap;
  d.dev = dev;
  d.s = s;
  return EMR_OK;
}

emr_status to_host(void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (bytes == 0) return EMR_OK;
  NET_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s));
  NET_HIP(hipStreamSynchronize(s));
  return EMR_OK;
}

emr_status to_device(void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (bytes == 0) return EMR_OK;
  NET_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s));
  return EMR_OK;
}

// One phase: its sources, discovery, and expressed connections.
struct Phase {
  std::vector<emr_source> sources;
  std::vector<int32_t> offs;  // per-genome sources (empty: the shared substrate)
  int64_t n_pairs = 0;
  Dev parent, w4, rcount, roffset;
  int64_t rcap = 0, rtotal = 0;
  Dev cell, w, ccount, coffset;
  int64_t ccap = 0, ctotal = 0;
  Dev src_cell;   // [sources] heap cells of the queried hidden nodes
  Dev src_offs;   // [n_genomes + 1] int64 copy of offs
  Dev ws;         // the discovery's workspace, released after the phase

  void release_idle() {
    for (Dev* d : {&parent, &w4, &rcount, &roffset, &cell, &w, &ccount, &coffset, &src_cell,
                   &src_offs, &ws})
      d->reset_idle();
  }

  bool shared() const { return offs.empty(); }
  const int32_t* offs_ptr() const { return offs.empty() ? nullptr : offs.data(); }
  int32_t n_shared() const { return offs.empty() ? (int32_t)sources.size() : 0; }
  emr_result result() const {
    emr_result r;
    r.parent = parent.as<uint32_t>();
    r.w4 = w4.as<float>();
    r.capacity = rcap;
    r.pair_count = rcount.as<int64_t>();
    r.pair_offset = roffset.as<int64_t>();
    r.workspace = ws.p;
    r.workspace_bytes = (int64_t)ws.bytes;
    return r;
  }
};

}  // namespace

struct emr_networks {
  int device = 0;
  int32_t n_genomes = 0, n_sub = 0, n_in = 0, n_out = 0, depth = 0;
  int64_t words = 0;
  std::vector<emr_source> substrate;
  std::vector<int32_t> slots;  // in_slot[n_sub], then out_slot[n_sub]
  std::vector<std::unique_ptr<Phase>> phases;
  Dev known;
  Dev node_offset, node_cell, node_in, in_offset, in_src, in_w, d_slots;
  Dev d_out_node;  // [n_out] substrate index of output o
  int64_t nodes = 0, edges = 0;
  Dev state, patterns;
  // pinned staging of an activation's patterns and targets, and the event of its last copy
  void* pin = nullptr;
  size_t pin_bytes = 0;
  hipEvent_t pin_done = nullptr;
  bool pin_pending = false;
  // the end of the last activation (its outputs written)
  hipEvent_t done = nullptr;
  bool done_pending = false;
  // The build synchronized with its stream before the handle was returned (or, failing, before
  // the handle was destroyed), and the last activation is waited for here: every buffer is idle.
  ~emr_networks() {
    if (done) {
      if (done_pending) (void)hipEventSynchronize(done);
      (void)hipEventDestroy(done);
    }
    if (pin_done) {
      if (pin_pending) (void)hipEventSynchronize(pin_done);
      (void)hipEventDestroy(pin_done);
    }
    if (pin) (void)hipHostFree(pin);
    for (auto& ph : phases) ph->release_idle();
    for (Dev* d : {&known, &node_offset, &node_cell, &node_in, &in_offset, &in_src, &in_w,
                   &d_slots, &d_out_node, &state, &patterns})
      d->reset_idle();
  }
};

namespace {

struct Build {
  const emr_population* pop;
  emr_networks* net;
  float theta;
  int32_t type_mask;
  float w_min;
  hipStream_t s;
};

// The phase's discovery, retried once with the exact capacity when the first guess was short.
emr_status discover_phase(Build& B, Phase& P) {
  emr_networks& N = *B.net;
  const emr_source* src = P.sources.data();
  const int32_t n = (int32_t)P.sources.size();
  P.n_pairs = P.shared() ? (int64_t)N.n_genomes * n : P.offs[N.n_genomes];
  NET_TRY(alloc(P.rcount, (size_t)P.n_pairs * 8, "pair counts", B.s));
  NET_TRY(alloc(P.roffset, (size_t)(P.n_pairs + 1) * 8, "pair offsets", B.s));
  int64_t n_pos = 0, Q = 0;
  NET_TRY(emr_grid_count(N.depth, &n_pos, &Q));
  // A first guess of 16M records (320 MB) holds the kept cells of every workload measured here,
  // so the retry (which runs the phase's discovery a second time) stays the exception.
  int64_t cap = P.n_pairs * Q;
  if (cap > (int64_t)1 << 24) cap = (int64_t)1 << 24;
  if (cap < 1) cap = 1;
  for (int attempt = 0;; ++attempt) {
    int64_t wsb = 0;
    NET_TRY(emr_workspace_bytes(B.pop, src, n, P.offs_ptr(), P.n_shared(), N.depth, cap, &wsb));
    NET_TRY(alloc(P.ws, (size_t)wsb, "discover workspace", B.s));
    NET_TRY(alloc(P.parent, (size_t)cap * 4, "records", B.s));
    NET_TRY(alloc(P.w4, (size_t)cap * 16, "records", B.s));
    P.rcap = cap;
    const emr_result r = P.result();
    NET_TRY(emr_discover(B.pop, src, n, P.offs_ptr(), P.n_shared(), N.depth, B.theta, &r, B.s));
    int64_t total = 0;
    const emr_status st = emr_result_check(&r, &total, nullptr, B.s);
    if (st == EMR_OK) {
      P.rtotal = total;
      return EMR_OK;
    }
    if (st != EMR_E_CAPACITY || attempt > 0) return st;
    cap = total;
  }
}

// The phase's new hidden nodes (or-ed into the bitmap); on return *out holds them for the next
// phase: host sources and offsets, device cells and offsets.
emr_status hidden_phase(Build& B, Phase& P, Phase* next, int64_t* n_new) {
  emr_networks& N = *B.net;
  const int64_t cap = P.rtotal * 4 > 0 ? P.rtotal * 4 : 1;  // every record adds 4 cells at most
  int64_t hb = 0;
  NET_TRY(emr_hidden_workspace_bytes(N.n_genomes, N.depth, &hb));
  Dev hws, hsrc, hcell, hoff;
  NET_TRY(alloc(hws, (size_t)hb, "hidden-node workspace", B.s));
  NET_TRY(alloc(hsrc, (size_t)cap * sizeof(emr_source), "hidden sources", B.s));
  NET_TRY(alloc(hcell, (size_t)cap * 4, "hidden cells", B.s));
  NET_TRY(alloc(hoff, (size_t)(N.n_genomes + 1) * 8, "hidden offsets", B.s));
  emr_hidden h;
  h.sources = hsrc.as<emr_source>();
  h.cell = hcell.as<uint32_t>();
  h.capacity = cap;
  h.offsets = hoff.as<int64_t>();
  h.known = N.known.as<uint32_t>();
  h.workspace = hws.p;
  h.workspace_bytes = hb;
  const emr_result r = P.result();
  NET_TRY(emr_hidden_sources(B.pop, P.sources.data(), (int32_t)P.sources.size(), P.offs_ptr(),
                             P.n_shared(), N.depth, &r, &h, B.s));
  int64_t total = 0;
  NET_TRY(emr_call_check(hws.p, cap, &total, nullptr, B.s));
  *n_new = total;
  if (!next || total == 0) return EMR_OK;
  if (total > INT32_MAX) return failf(EMR_E_LIMIT, "networks: %lld hidden sources in one phase",
                                      (long long)total);
  next->sources.resize((size_t)total);
  std::vector<int64_t> off((size_t)N.n_genomes + 1);
  NET_TRY(to_host(next->sources.data(), hsrc.p, (size_t)total * sizeof(emr_source), B.s));
  NET_TRY(to_host(off.data(), hoff.p, off.size() * 8, B.s));
  next->offs.resize(off.size());
  for (size_t g = 0; g < off.size(); ++g) next->offs[g] = (int32_t)off[g];
  next->src_cell.take(hcell);
  next->src_offs.take(hoff);
  return EMR_OK;
}

emr_status express_phase(Build& B, Phase& P) {
  emr_networks& N = *B.net;
  P.ccap = P.rtotal * 4 > 0 ? P.rtotal * 4 : 1;  // four children per record at most
  int64_t eb = 0;
  NET_TRY(emr_express_workspace_bytes(P.n_pairs, &eb));
  Dev cws;
  NET_TRY(alloc(cws, (size_t)eb, "connection workspace", B.s));
  NET_TRY(alloc(P.cell, (size_t)P.ccap * 4, "connections", B.s));
  NET_TRY(alloc(P.w, (size_t)P.ccap * 4, "connections", B.s));
  NET_TRY(alloc(P.ccount, (size_t)P.n_pairs * 8, "connection counts", B.s));
  NET_TRY(alloc(P.coffset, (size_t)(P.n_pairs + 1) * 8, "connection offsets", B.s));
  emr_connections c;
  c.cell = P.cell.as<uint32_t>();
  c.w = P.w.as<float>();
  c.capacity = P.ccap;
  c.pair_count = P.ccount.as<int64_t>();
  c.pair_offset = P.coffset.as<int64_t>();
  c.workspace = cws.p;
  c.workspace_bytes = eb;
  const emr_result r = P.result();
  NET_TRY(emr_express(B.pop, P.sources.data(), (int32_t)P.sources.size(), P.offs_ptr(),
                      P.n_shared(), N.depth, &r, B.type_mask, B.w_min, &c, B.s));
  NET_TRY(emr_call_check(cws.p, P.ccap, &P.ctotal, nullptr, B.s));
  return EMR_OK;
}

emr_status assemble(Build& B) {
  emr_networks& N = *B.net;
  const uint32_t G = (uint32_t)N.n_genomes;
  const hipStream_t s = B.s;
  Dev rank, hidden, err;
  NET_TRY(alloc(rank, (size_t)G * (size_t)N.words * 4, "bitmap ranks", s));
  NET_TRY(alloc(hidden, (size_t)G * 4, "hidden counts", s));
  NET_TRY(alloc(err, 8, "error and pass words", s));
  NET_HIP(hipMemsetAsync(err.p, 0, 8, s));
  uint32_t* d_err = err.as<uint32_t>();
  uint32_t* d_changed = d_err + 1;
  emr::NetRankArgs ra{N.known.as<uint32_t>(), rank.as<uint32_t>(), hidden.as<uint32_t>(), N.words,
                      G};
  NET_HIP(emr_launch_net(0, &ra, 0, s));
  std::vector<uint32_t> hid(G);
  NET_TRY(to_host(hid.data(), hidden.p, (size_t)G * 4, s));
  std::vector<int64_t> raw_node(G + 1, 0);
  for (uint32_t g = 0; g < G; ++g) raw_node[g + 1] = raw_node[g] + N.n_sub + hid[g];
  // raw edges: genome by genome, each genome's phases in order
  const size_t K = N.phases.size();
  std::vector<std::vector<int64_t>> len(K, std::vector<int64_t>(G));
  for (size_t k = 0; k < K; ++k) {
    Phase& P = *N.phases[k];
    std::vector<int64_t> off((size_t)P.n_pairs + 1);
    NET_TRY(to_host(off.data(), P.coffset.p, off.size() * 8, s));
    for (uint32_t g = 0; g < G; ++g) {
      const int64_t p0 = P.shared() ? (int64_t)g * N.n_sub : P.offs[g];
      const int64_t p1 = P.shared() ? (int64_t)(g + 1) * N.n_sub : P.offs[g + 1];
      len[k][g] = off[p1] - off[p0];
    }
  }
  std::vector<int64_t> raw_edge(G + 1, 0);
  std::vector<std::vector<int64_t>> seg(K, std::vector<int64_t>(G));
  for (uint32_t g = 0; g < G; ++g) {
    int64_t e = raw_edge[g];
    for (size_t k = 0; k < K; ++k) {
      seg[k][g] = e;
      e += len[k][g];
    }
    raw_edge[g + 1] = e;
  }
  const int64_t n_raw = raw_node[G], e_raw = raw_edge[G];
  // raw node and edge numbers are u32 (kNoNode, the largest, marks a dropped edge)
  if (n_raw >= (int64_t)emr::kNoNode)
    return failf(EMR_E_LIMIT, "networks: %lld raw nodes (at most 2^32 - 2)", (long long)n_raw);
  if (e_raw >= (int64_t)emr::kNoNode)
    return failf(EMR_E_LIMIT, "networks: %lld raw edges (at most 2^32 - 2)", (long long)e_raw);
  Dev d_raw_node, d_raw_edge, d_dir, eu, ev, ew, fwd, bwd, in_deg, kept_n, kept_e;
  std::vector<Dev> d_seg(K);
  NET_TRY(alloc(d_raw_node, (size_t)(G + 1) * 8, "node offsets", s));
  NET_TRY(alloc(d_raw_edge, (size_t)(G + 1) * 8, "edge offsets", s));
  NET_TRY(alloc(d_dir, (size_t)N.n_sub, "substrate directions", s));
  NET_TRY(alloc(eu, (size_t)e_raw * 4, "edges", s));
  NET_TRY(alloc(ev, (size_t)e_raw * 4, "edges", s));
  NET_TRY(alloc(ew, (size_t)e_raw * 4, "edges", s));
  NET_TRY(alloc(fwd, (size_t)n_raw, "node flags", s));
  NET_TRY(alloc(bwd, (size_t)n_raw, "node flags", s));
  NET_TRY(alloc(in_deg, (size_t)n_raw * 4, "in-degrees", s));
  NET_TRY(alloc(kept_n, (size_t)G * 4, "kept counts", s));
  NET_TRY(alloc(kept_e, (size_t)G * 4, "kept counts", s));
  std::vector<uint8_t> dir(N.n_sub);
  for (int32_t j = 0; j < N.n_sub; ++j) dir[j] = N.substrate[j].dir == EMR_DIR_OUT ? 0 : 1;
  NET_TRY(to_device(d_raw_node.p, raw_node.data(), raw_node.size() * 8, s));
  NET_TRY(to_device(d_raw_edge.p, raw_edge.data(), raw_edge.size() * 8, s));
  NET_TRY(to_device(d_dir.p, dir.data(), dir.size(), s));
  for (size_t k = 0; k < K; ++k) {
    Phase& P = *N.phases[k];
    NET_TRY(alloc(d_seg[k], (size_t)G * 8, "phase segments", s));
    NET_TRY(to_device(d_seg[k].p, seg[k].data(), (size_t)G * 8, s));
    emr::NetEdgeArgs ea{};
    ea.conn_offset = P.coffset.as<int64_t>();
    ea.conn_cell = P.cell.as<uint32_t>();
    ea.conn_w = P.w.as<float>();
    ea.n_pairs = P.n_pairs;
    ea.total = P.ctotal;
    ea.src_offsets = P.shared() ? nullptr : P.src_offs.as<int64_t>();
    ea.src_cell = P.shared() ? nullptr : P.src_cell.as<uint32_t>();
    ea.sub_dir = d_dir.as<uint8_t>();
    ea.n_sub = (uint32_t)N.n_sub;
    ea.n_genomes = G;
    ea.known = N.known.as<uint32_t>();
    ea.rank = rank.as<uint32_t>();
    ea.words = N.words;
    ea.seg = d_seg[k].as<int64_t>();
    ea.raw_edge = d_raw_edge.as<int64_t>();
    ea.raw_node = d_raw_node.as<int64_t>();
    ea.eu = eu.as<uint32_t>();
    ea.ev = ev.as<uint32_t>();
    ea.ew = ew.as<float>();
    ea.err = d_err;
    NET_HIP(emr_launch_net(1, &ea, 0, s));
  }
  // pruning: flags, then passes over every edge until one changes nothing
  emr::NetFlagArgs fa{d_dir.as<uint8_t>(), d_raw_node.as<int64_t>(), fwd.as<uint8_t>(),
                      bwd.as<uint8_t>(), in_deg.as<uint32_t>(), kept_n.as<uint32_t>(),
                      kept_e.as<uint32_t>(), (uint32_t)N.n_sub, G};
  NET_HIP(emr_launch_net(2, &fa, 0, s));
  emr::NetReachArgs rr{eu.as<uint32_t>(), ev.as<uint32_t>(), fwd.as<uint8_t>(), bwd.as<uint8_t>(),
                       in_deg.as<uint32_t>(), d_changed, e_raw, n_raw};
  // a pass that changes something sets at least one more flag: 2 n_raw passes bound the loop
  const int64_t max_pass = 2 * n_raw + 2;
  for (int64_t pass = 0;; ++pass) {
    if (pass > max_pass)
      return failf(EMR_E_DEVICE, "networks: pruning did not settle in %lld passes",
                   (long long)max_pass);
    NET_HIP(hipMemsetAsync(d_changed, 0, 4, s));
    NET_HIP(emr_launch_net(3, &rr, 0, s));
    uint32_t ch = 0;
    NET_TRY(to_host(&ch, d_changed, 4, s));
    if (ch == 0) break;
  }
  NET_HIP(emr_launch_net(4, &rr, 0, s));
  NET_HIP(emr_launch_net(5, &fa, 0, s));
  std::vector<uint32_t> kn(G), ke(G);
  NET_TRY(to_host(kn.data(), kept_n.p, (size_t)G * 4, s));
  NET_TRY(to_host(ke.data(), kept_e.p, (size_t)G * 4, s));
  std::vector<int64_t> node_off(G + 1, 0), edge_off(G + 1, 0);
  for (uint32_t g = 0; g < G; ++g) {
    node_off[g + 1] = node_off[g] + N.n_sub + kn[g];
    edge_off[g + 1] = edge_off[g] + ke[g];
  }
  N.nodes = node_off[G];
  N.edges = edge_off[G];
  if (N.nodes >= (int64_t)emr::kNoNode)
    return failf(EMR_E_LIMIT, "networks: %lld nodes in all (at most 2^32 - 2)", (long long)N.nodes);
  if (N.edges > e_raw)
    return failf(EMR_E_DEVICE, "networks: %lld kept edges of %lld", (long long)N.edges,
                 (long long)e_raw);
  Dev d_edge_off, gid;
  NET_TRY(alloc(N.node_offset, (size_t)(G + 1) * 8, "network node offsets", s));
  NET_TRY(alloc(d_edge_off, (size_t)(G + 1) * 8, "network edge offsets", s));
  NET_TRY(alloc(N.node_cell, (size_t)N.nodes * 4, "network nodes", s));
  NET_TRY(alloc(N.node_in, (size_t)N.nodes * 4, "network input numbers", s));
  NET_TRY(alloc(N.in_offset, (size_t)(N.nodes + 1) * 8, "network edge offsets", s));
  NET_TRY(alloc(N.in_src, (size_t)N.edges * 4, "network edges", s));
  NET_TRY(alloc(N.in_w, (size_t)N.edges * 4, "network edges", s));
  NET_TRY(alloc(gid, (size_t)n_raw * 4, "node numbers", s));
  NET_TRY(to_device(N.node_offset.p, node_off.data(), node_off.size() * 8, s));
  NET_TRY(to_device(d_edge_off.p, edge_off.data(), edge_off.size() * 8, s));
  emr::NetNodeArgs na{N.known.as<uint32_t>(), rank.as<uint32_t>(), N.words,
                      d_raw_node.as<int64_t>(), fwd.as<uint8_t>(), bwd.as<uint8_t>(),
                      in_deg.as<uint32_t>(), N.d_slots.as<int32_t>(),
                      N.node_offset.as<int64_t>(), d_edge_off.as<int64_t>(), gid.as<uint32_t>(),
                      N.node_cell.as<uint32_t>(), N.node_in.as<int32_t>(),
                      N.in_offset.as<int64_t>(), d_err, (uint32_t)N.n_sub, G};
  NET_HIP(emr_launch_net(6, &na, 0, s));
  // kept edges grouped by destination, each group in raw order: a stable sort by destination
  if (N.edges > 0) {
    Dev keys, vals, skeys, svals, tmp;
    NET_TRY(alloc(keys, (size_t)e_raw * 4, "edge keys", s));
    NET_TRY(alloc(vals, (size_t)e_raw * 4, "edge keys", s));
    NET_TRY(alloc(skeys, (size_t)e_raw * 4, "edge keys", s));
    NET_TRY(alloc(svals, (size_t)e_raw * 4, "edge keys", s));
    emr::NetKeyArgs ka{eu.as<uint32_t>(), ev.as<uint32_t>(), fwd.as<uint8_t>(), bwd.as<uint8_t>(),
                       gid.as<uint32_t>(), keys.as<uint32_t>(), vals.as<uint32_t>(), e_raw, n_raw,
                       (uint32_t)N.nodes, d_err};
    NET_HIP(emr_launch_net(7, &ka, 0, s));
    int bits = 1;
    while (bits < 32 && ((uint64_t)1 << bits) <= (uint64_t)N.nodes) ++bits;  // keys <= nodes
    size_t tb = 0;
    NET_HIP(emr_net_sort(nullptr, &tb, keys.as<uint32_t>(), skeys.as<uint32_t>(),
                         vals.as<uint32_t>(), svals.as<uint32_t>(), (uint32_t)e_raw, bits, s));
    NET_TRY(alloc(tmp, tb, "sort storage", s));
    NET_HIP(emr_net_sort(tmp.p, &tb, keys.as<uint32_t>(), skeys.as<uint32_t>(),
                         vals.as<uint32_t>(), svals.as<uint32_t>(), (uint32_t)e_raw, bits, s));
    emr::NetGatherArgs ga{skeys.as<uint32_t>(), svals.as<uint32_t>(), eu.as<uint32_t>(),
                          ew.as<float>(), gid.as<uint32_t>(), N.in_offset.as<int64_t>(),
                          N.in_src.as<uint32_t>(), N.in_w.as<float>(), N.edges, e_raw, n_raw,
                          N.nodes, d_err};
    NET_HIP(emr_launch_net(8, &ga, 0, s));
    uint32_t e = 0;
    NET_TRY(to_host(&e, d_err, 4, s));  // (the sort's buffers are released after this sync)
    if (e != 0)
      return failf(EMR_E_DEVICE, "networks: a network kernel flagged an internal error (0x%x)", e);
    return EMR_OK;
  }
  uint32_t e = 0;
  NET_TRY(to_host(&e, d_err, 4, s));
  if (e != 0)
    return failf(EMR_E_DEVICE, "networks: a network kernel flagged an internal error (0x%x)", e);
  return EMR_OK;
}

emr_status run_forward(const emr_networks* N, const float* patterns, int32_t n_patterns,
                       int32_t steps, float* outputs, float* fitness, const float* targets,
                       hipStream_t s) {
  emr_networks& M = const_cast<emr_networks&>(*N);
  int dev = 0;
  NET_HIP(hipGetDevice(&dev));
  if (dev != N->device)
    return failf(EMR_E_INVAL, "networks: built on device %d, current device is %d", N->device, dev);
  const int64_t pblocks = (n_patterns + 3) / 4;
  if (pblocks * (N->nodes ? N->nodes : 1) > ((int64_t)1 << 40))
    return failf(EMR_E_LIMIT, "networks: too many nodes x patterns");
  // two state buffers of [pblocks][nodes] float4
  const size_t half = (size_t)pblocks * (size_t)(N->nodes ? N->nodes : 1) * 16;
  if (M.state.bytes < 2 * half) NET_TRY(alloc(M.state, 2 * half, "node states", s));
  // patterns, then targets, staged in pinned memory and copied on the stream; the staging is
  // rewritten only after the previous call's copy has completed
  const size_t pat_bytes = (size_t)n_patterns * (size_t)N->n_in * 4;
  const size_t tgt_bytes = targets ? (size_t)n_patterns * 4 : 0;
  const size_t need = pat_bytes + tgt_bytes;
  if (!M.pin_done) NET_HIP(hipEventCreateWithFlags(&M.pin_done, hipEventDisableTiming));
  if (M.pin_pending) NET_HIP(hipEventSynchronize(M.pin_done));
  M.pin_pending = false;
  if (M.pin_bytes < need || !M.pin) {
    if (M.pin) (void)hipHostFree(M.pin);
    M.pin = nullptr;
    M.pin_bytes = 0;
    if (hipHostMalloc(&M.pin, need ? need : 16, hipHostMallocDefault) != hipSuccess) {
      M.pin = nullptr;
      (void)hipGetLastError();
      return failf(EMR_E_NOMEM, "networks: cannot allocate %zu bytes of pinned staging", need);
    }
    M.pin_bytes = need ? need : 16;
  }
  if (M.patterns.bytes < need || !M.patterns.p) NET_TRY(alloc(M.patterns, need, "input patterns", s));
  std::memcpy(M.pin, patterns, pat_bytes);
  if (tgt_bytes) std::memcpy(static_cast<char*>(M.pin) + pat_bytes, targets, tgt_bytes);
  NET_HIP(hipMemcpyAsync(M.patterns.p, M.pin, need, hipMemcpyHostToDevice, s));
  NET_HIP(hipEventRecord(M.pin_done, s));
  M.pin_pending = true;
  float* buf[2] = {M.state.as<float>(), reinterpret_cast<float*>(M.state.as<char>() + half)};
  emr::NetStateArgs sa{N->node_in.as<int32_t>(), M.patterns.as<float>(), buf[0], N->nodes,
                       (uint32_t)N->n_in, (uint32_t)n_patterns, (uint32_t)pblocks};
  NET_HIP(emr_launch_net(9, &sa, 0, s));
  int cur = 0;
  for (int32_t t = 0; t < steps; ++t, cur ^= 1) {
    emr::NetStepArgs st{N->node_in.as<int32_t>(), N->in_offset.as<int64_t>(),
                        N->in_src.as<uint32_t>(), N->in_w.as<float>(), buf[cur], buf[cur ^ 1],
                        N->nodes, (uint32_t)pblocks};
    NET_HIP(emr_launch_net(10, &st, 0, s));
  }
  emr::NetOutArgs oa{};
  oa.node_offset = N->node_offset.as<int64_t>();
  oa.out_node = N->d_out_node.as<int32_t>();
  oa.state = buf[cur];
  oa.targets = targets ? reinterpret_cast<const float*>(M.patterns.as<char>() + pat_bytes) : nullptr;
  oa.outputs = outputs;
  oa.fitness = fitness;
  oa.nodes = N->nodes;
  oa.n_genomes = (uint32_t)N->n_genomes;
  oa.n_outputs = (uint32_t)N->n_out;
  oa.n_patterns = (uint32_t)n_patterns;
  oa.pblocks = (uint32_t)pblocks;
  NET_HIP(emr_launch_net(11, &oa, 0, s));
  if (!M.done) NET_HIP(hipEventCreateWithFlags(&M.done, hipEventDisableTiming));
  NET_HIP(hipEventRecord(M.done, s));
  M.done_pending = true;
  return EMR_OK;
}

// Every phase and the assembly; synchronizes with the stream at the end.
emr_status build_all(Build& B, int32_t n_substrate, int32_t iterations) {
  emr_networks& N = *B.net;
  NET_TRY(alloc(N.known, (size_t)N.n_genomes * (size_t)N.words * 4, "hidden-cell bitmaps", B.s));
  NET_HIP(hipMemsetAsync(N.known.p, 0, N.known.bytes, B.s));
  NET_TRY(alloc(N.d_slots, N.slots.size() * 4, "substrate slots", B.s));
  NET_TRY(to_device(N.d_slots.p, N.slots.data(), N.slots.size() * 4, B.s));
  std::vector<int32_t> out_node((size_t)N.n_out);
  for (int32_t j = 0; j < n_substrate; ++j)
    if (N.slots[(size_t)n_substrate + j] >= 0) out_node[(size_t)N.slots[(size_t)n_substrate + j]] = j;
  NET_TRY(alloc(N.d_out_node, out_node.size() * 4, "output nodes", B.s));
  NET_TRY(to_device(N.d_out_node.p, out_node.data(), out_node.size() * 4, B.s));

  N.phases.push_back(std::make_unique<Phase>());
  N.phases[0]->sources = N.substrate;
  for (int32_t it = 0;; ++it) {
    Phase& P = *N.phases.back();
    NET_TRY(discover_phase(B, P));
    const bool more = it < iterations;
    auto next = more ? std::make_unique<Phase>() : nullptr;
    int64_t n_new = 0;
    NET_TRY(hidden_phase(B, P, next.get(), &n_new));
    NET_TRY(express_phase(B, P));
    P.ws.reset();
    if (!more || n_new == 0) break;
    N.phases.push_back(std::move(next));
  }
  NET_TRY(assemble(B));
  NET_HIP(hipStreamSynchronize(B.s));
  return EMR_OK;
}

constexpr int32_t kMaxSubstrate = 1024;
constexpr int32_t kMaxIterations = 64;
constexpr int32_t kMaxSteps = 1 << 20;
constexpr int32_t kMaxPatterns = 1 << 16;

}  // namespace

extern "C" {

emr_status emr_build_networks(const emr_population* pop, const emr_source* substrate,
                              int32_t n_substrate, int32_t depth, float theta, int32_t type_mask,
                              float w_min, int32_t iterations, emr_networks** out, void* stream) {
  if (!out) return failf(EMR_E_INVAL, "networks: out is NULL");
  *out = nullptr;
  if (!pop || !substrate) return failf(EMR_E_INVAL, "networks: NULL population or substrate");
  if (n_substrate < 1 || n_substrate > kMaxSubstrate)
    return failf(EMR_E_INVAL, "networks: n_substrate %d outside [1, %d]", n_substrate,
                 kMaxSubstrate);
  if (depth < 1 || depth > EMR_MAX_DEPTH)
    return failf(EMR_E_INVAL, "networks: depth %d outside [1, %d]", depth, EMR_MAX_DEPTH);
  if (type_mask < 1 || type_mask > EMR_CONN_ALL)
    return failf(EMR_E_INVAL, "networks: type_mask %d outside [1, 15]", type_mask);
  if (iterations < 0 || iterations > kMaxIterations)
    return failf(EMR_E_INVAL, "networks: iterations %d outside [0, %d]", iterations,
                 kMaxIterations);
  if (std::isnan(theta) || std::isnan(w_min))
    return failf(EMR_E_INVAL, "networks: theta and w_min must not be NaN");
  auto net = std::make_unique<emr_networks>();
  emr_networks& N = *net;
  N.n_sub = n_substrate;
  N.depth = depth;
  N.substrate.assign(substrate, substrate + n_substrate);
  N.slots.assign((size_t)2 * n_substrate, -1);
  for (int32_t j = 0; j < n_substrate; ++j) {
    const emr_source& q = substrate[j];
    if (q.dir != EMR_DIR_OUT && q.dir != EMR_DIR_IN)
      return failf(EMR_E_INVAL, "networks: substrate source %d has direction %d", j, q.dir);
    if (!std::isfinite(q.x) || !std::isfinite(q.y))
      return failf(EMR_E_INVAL, "networks: substrate source %d is not finite", j);
    if (q.dir == EMR_DIR_OUT) N.slots[j] = N.n_in++;
    else N.slots[(size_t)n_substrate + j] = N.n_out++;
  }
  if (N.n_in == 0 || N.n_out == 0)
    return failf(EMR_E_INVAL, "networks: the substrate needs an input and an output");
  NET_TRY(emr_population_info(pop, &N.n_genomes, nullptr, nullptr, nullptr));
  if (N.n_genomes < 1) return failf(EMR_E_INVAL, "networks: empty population");
  NET_HIP(hipGetDevice(&N.device));
  NET_TRY(emr_cell_words(depth, &N.words));
  Build B{pop, &N, theta, type_mask, w_min, (hipStream_t)stream};
  const emr_status st = build_all(B, n_substrate, iterations);
  // after a failure, nothing queued may still use the buffers the handle gives back
  if (st != EMR_OK) {
    (void)hipStreamSynchronize(B.s);
    return st;
  }
  *out = net.release();
  return EMR_OK;
}

emr_status emr_networks_info(const emr_networks* net, emr_network_info* info) {
  if (!net || !info) return failf(EMR_E_INVAL, "networks: NULL argument");
  info->n_genomes = net->n_genomes;
  info->n_substrate = net->n_sub;
  info->n_inputs = net->n_in;
  info->n_outputs = net->n_out;
  info->depth = net->depth;
  info->phases = (int32_t)net->phases.size();
  info->nodes = net->nodes;
  info->edges = net->edges;
  info->node_offset = net->node_offset.as<int64_t>();
  info->node_cell = net->node_cell.as<uint32_t>();
  info->in_offset = net->in_offset.as<int64_t>();
  info->in_src = net->in_src.as<uint32_t>();
  info->in_w = net->in_w.as<float>();
  info->known = net->known.as<uint32_t>();
  info->known_words = net->words;
  return EMR_OK;
}

emr_status emr_networks_phase(const emr_networks* net, int32_t phase, emr_network_phase* out) {
  if (!net || !out) return failf(EMR_E_INVAL, "networks: NULL argument");
  if (phase < 0 || phase >= (int32_t)net->phases.size())
    return failf(EMR_E_INVAL, "networks: phase %d outside [0, %zu)", phase, net->phases.size());
  const Phase& P = *net->phases[phase];
  out->sources = P.sources.data();
  out->n_sources = (int32_t)P.sources.size();
  out->src_offsets = P.offs_ptr();
  out->src_cell = P.shared() ? nullptr : P.src_cell.as<uint32_t>();
  out->n_pairs = P.n_pairs;
  out->parent = P.parent.as<uint32_t>();
  out->w4 = P.w4.as<float>();
  out->pair_offset = P.roffset.as<int64_t>();
  out->records = P.rtotal;
  out->conn_cell = P.cell.as<uint32_t>();
  out->conn_w = P.w.as<float>();
  out->conn_offset = P.coffset.as<int64_t>();
  out->connections = P.ctotal;
  return EMR_OK;
}

emr_status emr_activate(const emr_networks* net, const float* inputs, int32_t n_patterns,
                        int32_t steps, float* outputs, void* stream) {
  if (!net || !outputs) return failf(EMR_E_INVAL, "networks: NULL argument");
  if (n_patterns < 1 || n_patterns > kMaxPatterns)
    return failf(EMR_E_INVAL, "networks: n_patterns %d outside [1, %d]", n_patterns, kMaxPatterns);
  if (steps < 0 || steps > kMaxSteps)
    return failf(EMR_E_INVAL, "networks: steps %d outside [0, %d]", steps, kMaxSteps);
  if (!inputs) return failf(EMR_E_INVAL, "networks: inputs is NULL");
  return run_forward(net, inputs, n_patterns, steps, outputs, nullptr, nullptr,
                     (hipStream_t)stream);
}

emr_status emr_xor_fitness(const emr_networks* net, int32_t bias_input, int32_t steps,
                           float* fitness, void* stream) {
  if (!net || !fitness) return failf(EMR_E_INVAL, "networks: NULL argument");
  if (steps < 0 || steps > kMaxSteps)
    return failf(EMR_E_INVAL, "networks: steps %d outside [0, %d]", steps, kMaxSteps);
  if (net->n_out != 1) return failf(EMR_E_INVAL, "networks: XOR needs one output");
  if (bias_input < -1 || bias_input >= net->n_in || net->n_in != 2 + (bias_input >= 0 ? 1 : 0))
    return failf(EMR_E_INVAL, "networks: XOR needs inputs a, b and at most one bias input "
                 "(%d inputs, bias input %d)", net->n_in, bias_input);
  // (a, b) = (0,0), (0,1), (1,0), (1,1) on the non-bias inputs in order; the bias input holds 1
  static const float ab[4][2] = {{0.f, 0.f}, {0.f, 1.f}, {1.f, 0.f}, {1.f, 1.f}};
  static const float target[4] = {0.f, 1.f, 1.f, 0.f};
  std::vector<float> pat((size_t)4 * net->n_in);
  for (int p = 0; p < 4; ++p) {
    int c = 0;
    for (int j = 0; j < net->n_in; ++j) pat[(size_t)p * net->n_in + j] = j == bias_input ? 1.f : ab[p][c++];
  }
  return run_forward(net, pat.data(), 4, steps, nullptr, fitness, target, (hipStream_t)stream);
}

emr_status emr_copy_to_host(void* host, const void* device, int64_t bytes, void* stream) {
  if (bytes < 0 || (bytes > 0 && (!host || !device)))
    return failf(EMR_E_INVAL, "copy: bad arguments");
  return to_host(host, device, (size_t)bytes, (hipStream_t)stream);
}

void emr_free_networks(emr_networks* net) { delete net; }

}  // extern "C"
