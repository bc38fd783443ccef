// Host runtime behind include/emr.h: argument checks, packing, per-call planning (grouping the
// sources of a genome into the lanes' member sets), workspace layout, and kernel launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/emr.h"
#include "band.h"
#include "emr_internal.h"
#include "jit.h"
#include "pack.h"
#include "plan.h"
#include "sched.h"

// Launchers (kernels.hip).
extern "C" hipError_t emr_launch_fill(void* p, int64_t n_words, uint32_t value, hipStream_t s);
extern "C" hipError_t emr_launch_grid(float* xy, int64_t n, hipStream_t s);
extern "C" hipError_t emr_launch_bind(const emr::BindArgs* a, hipStream_t s);
extern "C" hipError_t emr_launch_discover(const emr::DiscoverArgs* a, int mode, uint32_t blocks,
                                          hipStream_t s, hipEvent_t start, hipEvent_t stop);
extern "C" hipError_t emr_launch_compact(const emr::ScanArgs* S, const emr::MoveArgs* M,
                                         hipStream_t s);
extern "C" hipError_t emr_launch_finalize(uint32_t* flags, uint32_t* host, hipStream_t s);
extern "C" hipError_t emr_launch_scan(const emr::ScanArgs* S, hipStream_t s);
extern "C" hipError_t emr_launch_hidden(const emr::HiddenArgs* A, int step, hipStream_t s);
extern "C" hipError_t emr_launch_express(const emr::ExpressArgs* A, int emit, hipStream_t s);
extern "C" hipError_t emr_launch_chain(const emr::ChainArgs* A, int step, hipStream_t s);
extern "C" hipError_t emr_launch_band(const emr::BandArgs* A, hipStream_t s);
extern "C" hipError_t emr_launch_band_select(const emr::BandSelectArgs* A, int emit,
                                              hipStream_t s);
extern "C" hipError_t emr_launch_tile_geo(uint32_t* out, uint32_t tiles, uint32_t rows,
                                          hipStream_t s);
extern "C" hipError_t emr_noalloc_scratch(void** out);
extern "C" int emr_discover_per_cu(int mode);
extern "C" hipError_t emr_discover_setup(const emr::DiscoverArgs* a, uint32_t blocks, int per_cu,
                                         int cus, emr::DiscoverScalars* out, uint32_t* grid);
// The compiled tier's template code object (jit_image.cpp).
extern "C" const uint8_t emr_jit_template_begin[], emr_jit_template_end[];

namespace {

thread_local std::string g_err;

emr_status fail(emr_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_OR_FAIL(call)                                                                    \
  do {                                                                                       \
    hipError_t e_ = (call);                                                                  \
    if (e_ != hipSuccess) return fail(EMR_E_DEVICE, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

using emr::align256;

// Compute units of the current device, queried once per device.
// Host worker threads for the library's parallel host work (packing, the compiled tier's
// translation), started on first use and kept for the process: run(n, f) calls f(0) .. f(n - 1)
// on the workers and the calling thread and returns when every call has returned. One job runs at
// a time (concurrent callers queue).
class WorkerPool {
 public:
  static WorkerPool& get() {
    static WorkerPool p;
    return p;
  }
  int size() const { return (int)workers_.size() + 1; }
  void run(int n, const std::function<void(int)>& f) {
    if (n <= 1 || workers_.empty()) {
      for (int i = 0; i < n; ++i) f(i);
      return;
    }
    std::lock_guard<std::mutex> one_job(job_mu_);
    {
      std::lock_guard<std::mutex> l(mu_);
      fn_ = &f;
      next_ = 0;
      n_ = n;
      done_ = 0;
      ++gen_;
    }
    cv_.notify_all();
    take();
    std::unique_lock<std::mutex> l(mu_);
    done_cv_.wait(l, [&] { return done_ == n_; });
    fn_ = nullptr;
  }
  ~WorkerPool() {
    {
      std::lock_guard<std::mutex> l(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto& t : workers_) t.join();
  }

 private:
  WorkerPool() {
    const int hw = (int)std::max(1u, std::thread::hardware_concurrency());
    for (int i = 1; i < std::min(hw, 16); ++i) workers_.emplace_back([this] { loop(); });
  }
  void take() {
    for (;;) {
      const std::function<void(int)>* fn;
      int i;
      {
        std::lock_guard<std::mutex> l(mu_);
        if (!fn_ || next_ >= n_) return;
        fn = fn_;
        i = next_++;
      }
      (*fn)(i);
      std::lock_guard<std::mutex> l(mu_);
      if (++done_ == n_) done_cv_.notify_all();
    }
  }
  void loop() {
    uint64_t seen = 0;
    for (;;) {
      {
        std::unique_lock<std::mutex> l(mu_);
        cv_.wait(l, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
      }
      take();
    }
  }
  std::vector<std::thread> workers_;
  std::mutex job_mu_, mu_;
  std::condition_variable cv_, done_cv_;
  const std::function<void(int)>* fn_ = nullptr;
  int next_ = 0, n_ = 0, done_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

// The current device's XCDs (each with its own L2), 1 when unknown.
int device_xcd_count() {
  static std::atomic<int> cached[64];
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 1;
  if (dev >= 0 && dev < 64 && cached[dev].load(std::memory_order_relaxed) > 0)
    return cached[dev].load(std::memory_order_relaxed);
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || n <= 0)
    n = 1;
  if (dev >= 0 && dev < 64) cached[dev].store(n, std::memory_order_relaxed);
  return n;
}

int device_cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev >= 0 && dev < 64 && cached[dev].load(std::memory_order_relaxed) > 0)
    return cached[dev].load(std::memory_order_relaxed);
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return 256;
  if (dev >= 0 && dev < 64) cached[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// The library's own stream per thread and device, for uploads the caller's stream does not order
// (population and plan tables, waited for before use). Created on first use at default priority.
struct StreamPool {
  int device = -1;
  hipStream_t aux[1] = {};
};
thread_local std::vector<StreamPool> g_pools;

emr_status stream_pool(StreamPool** out) {
  int dev = 0;
  HIP_OR_FAIL(hipGetDevice(&dev));
  for (StreamPool& p : g_pools)
    if (p.device == dev) {
      *out = &p;
      return EMR_OK;
    }
  StreamPool p;
  p.device = dev;
  HIP_OR_FAIL(hipStreamCreateWithFlags(&p.aux[0], hipStreamNonBlocking));
  g_pools.push_back(p);
  *out = &g_pools.back();
  return EMR_OK;
}

// Per-thread profiling of the discover-kernel launches.
struct Profiler {
  bool on = false;
  bool first_only = false;               // time only a call's first launch
  int32_t every = 1;                     // time one call in `every`
  int64_t seen = 0;                      // calls since enabled
  double rT = 4.0;
  int32_t calls = 0;                     // profiled calls since enabled or read
  std::vector<hipEvent_t> events;        // 2 per record, created lazily and reused
  std::vector<emr_launch_profile> recs;  // accumulated since enabled or read
};
thread_local Profiler g_prof;

using emr::query_base;
using emr::query_trans;
using emr::query_slots;
using emr::query_flops;

}  // namespace

namespace {
struct Plan;
}

struct emr_population {
  int32_t n_genomes = 0;
  std::vector<emr::ProgDesc> desc;      // [2 * n_genomes]
  std::vector<emr::GenomeInfo> info;    // [2 * n_genomes]
  uint32_t* d_blob = nullptr;
  emr::ProgDesc* d_desc = nullptr;
  size_t blob_words = 0;
  std::vector<uint32_t> h_blob;         // host copy of the program words (the code generator's input)
  // The plan of the last call (see plan_for): calls with the same sources and depth reuse it.
  mutable std::mutex plan_mu;
  mutable std::shared_ptr<const Plan> plan;
  // The plans of emr_eval_raw_noalloc calls (host memory only: they never get device tables or a
  // compiled tier), one per distinct sources and depth, kept with the population so that a table
  // image stays valid while its copy is in flight.
  mutable std::vector<std::shared_ptr<const Plan>> noalloc_plans;
};

namespace {

using emr::window_bucket;

void wait_library_calls(int dev);

// The compiled tier of one plan: its groups' programs translated to machine code, written into the
// code area of a copy of the template code object, loaded as a module on one device.
struct JitModule {
  int device = -1;
  hipModule_t mod = nullptr;
  hipFunction_t fn[2] = {};   // by output mode: raw, records
  int per_cu[2] = {1, 1};     // workgroups per CU of each
  uint32_t code_bytes = 0;    // size of the code area
  emr::Group* d_groups = nullptr;  // the plan's group table with the code offsets
  size_t programs = 0, program_bytes = 0, image_bytes = 0;
  double compile_ms = 0.0, load_ms = 0.0;
  JitModule() = default;
  JitModule(const JitModule&) = delete;
  JitModule& operator=(const JitModule&) = delete;
  ~JitModule() {
    // Nothing queued may still run the module's code or read its tables, so every call the
    // library has enqueued on the module's device finishes first (a module goes only when its
    // plan is replaced or its population freed).
    if (!mod && !d_groups) return;
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (device >= 0 && cur != device) (void)hipSetDevice(device);
    wait_library_calls(device);
    if (d_groups) (void)hipFree(d_groups);
    if (mod) (void)hipModuleUnload(mod);
    if (device >= 0 && cur >= 0 && cur != device) (void)hipSetDevice(cur);
  }
};

// Everything one discover / raw-eval call needs besides the population: the host-built tables
// (emr::PlanTables) and their device copies, schedules and compiled tier.
std::atomic<uint64_t> g_plan_ids{0};

struct Plan : emr::PlanTables {
  // Distinct for every plan the process builds (a freed plan's address may be reused).
  const uint64_t id = ++g_plan_ids;
  mutable std::mutex dev_mu;
  // The tables' device copy, uploaded on first use and freed with the plan.
  mutable char* d_tables = nullptr;
  // The bias rows of the plan's groups (the bind kernel's output: every position-independent
  // contribution per (genome, source)), computed on the device once, on first use (dev_mu).
  mutable float* d_bias = nullptr;
  // The workgroups' chunk lists of the plan's launches (plan_schedule), one per launch shape, on
  // the device (dev_mu).
  struct Sched {
    uint32_t grid, tiles, n_parts;
    emr::DiscoverPart part[emr::kMaxParts];
    uint32_t* d;
    uint32_t stride;
  };
  mutable std::vector<Sched> scheds;
  // Split parts of the plan's scheduled launches (cached_split_parts), one per launch shape.
  struct Split {
    bool skip_uniform;
    int64_t n_tiles;
    double waves;
    bool ok;
    uint32_t n_parts;
    uint32_t S[emr::kMaxParts], W[emr::kMaxParts], group0[emr::kMaxParts],
        groups[emr::kMaxParts], chunk[emr::kMaxParts];
  };
  mutable std::mutex split_mu;
  mutable std::vector<Split> splits;
  Plan() = default;
  Plan(const Plan&) = delete;
  Plan& operator=(const Plan&) = delete;
  ~Plan() {
    jit.reset();  // drains the device before the compiled tier's module goes
    if (d_tables) (void)hipFree(d_tables);
    if (d_bias) (void)hipFree(d_bias);
    for (const Sched& x : scheds) (void)hipFree(x.d);
  }
  // The compiled tier (jit_use): built at most once per plan, under jit_mu.
  mutable std::mutex jit_mu;
  mutable std::unique_ptr<JitModule> jit;
  mutable int jit_state = 0;  // 0 not built, 1 ready, -1 failed (reason in jit_error)
  mutable std::string jit_error;
  mutable std::atomic<int> calls{0};  // calls that ran this plan
};

// The record pool after a plan's fixed workspace: `capacity` parent indices, then (16-byte
// aligned) their float4 outputs.
size_t pool_w4_offset(const Plan& P, int64_t capacity) {
  return align256(P.total + (size_t)capacity * 4);
}
size_t workspace_need(const Plan& P, int64_t capacity) {
  return capacity > 0 ? align256(pool_w4_offset(P, capacity) + (size_t)capacity * 16) : P.total;
}

emr_status build_plan(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                      const int32_t* offs, int32_t n_shared, int32_t depth, Plan* plan) {
  if (!pop) return fail(EMR_E_INVAL, "population is NULL");
  std::string msg;
  emr_status st = emr::build_plan_tables(pop->desc.data(), pop->info.data(), pop->n_genomes,
                                         sources, n_sources, offs, n_shared, depth, plan, &msg);
  if (st != EMR_OK) return fail(st, "%s", msg.c_str());
  // every offset the kernels take from the tables, checked before any of them is uploaded
  if (!emr::check_plan_tables(*plan, pop->desc.data(), pop->blob_words, &msg))
    return fail(EMR_E_LIMIT, "the call's tables failed their bounds check: %s", msg.c_str());
  return EMR_OK;
}

bool plan_matches(const Plan& P, const emr_source* sources, int32_t n_sources, const int32_t* offs,
                  int32_t n_shared, int32_t depth, int32_t n_genomes) {
  if (P.depth != depth || (int64_t)P.key_sources.size() != n_sources ||
      P.key_has_offs != (offs != nullptr) || P.key_n_shared != n_shared)
    return false;
  if (n_sources > 0 &&
      std::memcmp(P.key_sources.data(), sources, sizeof(emr_source) * (size_t)n_sources) != 0)
    return false;
  return !offs ||
         std::memcmp(P.key_offs.data(), offs, sizeof(int32_t) * (size_t)(n_genomes + 1)) == 0;
}

// The plan for these sources and depth: the population's last plan when it was built for exactly
// the same arguments, else a new one (which then replaces it). Planning is host work that depends
// only on the population, the sources and the depth; every call still runs all kernels.
emr_status plan_for(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                    const int32_t* offs, int32_t n_shared, int32_t depth,
                    std::shared_ptr<const Plan>* out) {
  if (!pop) return fail(EMR_E_INVAL, "population is NULL");
  {
    std::lock_guard<std::mutex> lock(pop->plan_mu);
    if (pop->plan && (n_sources == 0 || sources) && n_sources >= 0 &&
        plan_matches(*pop->plan, sources, n_sources, offs, n_shared, depth, pop->n_genomes)) {
      *out = pop->plan;
      return EMR_OK;
    }
  }
  auto P = std::make_shared<Plan>();
  emr_status st = build_plan(pop, sources, n_sources, offs, n_shared, depth, P.get());
  if (st != EMR_OK) return st;
  std::lock_guard<std::mutex> lock(pop->plan_mu);
  pop->plan = P;
  *out = P;
  return EMR_OK;
}

// The plan's tables on the device, uploaded (and waited for) on first use.
emr_status plan_tables(const Plan& P, char** out) {
  std::lock_guard<std::mutex> lock(P.dev_mu);
  if (!P.d_tables) {
    char* d = nullptr;
    if (hipMalloc((void**)&d, P.img.size()) != hipSuccess)
      return fail(EMR_E_NOMEM, "device tables of %zu bytes", P.img.size());
    StreamPool* sp = nullptr;
    emr_status st = stream_pool(&sp);
    if (st == EMR_OK &&
        (hipMemcpyAsync(d, P.img.data(), P.img.size(), hipMemcpyHostToDevice, sp->aux[0]) !=
             hipSuccess ||
         hipStreamSynchronize(sp->aux[0]) != hipSuccess))
      st = fail(EMR_E_DEVICE, "upload of the call tables failed");
    if (st != EMR_OK) {
      (void)hipFree(d);
      return st;
    }
    P.d_tables = d;
  }
  *out = P.d_tables;
  return EMR_OK;
}

// Chunk cost estimates for the schedule, in lane-slots: the queries' cost-model slots (one tile is
// kTile / kWave positions per lane, for each source of the walk), plus per walk (positions, the
// variance, records) and per chunk (the group's tables) overheads. A position-independent group
// (a record-less walk) costs about one output row per query.
constexpr double kSchedWalkSlots = 40.0, kSchedChunkSlots = 200.0, kSchedUniformQuery = 2.5;
// A scheduled launch's chunks are sized so that none costs more than this share of a wave's mean
// load: the costliest chunks, taken first, end well before the launch does.
constexpr double kChunkCostShare = 0.5;

// Estimated cost of a chunk of nt tiles of group gi (sources per walk S, tiles per walk tpw).
double chunk_cost(const Plan& P, uint64_t gi, uint32_t S, double tpw, double nt) {
  const double q = (P.groups[gi].flags & 1u) ? (double)P.group_cost[gi] : kSchedUniformQuery;
  return S * q * nt * (emr::kTile / emr::kWave) + nt / tpw * kSchedWalkSlots + kSchedChunkSlots;
}
constexpr size_t kMaxScheds = 16;            // launch shapes a plan keeps lists for
constexpr uint64_t kSchedMaxChunks = 1u << 22;
constexpr uint64_t kSchedMaxBytes = 64u << 20;

// The waves' chunk lists of a discover launch with scalars sc on `grid` workgroups, made and
// uploaded on first use of that launch shape (the plan keeps them until it goes). *d is NULL when
// the launch runs round-robin instead: no chunks, beyond the bounds above, or cost estimates the
// scheduler refuses (not finite).
emr_status plan_schedule(const Plan& P, const emr::DiscoverScalars& sc, uint32_t grid,
                         const uint32_t** d, uint32_t* stride) {
  *d = nullptr;
  *stride = 0;
  if (grid == 0 || sc.n_chunks == 0 || sc.n_chunks > kSchedMaxChunks) return EMR_OK;
  std::lock_guard<std::mutex> lock(P.dev_mu);
  for (const Plan::Sched& x : P.scheds)
    if (x.grid == grid && x.tiles == sc.tiles && x.n_parts == sc.n_parts &&
        std::memcmp(x.part, sc.part, sizeof(emr::DiscoverPart) * sc.n_parts) == 0) {
      *d = x.d;
      *stride = x.stride;
      return EMR_OK;
    }
  if (P.scheds.size() >= kMaxScheds) return EMR_OK;
  std::vector<float> cost;
  std::vector<uint32_t> key;    // each chunk's group: a group's chunks share one XCD
  std::vector<uint32_t> entry;  // each chunk's list entry: part << kEntryPartShift | index
  cost.reserve(sc.n_chunks);
  key.reserve(sc.n_chunks);
  entry.reserve(sc.n_chunks);
  for (uint32_t k = 0; k < sc.n_parts; ++k) {
    const emr::DiscoverPart& pt = sc.part[k];
    if (pt.n_chunks >= (1u << emr::kEntryPartShift)) return EMR_OK;
    const double tpw = (double)(emr::positions_per_lane((int)pt.S, (int)pt.W) / emr::kTileIters);
    for (uint32_t cl = 0; cl < pt.n_chunks; ++cl) {
      const uint64_t gi = (uint64_t)pt.group0 + cl / pt.chunks_per_group;
      const uint32_t t0 = (cl % pt.chunks_per_group) * pt.chunk_tiles;
      if (gi >= P.groups.size() || t0 >= sc.tiles) return EMR_OK;  // not this plan's launch
      const double nt = (double)std::min(pt.chunk_tiles, sc.tiles - t0);
      cost.push_back((float)chunk_cost(P, gi, pt.S, tpw, nt));
      key.push_back((uint32_t)gi);
      entry.push_back(k << emr::kEntryPartShift | cl);
    }
  }
  if (cost.size() != sc.n_chunks) return EMR_OK;
  std::vector<uint32_t> table;
  uint32_t st = 0;
  // one list per workgroup (a CU); workgroups go to the XCDs round-robin (from a starting XCD
  // that changes between launches), so workgroups b with equal b % xcds share an XCD
  const uint32_t xcds = (uint32_t)device_xcd_count();
  if (!emr::lpt_schedule(cost.data(), key.data(), (uint32_t)P.groups.size(), sc.n_chunks, grid,
                         1u, grid >= xcds ? xcds : 1u, &table, &st) ||
      st > emr::kListLds || table.size() * sizeof(uint32_t) > kSchedMaxBytes)
    return EMR_OK;
  // every entry names a part of the launch and a chunk inside it (the kernel relies on it)
  for (uint32_t& t : table) {
    if (t == emr::kNoChunk) continue;
    if (t >= entry.size()) return fail(EMR_E_LIMIT, "chunk schedule: bad chunk %u", t);
    t = entry[t];
    const uint32_t k = t >> emr::kEntryPartShift, cl = t & ((1u << emr::kEntryPartShift) - 1u);
    if (k >= sc.n_parts || cl >= sc.part[k].n_chunks)
      return fail(EMR_E_LIMIT, "chunk schedule: entry %u outside its part", t);
  }
  uint32_t* dev = nullptr;
  if (hipMalloc((void**)&dev, table.size() * sizeof(uint32_t)) != hipSuccess)
    return fail(EMR_E_NOMEM, "chunk schedule of %zu bytes", table.size() * sizeof(uint32_t));
  StreamPool* sp = nullptr;
  emr_status rs = stream_pool(&sp);
  if (rs == EMR_OK &&
      (hipMemcpyAsync(dev, table.data(), table.size() * sizeof(uint32_t), hipMemcpyHostToDevice,
                      sp->aux[0]) != hipSuccess ||
       hipStreamSynchronize(sp->aux[0]) != hipSuccess))
    rs = fail(EMR_E_DEVICE, "upload of the chunk schedule failed");
  if (rs != EMR_OK) {
    (void)hipFree(dev);
    return rs;
  }
  Plan::Sched x{};
  x.grid = grid;
  x.tiles = sc.tiles;
  x.n_parts = sc.n_parts;
  std::memcpy(x.part, sc.part, sizeof(emr::DiscoverPart) * sc.n_parts);
  x.d = dev;
  x.stride = st;
  P.scheds.push_back(x);
  *d = dev;
  *stride = st;
  return EMR_OK;
}

// ------------------------------------------------------------------ call flags
// Each call's kernels raise their error bits (word 0) and largest pair count (word 1) into a slot
// of a library-owned ring in device memory. A slot is zero when a call takes it; the call's last
// kernel (k_scan for a record call, k_finalize otherwise) writes the words to the slot's pinned
// host words and clears them again. So
// no copy of the flags goes either way, and the caller's workspace keeps no state from one call
// to the next.
constexpr int kFlagSlots = 256;
constexpr int kSlotWords = 16;  // the kFlag* words, then padding

struct FlagRing {
  uint32_t* dev = nullptr;
  uint32_t* host = nullptr;      // pinned (host view)
  uint32_t* host_dev = nullptr;  // the same words, device view
  hipEvent_t done[kFlagSlots] = {};
  const void* ws[kFlagSlots] = {};  // workspace of the slot's last call (NULL: nothing to check)
  uint64_t seq[kFlagSlots] = {};    // order of the calls
  bool pending[kFlagSlots] = {};    // done[k] is recorded after the slot's last call
  bool dirty[kFlagSlots] = {};      // a call failed after taking the slot: cleared before reuse
  int next = 0;
  uint64_t calls = 0;
};
std::mutex g_ring_mu;
std::vector<std::pair<int, FlagRing*>> g_rings;  // one per device, kept for the process

// The ring of the current device (g_ring_mu held).
emr_status flag_ring(FlagRing** out) {
  int dev = 0;
  HIP_OR_FAIL(hipGetDevice(&dev));
  for (const auto& e : g_rings)
    if (e.first == dev) {
      *out = e.second;
      return EMR_OK;
    }
  std::unique_ptr<FlagRing> R(new FlagRing());
  const size_t bytes = (size_t)kFlagSlots * kSlotWords * 4;
  if (hipMalloc((void**)&R->dev, bytes) != hipSuccess) return fail(EMR_E_NOMEM, "flag slots");
  if (hipMemset(R->dev, 0, bytes) != hipSuccess ||
      hipHostMalloc((void**)&R->host, bytes, hipHostMallocDefault) != hipSuccess) {
    (void)hipFree(R->dev);
    return fail(EMR_E_NOMEM, "flag slots");
  }
  std::memset(R->host, 0, bytes);
  if (hipHostGetDevicePointer((void**)&R->host_dev, R->host, 0) != hipSuccess)
    return fail(EMR_E_DEVICE, "device view of the pinned flag words");
  for (int k = 0; k < kFlagSlots; ++k)
    HIP_OR_FAIL(hipEventCreateWithFlags(&R->done[k], hipEventDisableTiming));
  g_rings.push_back({dev, R.get()});
  *out = R.release();
  return EMR_OK;
}

// Waits for every call the library has enqueued on device `dev`: each call's last kernel is
// followed by its flag slot's event, and a slot is taken again only after its previous call's
// event has completed, so the slots' latest events cover every call ever enqueued.
void wait_library_calls(int dev) {
  std::vector<hipEvent_t> evs;
  {
    std::lock_guard<std::mutex> lock(g_ring_mu);
    for (const auto& e : g_rings)
      if (e.first == dev)
        for (int k = 0; k < kFlagSlots; ++k)
          if (e.second->pending[k]) evs.push_back(e.second->done[k]);
  }
  for (hipEvent_t ev : evs) (void)hipEventSynchronize(ev);
}

// One call's slot: taken before its first kernel, given back after its last (or on failure).
struct CallFlags {
  FlagRing* ring = nullptr;
  int slot = -1;
  uint32_t* dev = nullptr;       // the device words the kernels raise into
  uint32_t* host = nullptr;      // the pinned words (host view)
  uint32_t* host_dev = nullptr;  // the pinned words (device view)
  hipStream_t s = nullptr;
  const void* ws = nullptr;
  bool ok = false;  // the call's last kernel is enqueued
  CallFlags() = default;
  CallFlags(const CallFlags&) = delete;
  CallFlags& operator=(const CallFlags&) = delete;
  ~CallFlags() {
    if (!ring) return;
    std::lock_guard<std::mutex> lock(g_ring_mu);
    // the slot's next user waits for whatever this call enqueued
    ring->pending[slot] = hipEventRecord(ring->done[slot], s) == hipSuccess;
    ring->ws[slot] = ok ? ws : nullptr;
    ring->seq[slot] = ++ring->calls;
    ring->dirty[slot] = !ok;
  }
};

emr_status take_flags(const void* workspace, hipStream_t s, CallFlags* f) {
  std::lock_guard<std::mutex> lock(g_ring_mu);
  FlagRing* R = nullptr;
  emr_status st = flag_ring(&R);
  if (st != EMR_OK) return st;
  const int k = R->next;
  R->next = (k + 1) % kFlagSlots;
  // the slot's previous call (kFlagSlots calls ago) must have finished with its words
  if (R->pending[k]) HIP_OR_FAIL(hipEventSynchronize(R->done[k]));
  R->pending[k] = false;
  R->ws[k] = nullptr;
  f->ring = R;
  f->slot = k;
  f->dev = R->dev + (size_t)k * kSlotWords;
  f->host = R->host + (size_t)k * kSlotWords;
  f->host_dev = R->host_dev + (size_t)k * kSlotWords;
  f->s = s;
  f->ws = workspace;
  for (int k = 0; k < emr::kFlagWords; ++k) f->host[k] = 0u;
  if (R->dirty[k]) {
    HIP_OR_FAIL(emr_launch_fill(f->dev, kSlotWords, 0u, s));
    R->dirty[k] = false;
  }
  return EMR_OK;
}

// Where a call's kernels find the plan's tables, the depth's tile geometry and the bias rows: the
// plan's own device copies (call_tables), or copies in the allocation-free scratch.
struct CallTables {
  const char* tables = nullptr;
  const uint32_t* geo = nullptr;
  uint32_t geo_rows = 0;
  const float* bias = nullptr;
};

// The bind kernel's arguments over the plan's tables: bias rows to `bias` (bias_table_floats()),
// table errors raised into *err.
emr::BindArgs bind_args(const emr_population* pop, const Plan& P, const char* tables, float* bias,
                        uint32_t* err) {
  emr::BindArgs b{};
  b.blob = pop->d_blob;
  b.desc = pop->d_desc;
  b.members = (const emr::Member*)(tables + P.t_members);
  b.src_xy = (const float*)(tables + P.t_srcxy);
  b.bias_tab = bias;
  b.err = err;
  b.n_members = (uint32_t)P.members.size();
  b.n_desc = (uint32_t)pop->desc.size();
  b.n_sources = (uint32_t)(P.src_xy.size() / 2);
  b.blob_words = (uint32_t)pop->blob_words;
  b.bias_floats = P.bias_floats;
  return b;
}

// The plan's bias rows on the device, computed on first use by the bind kernel on the library's
// stream and waited for (a table error found then fails the call that needed them).
emr_status plan_bias(const emr_population* pop, const Plan& P, const char* tables,
                     const float** out) {
  std::lock_guard<std::mutex> lock(P.dev_mu);
  if (!P.d_bias) {
    const size_t n = P.bias_table_floats();
    float* d = nullptr;
    if (hipMalloc((void**)&d, (n + 64) * sizeof(float)) != hipSuccess)
      return fail(EMR_E_NOMEM, "bias rows of %zu floats", n);
    uint32_t* err = (uint32_t*)(d + n);  // one word after the rows and their padding
    StreamPool* sp = nullptr;
    emr_status st = stream_pool(&sp);
    uint32_t host_err = 0;
    if (st == EMR_OK) {
      const emr::BindArgs b = bind_args(pop, P, tables, d, err);
      if (emr_launch_fill(d, (int64_t)n + 1, 0u, sp->aux[0]) != hipSuccess ||
          emr_launch_bind(&b, sp->aux[0]) != hipSuccess ||
          hipMemcpyAsync(&host_err, err, 4, hipMemcpyDeviceToHost, sp->aux[0]) != hipSuccess ||
          hipStreamSynchronize(sp->aux[0]) != hipSuccess)
        st = fail(EMR_E_DEVICE, "computing the bias rows failed");
      else if (host_err)
        st = fail(EMR_E_DEVICE, "the bind kernel reported error flags 0x%x (2: a table entry out "
                  "of range)", host_err);
    }
    if (st != EMR_OK) {
      (void)hipFree(d);
      return st;
    }
    P.d_bias = d;
  }
  *out = P.d_bias;
  return EMR_OK;
}

// A call's workspace: at least `need` bytes, 256-byte aligned.
emr_status check_call_workspace(const void* workspace, int64_t workspace_bytes, int64_t need) {
  if (!workspace || workspace_bytes < need)
    return fail(EMR_E_INVAL, "workspace of %lld bytes is smaller than the %lld needed",
                (long long)workspace_bytes, (long long)need);
  if (((uintptr_t)workspace & 255) != 0) return fail(EMR_E_INVAL, "workspace not 256-byte aligned");
  return EMR_OK;
}

// The tile geometry table of a depth on the current device (k_tile_geo), built on first use and
// kept for the life of the process (tiles_per_pair(depth) + kGeoPadRows rows of 16 bytes: 5.6 MB
// at depth 13).
emr_status tile_geo_table(int depth, const uint32_t** out, uint32_t* rows) {
  static std::mutex mu;
  static std::vector<std::pair<std::pair<int, int>, uint32_t*>> cache;  // (device, depth)
  int dev = 0;
  HIP_OR_FAIL(hipGetDevice(&dev));
  const int64_t tiles = emr::tiles_per_pair(depth), n = tiles + emr::kGeoPadRows;
  if (n > 0xFFFFFFFFll / 4) return fail(EMR_E_LIMIT, "depth %d has too many tiles", depth);
  *rows = (uint32_t)n;
  std::lock_guard<std::mutex> lock(mu);
  for (const auto& e : cache)
    if (e.first == std::make_pair(dev, depth)) {
      *out = e.second;
      return EMR_OK;
    }
  uint32_t* d = nullptr;
  if (hipMalloc((void**)&d, (size_t)n * 16) != hipSuccess)
    return fail(EMR_E_NOMEM, "tile geometry table of %lld rows", (long long)n);
  StreamPool* sp = nullptr;
  emr_status st = stream_pool(&sp);
  if (st == EMR_OK &&
      (emr_launch_tile_geo(d, (uint32_t)tiles, (uint32_t)n, sp->aux[0]) != hipSuccess ||
       hipStreamSynchronize(sp->aux[0]) != hipSuccess))
    st = fail(EMR_E_DEVICE, "building the tile geometry table failed");
  if (st != EMR_OK) {
    (void)hipFree(d);
    return st;
  }
  cache.push_back({{dev, depth}, d});
  *out = d;
  return EMR_OK;
}

// ------------------------------------------------------------------ compiled tier
std::atomic<int> g_jit_policy{EMR_JIT_AUTO};

// The template's code area: 1024 words of s_endpgm (jit.hip).
constexpr size_t kTemplateArea = 4096;

// Translates every distinct (program, sources per walk, window) of the plan's groups to machine
// code, writes the programs (64-byte aligned) into a copy of the template whose code area is
// grown to fit them, loads the copy as a module on the current device, and uploads the plan's
// group table with each group's code offset.
emr_status jit_build(const emr_population* pop, const Plan& P, std::unique_ptr<JitModule>* out) {
  using clock = std::chrono::steady_clock;
  const auto t0 = clock::now();
  auto M = std::make_unique<JitModule>();
  // distinct programs: key (desc, bucket) -> index
  struct Job {
    uint32_t desc;
    int S, W;
  };
  std::vector<Job> jobs;
  std::vector<uint32_t> job_of_group(P.groups.size());
  {
    std::vector<std::pair<uint64_t, uint32_t>> keys;
    keys.reserve(P.groups.size());
    for (const Plan::Bucket& b : P.buckets)
      for (uint32_t g = b.first; g < b.first + b.count; ++g) {
        const uint32_t desc = P.members[P.group_member0[g]].desc;
        keys.push_back({((uint64_t)desc << 16) | ((uint64_t)b.S << 8) | (uint64_t)b.window, g});
      }
    std::sort(keys.begin(), keys.end());
    for (size_t i = 0; i < keys.size(); ++i) {
      if (i == 0 || keys[i].first != keys[i - 1].first)
        jobs.push_back({(uint32_t)(keys[i].first >> 16), (int)((keys[i].first >> 8) & 0xFF),
                        (int)(keys[i].first & 0xFF)});
      job_of_group[keys[i].second] = (uint32_t)(jobs.size() - 1);
    }
  }
  std::vector<emr::jit::Code> code(jobs.size());
  std::vector<std::string> errs(jobs.size());
  std::vector<char> ok(jobs.size(), 0);
  auto work = [&](size_t lo, size_t hi) {
    for (size_t j = lo; j < hi; ++j) {
      const Job& J = jobs[j];
      const emr::ProgDesc& d = pop->desc[J.desc];
      if ((uint64_t)d.var_off + 16ull * d.n_rec > pop->h_blob.size()) {
        errs[j] = "program outside the population table";
        continue;
      }
      ok[j] = emr::jit::compile_program(pop->h_blob.data() + d.var_off, d.n_rec,
                                        (d.flags & 1u) != 0, J.S,
                                        emr::positions_per_lane(J.S, J.W), J.W, false, &code[j],
                                        &errs[j]);
    }
  };
  const int n_threads = (int)std::max<size_t>(
      1, std::min<size_t>({(size_t)WorkerPool::get().size(), 16, jobs.size() / 64}));
  WorkerPool::get().run(n_threads, [&](int t) {
    work(jobs.size() * t / n_threads, jobs.size() * (t + 1) / n_threads);
  });
  std::vector<uint32_t> offs(jobs.size());
  size_t bytes = 0;
  for (size_t j = 0; j < jobs.size(); ++j) {
    if (!ok[j]) return fail(EMR_E_INVAL, "compiling a program: %s", errs[j].c_str());
    offs[j] = (uint32_t)bytes;
    bytes += (code[j].words.size() * 4 + 63) & ~size_t(63);
    if (bytes > (size_t(1) << 30)) return fail(EMR_E_LIMIT, "compiled programs exceed 1 GiB");
  }
  const size_t need = bytes + emr::kJitTailPad;
  const size_t area = need <= kTemplateArea ? kTemplateArea
                                            : kTemplateArea + ((need - kTemplateArea + 4095) & ~size_t(4095));
  // the template copy, grown, with the programs written into its area
  const uint8_t* tpl = emr_jit_template_begin;
  const size_t tpl_n = (size_t)(emr_jit_template_end - emr_jit_template_begin);
  emr::jit::AreaInfo ai;
  std::string msg;
  std::vector<uint8_t> img;
  if (!emr::jit::find_area(tpl, tpl_n, kTemplateArea, &ai, &msg) ||
      !emr::jit::grow_area(tpl, tpl_n, ai, area, &img, &msg))
    return fail(EMR_E_DEVICE, "compiled tier: %s", msg.c_str());
  for (size_t j = 0; j < jobs.size(); ++j)
    std::memcpy(img.data() + ai.file_off + offs[j], code[j].words.data(), code[j].words.size() * 4);
  const auto t1 = clock::now();
  HIP_OR_FAIL(hipGetDevice(&M->device));
  HIP_OR_FAIL(hipModuleLoadData(&M->mod, img.data()));
  static const char* names[2] = {"emr_discover_jit_raw", "emr_discover_jit_records"};
  for (int k = 0; k < 2; ++k) {
    HIP_OR_FAIL(hipModuleGetFunction(&M->fn[k], M->mod, names[k]));
    int n = 0;
    if (hipModuleOccupancyMaxActiveBlocksPerMultiprocessor(&n, M->fn[k], emr::kDiscoverThreads, 0) ==
            hipSuccess &&
        n > 0)
      M->per_cu[k] = n;
  }
  M->code_bytes = (uint32_t)area;
  std::vector<emr::Group> groups = P.groups;
  for (size_t g = 0; g < groups.size(); ++g) groups[g].code_off = offs[job_of_group[g]];
  if (!groups.empty()) {
    HIP_OR_FAIL(hipMalloc((void**)&M->d_groups, groups.size() * sizeof(emr::Group)));
    HIP_OR_FAIL(hipMemcpy(M->d_groups, groups.data(), groups.size() * sizeof(emr::Group),
                          hipMemcpyHostToDevice));
  }
  const auto t2 = clock::now();
  M->programs = jobs.size();
  M->program_bytes = bytes;
  M->image_bytes = img.size();
  M->compile_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  M->load_ms = std::chrono::duration<double, std::milli>(t2 - t1).count();
  *out = std::move(M);
  return EMR_OK;
}

// Whether a call of `slots` algorithmic slots runs the plan's compiled programs, building them
// first when the policy asks for it: EMR_JIT_ALWAYS builds on the first call (and a failed build
// fails the call); EMR_JIT_AUTO builds when the plan is run a second time (the same population
// and sources again: a benchmark loop, or repeated queries), or at once for a call large enough
// that the faster kernel repays the build (an interpreted call above ~10 ms); a failed build
// leaves the plan interpreted (the reason is kept for emr_jit_info).
emr_status jit_use(const emr_population* pop, const Plan& P, double slots, bool* use) {
  *use = false;
  const int policy = g_jit_policy.load();
  const int n = ++P.calls;
  if (policy == EMR_JIT_OFF || P.groups.empty()) return EMR_OK;
  std::lock_guard<std::mutex> lock(P.jit_mu);
  int dev = 0;
  HIP_OR_FAIL(hipGetDevice(&dev));
  if (P.jit_state == 1) {
    *use = P.jit->device == dev;
    return EMR_OK;
  }
  if (P.jit_state == -1) {
    if (policy == EMR_JIT_ALWAYS)
      return fail(EMR_E_DEVICE, "the compiled tier failed for this plan: %s", P.jit_error.c_str());
    return EMR_OK;
  }
  const double interp_ms = slots / 2.2e10;  // the interpreter's measured rate, ~22 T slots/s
  if (policy == EMR_JIT_AUTO && n < 2 && interp_ms < 10.0) return EMR_OK;
  std::unique_ptr<JitModule> M;
  emr_status st = jit_build(pop, P, &M);
  if (st != EMR_OK) {
    P.jit_state = -1;
    P.jit_error = g_err;
    return policy == EMR_JIT_ALWAYS ? st : EMR_OK;
  }
  P.jit = std::move(M);
  P.jit_state = 1;
  *use = true;
  return EMR_OK;
}

// Algorithmic slots of a whole call (every tile of every pair) under the default cost model.
double plan_slots(const Plan& P) {
  double s = 0.0;
  for (const Plan::Launch& L : P.launches) s += L.slots_base + 4.0 * L.slots_trans;
  return s * (double)emr::n_positions(P.depth);
}

// The compiled tier's discover launch: the same scalars and grid sizing as the interpreter's,
// through the plan's module.
emr_status jit_launch(const Plan& P, const emr::DiscoverArgs& a, int mode, uint32_t blocks,
                      hipStream_t s, hipEvent_t start, hipEvent_t stop) {
  const JitModule& M = *P.jit;
  emr::DiscoverScalars sc{};
  uint32_t grid = 0;
  HIP_OR_FAIL(emr_discover_setup(&a, blocks, M.per_cu[mode], device_cu_count(), &sc, &grid));
  sc.code_bytes = M.code_bytes;
  if (start) HIP_OR_FAIL(hipEventRecord(start, s));
  if (grid > 0) {
    const uint32_t* geo = a.geo;
    const uint32_t* blob = a.blob;
    const emr::Group* grp = a.groups;
    const float* bias_tab = a.bias_tab;
    uint64_t* status = a.status;
    uint32_t* err = a.err;
    float* raw = a.raw;
    void* args[] = {&geo, &blob, &grp, &bias_tab, &status, &err, &raw, &sc};
    HIP_OR_FAIL(hipModuleLaunchKernel(M.fn[mode], grid, 1, 1, emr::kDiscoverThreads, 1, 1, 0, s, args,
                                      nullptr));
  }
  if (stop) HIP_OR_FAIL(hipEventRecord(stop, s));
  return EMR_OK;
}

// The parts of a scheduled launch: each bucket of L (its groups in decreasing cost) split into
// runs of groups that share a chunk size, the largest power of two of at most kChunkTilesMax
// tiles (and at least one walk's) whose chunk costs no more than kChunkCostShare of a wave's mean
// load over `waves` waves. False (a is left for the caller) when the launch has no groups.
bool split_parts(const Plan& P, const Plan::Launch& L, bool skip_uniform, int64_t n_tiles,
                 double waves, emr::DiscoverArgs* a) {
  double total = 0.0;  // the launch's queries and walks (per-chunk costs aside)
  for (int k = 0; k < L.n_parts; ++k) {
    const Plan::Bucket& bk = P.buckets[(size_t)L.part[k]];
    const uint32_t n = skip_uniform ? bk.varying : bk.count;
    const double tpw = (double)(emr::positions_per_lane(bk.S, bk.window) / emr::kTileIters);
    for (uint32_t g = 0; g < n; ++g)
      total += chunk_cost(P, bk.first + g, (uint32_t)bk.S, tpw, (double)n_tiles) - kSchedChunkSlots;
  }
  if (total <= 0.0 || waves <= 0.0) return false;
  const double limit = kChunkCostShare * total / waves;
  uint32_t np = 0;
  for (int k = 0; k < L.n_parts; ++k) {
    const Plan::Bucket& bk = P.buckets[(size_t)L.part[k]];
    const uint32_t n = skip_uniform ? bk.varying : bk.count;
    const uint32_t tpw = (uint32_t)emr::positions_per_lane(bk.S, bk.window) / emr::kTileIters;
    auto size_of = [&](uint32_t g) {
      for (uint32_t t = emr::kChunkTilesMax; t > tpw; t /= 2)
        if (chunk_cost(P, bk.first + g, (uint32_t)bk.S, (double)tpw, (double)t) <= limit) return t;
      return tpw;
    };
    for (uint32_t g = 0; g < n;) {
      const uint32_t t = size_of(g);
      uint32_t h = g + 1;
      while (h < n && size_of(h) == t) ++h;
      if (np == (uint32_t)emr::kMaxParts) return false;
      a->part_S[np] = (uint32_t)bk.S;
      a->part_W[np] = (uint32_t)bk.window;
      a->part_group0[np] = bk.first + g;
      a->part_groups[np] = h - g;
      a->part_chunk[np] = t;
      ++np;
      g = h;
    }
  }
  if (np == 0) return false;
  a->n_parts = np;
  return true;
}

// split_parts, remembered per launch shape (a plan's repeated calls split the same way).
constexpr size_t kMaxSplits = 8;
bool cached_split_parts(const Plan& P, const Plan::Launch& L, bool skip_uniform, int64_t n_tiles,
                        double waves, emr::DiscoverArgs* a) {
  std::lock_guard<std::mutex> lock(P.split_mu);
  const Plan::Split* hit = nullptr;
  for (const Plan::Split& x : P.splits)
    if (x.skip_uniform == skip_uniform && x.n_tiles == n_tiles && x.waves == waves) hit = &x;
  if (!hit) {
    Plan::Split x{};
    x.skip_uniform = skip_uniform;
    x.n_tiles = n_tiles;
    x.waves = waves;
    emr::DiscoverArgs t{};
    x.ok = split_parts(P, L, skip_uniform, n_tiles, waves, &t);
    x.n_parts = x.ok ? t.n_parts : 0u;
    for (uint32_t k = 0; k < x.n_parts; ++k) {
      x.S[k] = t.part_S[k];
      x.W[k] = t.part_W[k];
      x.group0[k] = t.part_group0[k];
      x.groups[k] = t.part_groups[k];
      x.chunk[k] = t.part_chunk[k];
    }
    if (P.splits.size() >= kMaxSplits) P.splits.erase(P.splits.begin());
    P.splits.push_back(x);
    hit = &P.splits.back();
  }
  if (!hit->ok) return false;
  a->n_parts = hit->n_parts;
  for (uint32_t k = 0; k < hit->n_parts; ++k) {
    a->part_S[k] = hit->S[k];
    a->part_W[k] = hit->W[k];
    a->part_group0[k] = hit->group0[k];
    a->part_groups[k] = hit->groups[k];
    a->part_chunk[k] = hit->chunk[k];
  }
  return true;
}

// Enqueues the discover launch (every bucket, on the caller's stream) for tiles
// tile_lo .. tile_lo + n_tiles - 1 of every pair, then, for records, the compaction: the range's
// records go to `out` pair after pair (pair_offset, pair_count), its capacity also bounding the
// pool in the workspace; raw outputs go to raw[r * N(D) + p].
// jit: run the plan's compiled programs (jit_use said so) instead of the interpreter. With
// `finalize`, the range's last kernel (k_scan for records, k_finalize for raw outputs) then hands
// the call's flags to their pinned words.
// With `clear` (record mode), the workspace's group marks and per-pair totals are cleared right
// before the discover launch, once every argument of that launch is ready on the host.
// flags: the call's device flag words (error bits, largest count); flags_host: their pinned words
// (device view) for that hand-over.
// may_alloc: the call may allocate on first use: the thread's launch profiling (its events) and
// the launch's chunk schedule apply (off for the allocation-free call, which runs its chunks
// round-robin). A compiled-tier launch gets its workgroups' chunk lists once its plan runs again
// (a second call) or runs in several ranges (a streamed call): placing the chunks of a plan used
// once would cost its single call more than the balance saves. Interpreted launches run
// round-robin.
emr_status launch_range(const emr_population* pop, const Plan& P, const CallTables& T,
                        float theta, const emr_result* out, float* raw, void* workspace,
                        hipStream_t s, int64_t tile_lo, int64_t n_tiles, bool jit,
                        uint32_t* flags, uint32_t* flags_host, bool finalize, bool clear,
                        bool may_alloc = true, int64_t* host_counts = nullptr) {
  char* ws = (char*)workspace;
  const char* tables = T.tables;
  const uint32_t* geo_tab = T.geo;
  const uint32_t geo_rows = T.geo_rows;
  const int cus = device_cu_count();
  const bool records = out != nullptr && raw == nullptr;
  const int mode = records ? emr::kModeRecords : emr::kModeRaw;
  // With theta >= 0 a position-independent output keeps no cell (its variance is exactly 0): the
  // record mode leaves those groups (the last of each part) out of the launch, and the
  // compaction gives their pairs no records without reading their counts.
  const bool skip_uniform = records && !(0.0f > theta);
  const int64_t cap = records ? out->capacity : 0;
  uint32_t* pool_parent = records ? (uint32_t*)(ws + P.total) : nullptr;
  float* pool_w4 = records ? (float*)(ws + pool_w4_offset(P, cap)) : nullptr;
  Profiler& prof = g_prof;
  const size_t rec0 = prof.recs.size();
  const bool timed_call = may_alloc && prof.on && prof.seen++ % prof.every == 0;
  const size_t n_timed = timed_call ? (prof.first_only ? 1 : P.launches.size()) : 0;
  while (prof.events.size() < 2 * (rec0 + n_timed)) {
    hipEvent_t e;
    HIP_OR_FAIL(hipEventCreate(&e));
    prof.events.push_back(e);
  }
  // queries of the range per source: every tile holds 256 positions but the head tile
  const double npos = (double)(tile_lo == 0 ? emr::n_positions(P.depth) -
                                                  emr::kTile * (P.tiles - n_tiles)
                                            : emr::kTile * n_tiles);
  for (size_t li = 0; li < P.launches.size(); ++li) {
    const Plan::Launch& L = P.launches[li];
    emr::DiscoverArgs a{};
    a.geo = geo_tab;
    a.geo_rows = geo_rows;
    a.blob = pop->d_blob;
    a.groups = jit ? P.jit->d_groups : (const emr::Group*)(tables + P.t_groups);
    a.bias_tab = T.bias;
    a.status = (uint64_t*)(ws + P.off_status);
    a.nz = (uint64_t*)(ws + P.off_nz);
    a.err = flags;
    a.pool_parent = pool_parent;
    a.pool_w4 = pool_w4;
    a.pair_total = records ? (uint32_t*)(ws + P.off_ptotal) : nullptr;
    a.raw = raw;
    a.cap = cap;
    a.n_pos = emr::n_positions(P.depth);
    const bool scheduled = may_alloc && jit && (P.calls.load() >= 2 || n_tiles < P.tiles);
    const int per_cu = jit ? P.jit->per_cu[mode] : emr_discover_per_cu(mode);
    if (!scheduled || !cached_split_parts(P, L, skip_uniform, n_tiles,
                                          (double)emr::kDiscoverWaves * per_cu * cus, &a)) {
      a.n_parts = (uint32_t)L.n_parts;
      for (int k = 0; k < L.n_parts; ++k) {
        const Plan::Bucket& bk = P.buckets[(size_t)L.part[k]];
        a.part_S[k] = (uint32_t)bk.S;
        a.part_W[k] = (uint32_t)bk.window;
        a.part_group0[k] = bk.first;
        a.part_groups[k] = skip_uniform ? bk.varying : bk.count;
        a.part_chunk[k] = 0;  // the launcher's rule
      }
    }
    a.tile_lo = (uint32_t)tile_lo;
    a.tiles = (uint32_t)n_tiles;
    a.depth = P.depth;
    a.theta = theta;
    a.blob_words = (uint32_t)pop->blob_words;
    a.n_pairs = (uint32_t)P.n_pairs;
    a.bias_floats = P.bias_floats;
    const uint32_t blocks = (uint32_t)cus * 16;  // the launcher sizes the grid below this
    if (scheduled) {
      // the launch's grid and chunks, as its launcher will size them, for the workgroups' lists
      emr::DiscoverScalars sc{};
      uint32_t grid = 0;
      HIP_OR_FAIL(emr_discover_setup(&a, blocks, per_cu, cus, &sc, &grid));
      const uint32_t* sched = nullptr;
      uint32_t stride = 0;
      emr_status ss = plan_schedule(P, sc, grid, &sched, &stride);
      if (ss != EMR_OK) return ss;
      if (sched) {
        a.sched = sched;
        a.sched_stride = stride;
        a.sched_lists = grid;
      }
    }
    const bool timed = li < n_timed;
    hipEvent_t e0 = timed ? prof.events[2 * (rec0 + li)] : nullptr;
    hipEvent_t e1 = timed ? prof.events[2 * (rec0 + li) + 1] : nullptr;
    if (li == 0 && clear && records)
      HIP_OR_FAIL(emr_launch_fill(ws + P.off_nz, P.clear_words, 0u, s));
    if (jit) {
      emr_status js = jit_launch(P, a, mode, blocks, s, e0, e1);
      if (js != EMR_OK) return js;
    } else {
      HIP_OR_FAIL(emr_launch_discover(&a, mode, blocks, s, e0, e1));
    }
    if (timed) {
      emr_launch_profile r{};
      r.call = prof.calls;
      const Plan::Bucket& b0 = P.buckets[(size_t)L.part[0]];
      r.group_size = b0.S;
      r.window = b0.window;
      r.positions = emr::positions_per_lane(b0.S, b0.window);
      for (int k = 0; k < L.n_parts; ++k)
        r.tiles += (int64_t)P.buckets[(size_t)L.part[k]].count * n_tiles;
      r.slots = npos * (L.slots_base + prof.rT * L.slots_trans);
      r.queries = (int64_t)(npos * L.sources);
      r.compiled = jit ? 1 : 0;
      r.listed = a.sched != nullptr ? 1 : 0;
      r.parts = (int32_t)a.n_parts;
      prof.recs.push_back(r);
    }
  }
  if (timed_call) prof.calls++;
  if (clear && records && P.launches.empty())
    HIP_OR_FAIL(emr_launch_fill(ws + P.off_nz, P.clear_words, 0u, s));
  if (records && P.n_pairs > 0) {
    emr::ScanArgs S{};
    S.pair_total = (uint32_t*)(ws + P.off_ptotal);
    S.pair_count = out->pair_count;
    S.pair_offset = out->pair_offset;
    S.flags = flags;
    S.host = finalize ? flags_host : nullptr;  // k_scan then ends the call's flag writes
    S.host_counts = host_counts;
    S.n_pairs = (uint32_t)P.n_pairs;
    emr::MoveArgs M{};
    M.status = (const uint64_t*)(ws + P.off_status);
    M.pool_parent = pool_parent;
    M.pool_w4 = pool_w4;
    M.parent = out->parent;
    M.w4 = out->w4;
    M.pair_count = out->pair_count;
    M.pair_offset = out->pair_offset;
    M.nz = (uint64_t*)(ws + P.off_nz);
    M.skip = skip_uniform ? (const uint8_t*)(tables + P.t_uniform) : nullptr;
    M.cap = cap;
    M.tiles = (uint32_t)n_tiles;
    M.n_pairs = (uint32_t)P.n_pairs;
    M.nz_words = emr::nz_words((uint32_t)n_tiles);
    HIP_OR_FAIL(emr_launch_compact(&S, &M, s));
    return EMR_OK;
  }
  if (records) HIP_OR_FAIL(emr_launch_fill(out->pair_offset, 2, 0u, s));  // no pairs: offset 0
  if (finalize) HIP_OR_FAIL(emr_launch_finalize(flags, flags_host, s));
  return EMR_OK;
}

// The plan's own device tables and bias rows and the depth's tile geometry table (each made on
// first use).
emr_status call_tables(const emr_population* pop, const Plan& P, CallTables* T) {
  char* tables = nullptr;
  emr_status st = plan_tables(P, &tables);
  if (st != EMR_OK) return st;
  T->tables = tables;
  if ((st = plan_bias(pop, P, tables, &T->bias)) != EMR_OK) return st;
  return tile_geo_table(P.depth, &T->geo, &T->geo_rows);
}

// Workspaces whose counters a record call left cleared: its k_scan zeroes every pair total and
// its k_move every tile-group mark, so the next record call of the same plan on the same stream
// (stream order puts it after those kernels) needs no clearing launch. Any other call with the
// workspace forgets it. (A few entries: the latest workspaces of the process.)
struct CleanWorkspace {
  const void* ws;
  uint64_t plan;
  hipStream_t s;
  int64_t capacity;
};
std::mutex g_clean_mu;
std::vector<CleanWorkspace> g_clean;
constexpr size_t kCleanEntries = 64;

bool workspace_clean(const void* ws, const Plan& P, hipStream_t s, int64_t capacity) {
  std::lock_guard<std::mutex> lock(g_clean_mu);
  for (const CleanWorkspace& c : g_clean)
    if (c.ws == ws) return c.plan == P.id && c.s == s && c.capacity == capacity;
  return false;
}
void workspace_forget(const void* ws) {
  std::lock_guard<std::mutex> lock(g_clean_mu);
  for (size_t i = 0; i < g_clean.size(); ++i)
    if (g_clean[i].ws == ws) {
      g_clean.erase(g_clean.begin() + (std::ptrdiff_t)i);
      return;
    }
}
void workspace_mark_clean(const void* ws, const Plan& P, hipStream_t s, int64_t capacity) {
  std::lock_guard<std::mutex> lock(g_clean_mu);
  for (CleanWorkspace& c : g_clean)
    if (c.ws == ws) {
      c = CleanWorkspace{ws, P.id, s, capacity};
      return;
    }
  if (g_clean.size() >= kCleanEntries) g_clean.erase(g_clean.begin());
  g_clean.push_back(CleanWorkspace{ws, P.id, s, capacity});
}

// Enqueue a whole call: take a flag slot, then every tile of every pair.
emr_status run_plan(const emr_population* pop, const Plan& P, float theta, const emr_result* out,
                    float* raw, void* workspace, int64_t workspace_bytes, hipStream_t s) {
  emr_status st = check_call_workspace(workspace, workspace_bytes,
                                       (int64_t)workspace_need(P, out ? out->capacity : 0));
  if (st != EMR_OK) return st;
  CallTables T;
  if ((st = call_tables(pop, P, &T)) != EMR_OK) return st;
  CallFlags f;
  if ((st = take_flags(workspace, s, &f)) != EMR_OK) return st;
  bool jit = false;
  if ((st = jit_use(pop, P, plan_slots(P), &jit)) != EMR_OK) return st;
  const bool records = out != nullptr && raw == nullptr;
  const int64_t capacity = records ? out->capacity : -1;
  const bool clean = records && workspace_clean(workspace, P, s, capacity);
  workspace_forget(workspace);
  st = launch_range(pop, P, T, theta, out, raw, workspace, s, 0, P.tiles, jit, f.dev, f.host_dev,
                    true, !clean);
  if (st != EMR_OK) return st;
  if (records) workspace_mark_clean(workspace, P, s, capacity);
  f.ok = true;
  return EMR_OK;
}

}  // namespace

namespace emr {
// Sets the calling thread's last error from other host modules of the library.
emr_status set_error(emr_status st, const std::string& msg) {
  g_err = msg;
  return st;
}
}  // namespace emr

extern "C" {

const char* emr_last_error(void) { return g_err.c_str(); }

int32_t emr_version(void) { return 100; }

emr_status emr_grid_count(int32_t depth, int64_t* n_positions, int64_t* n_parents) {
  if (depth < 0 || depth > EMR_MAX_DEPTH)
    return fail(EMR_E_INVAL, "depth %d outside [0, %d]", depth, EMR_MAX_DEPTH);
  if (n_positions) *n_positions = emr::n_positions(depth);
  if (n_parents) *n_parents = emr::n_parents(depth);
  return EMR_OK;
}

emr_status emr_build_grids(int32_t depth, float* xy_dev, void* stream) {
  if (depth < 0 || depth > EMR_MAX_DEPTH)
    return fail(EMR_E_INVAL, "depth %d outside [0, %d]", depth, EMR_MAX_DEPTH);
  const int64_t n = emr::n_positions(depth);
  if (n > 0 && !xy_dev) return fail(EMR_E_INVAL, "xy_dev is NULL");
  HIP_OR_FAIL(emr_launch_grid(xy_dev, n, (hipStream_t)stream));
  return EMR_OK;
}

}  // extern "C"

namespace {

// Packs genomes on host threads (emr::pack_genomes: each thread a contiguous range into its own
// word vector, then the vectors concatenated and their genomes' descriptors moved by the vector's
// base), and uploads the tables through pinned staging. *bad_index receives the lowest failing
// genome.
emr_status pack_and_upload(int32_t n, const std::function<emr_genome(int32_t)>& genome_at,
                           emr_population** out, int32_t* bad_index) {
  std::vector<emr::ProgDesc> desc;
  std::vector<emr::GenomeInfo> info;
  std::vector<uint32_t> words;
  const int n_threads = std::max(1, std::min({WorkerPool::get().size(), 16, n / 32}));
  std::string msg;
  int32_t bad = -1;
  emr_status pst = emr::pack_genomes(
      n, genome_at, n_threads,
      [](int k, const std::function<void(int)>& f) { WorkerPool::get().run(k, f); }, &desc, &info,
      &words, &bad, &msg);
  if (pst != EMR_OK) {
    if (bad_index && bad >= 0) *bad_index = bad;
    return fail(pst, "%s", msg.c_str());
  }
  const size_t total = words.size();
  emr_population* pop = new (std::nothrow) emr_population;
  if (!pop) return fail(EMR_E_NOMEM, "host allocation failed");
  std::unique_ptr<emr_population, void (*)(emr_population*)> guard(pop, emr_free_population);
  pop->n_genomes = n;
  pop->desc = std::move(desc);
  pop->info = std::move(info);
  pop->blob_words = total;
  const size_t blob_bytes = total * 4, desc_bytes = std::max<size_t>(1, pop->desc.size()) *
                                                    sizeof(emr::ProgDesc);
  if (hipMalloc((void**)&pop->d_blob, blob_bytes) != hipSuccess ||
      hipMalloc((void**)&pop->d_desc, desc_bytes) != hipSuccess)
    return fail(EMR_E_NOMEM, "device allocation of %zu words failed", total);
  // one pinned image (words, then descriptors), copied on a library stream and waited for: the
  // tables are complete on the device before the call returns, whatever stream reads them next
  static std::mutex up_mu;
  static void* up_buf = nullptr;
  static size_t up_size = 0;
  std::lock_guard<std::mutex> lock(up_mu);
  if (up_size < blob_bytes + desc_bytes) {
    if (up_buf) (void)hipHostFree(up_buf);
    up_buf = nullptr;
    up_size = 0;
    const size_t want = std::max<size_t>(blob_bytes + desc_bytes, size_t(4) << 20);
    if (hipHostMalloc(&up_buf, want, hipHostMallocDefault) != hipSuccess)
      return fail(EMR_E_NOMEM, "pinned upload staging of %zu bytes failed", want);
    up_size = want;
  }
  pop->h_blob = std::move(words);
  char* img = (char*)up_buf;
  std::memcpy(img, pop->h_blob.data(), blob_bytes);
  std::memcpy(img + blob_bytes, pop->desc.data(), pop->desc.size() * sizeof(emr::ProgDesc));
  StreamPool* sp = nullptr;
  emr_status st = stream_pool(&sp);
  if (st != EMR_OK) return st;
  HIP_OR_FAIL(hipMemcpyAsync(pop->d_blob, img, blob_bytes, hipMemcpyHostToDevice, sp->aux[0]));
  if (!pop->desc.empty())
    HIP_OR_FAIL(hipMemcpyAsync(pop->d_desc, img + blob_bytes,
                               pop->desc.size() * sizeof(emr::ProgDesc), hipMemcpyHostToDevice,
                               sp->aux[0]));
  HIP_OR_FAIL(hipStreamSynchronize(sp->aux[0]));
  *out = guard.release();
  return EMR_OK;
}

}  // namespace

extern "C" {

emr_status emr_pack_population(const emr_genome* genomes, int32_t n, emr_population** out,
                               int32_t* bad_index) {
  if (bad_index) *bad_index = -1;
  if (!out) return fail(EMR_E_INVAL, "out is NULL");
  if (n < 0 || (n > 0 && !genomes)) return fail(EMR_E_INVAL, "bad genome array");
  return pack_and_upload(n, [&](int32_t g) { return genomes[g]; }, out, bad_index);
}

emr_status emr_pack_population_flat(int32_t n, const int64_t* node_off, const uint8_t* kind,
                                    const uint8_t* act, const float* bias, const int64_t* edge_off,
                                    const int32_t* src, const int32_t* dst, const float* w,
                                    const uint8_t* enabled, emr_population** out,
                                    int32_t* bad_index) {
  if (bad_index) *bad_index = -1;
  if (!out) return fail(EMR_E_INVAL, "out is NULL");
  if (n < 0 || (n > 0 && (!node_off || !edge_off))) return fail(EMR_E_INVAL, "bad offsets");
  if (n > 0 && (node_off[0] != 0 || edge_off[0] != 0))
    return fail(EMR_E_INVAL, "node_off[0] and edge_off[0] must be 0");
  for (int32_t g = 0; g < n; ++g) {
    const int64_t nn = node_off[g + 1] - node_off[g], ne = edge_off[g + 1] - edge_off[g];
    if (nn < 0 || ne < 0 || nn > EMR_MAX_NODES || ne > EMR_MAX_EDGES) {
      if (bad_index) *bad_index = g;
      return fail(nn < 0 || ne < 0 ? EMR_E_INVAL : EMR_E_LIMIT,
                  "genome %d: %lld nodes, %lld edges", g, (long long)nn, (long long)ne);
    }
  }
  if (n > 0 && ((node_off[n] > 0 && (!kind || !act)) ||
                (edge_off[n] > 0 && (!src || !dst || !w))))
    return fail(EMR_E_INVAL, "a node or edge array is NULL");
  auto at = [&](int32_t g) {
    emr_genome e;
    const int64_t n0 = node_off[g], e0 = edge_off[g];
    e.n_nodes = (int32_t)(node_off[g + 1] - n0);
    e.n_edges = (int32_t)(edge_off[g + 1] - e0);
    e.kind = kind ? kind + n0 : nullptr;
    e.act = act ? act + n0 : nullptr;
    e.bias = bias ? bias + n0 : nullptr;
    e.src = src ? src + e0 : nullptr;
    e.dst = dst ? dst + e0 : nullptr;
    e.w = w ? w + e0 : nullptr;
    e.enabled = enabled ? enabled + e0 : nullptr;
    return e;
  };
  return pack_and_upload(n, at, out, bad_index);
}

void emr_free_population(emr_population* pop) {
  if (!pop) return;
  if (pop->d_blob) (void)hipFree(pop->d_blob);
  if (pop->d_desc) (void)hipFree(pop->d_desc);
  delete pop;
}

emr_status emr_population_info(const emr_population* pop, int32_t* n_genomes, int32_t* steps2,
                               int32_t* var_edges2, int32_t* window) {
  if (!pop) return fail(EMR_E_INVAL, "population is NULL");
  if (n_genomes) *n_genomes = pop->n_genomes;
  for (int32_t g = 0; g < pop->n_genomes; ++g) {
    for (int d = 0; d < 2; ++d) {
      const emr::GenomeInfo& inf = pop->info[2 * g + d];
      if (steps2) steps2[2 * g + d] = inf.n_steps;
      if (var_edges2) var_edges2[2 * g + d] = inf.fma_xy + inf.fma_node;
    }
    if (window)
      window[g] = std::max(pop->info[2 * g].window, pop->info[2 * g + 1].window);
  }
  return EMR_OK;
}

emr_status emr_workspace_bytes(const emr_population* pop, const emr_source* sources,
                               int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                               int32_t depth, int64_t capacity, int64_t* bytes) {
  if (!bytes) return fail(EMR_E_INVAL, "bytes is NULL");
  if (capacity < 0 || capacity > (int64_t)0xFFFFFFFFll)
    return fail(EMR_E_INVAL, "capacity %lld outside [0, 2^32 - 1]", (long long)capacity);
  std::shared_ptr<const Plan> plan;
  emr_status st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  *bytes = (int64_t)workspace_need(*plan, capacity);
  return EMR_OK;
}

emr_status emr_discover(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                        const int32_t* src_offsets, int32_t n_shared, int32_t depth, float theta,
                        const emr_result* out, void* stream) {
  if (!out) return fail(EMR_E_INVAL, "out is NULL");
  std::shared_ptr<const Plan> plan;
  emr_status st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  const Plan& P = *plan;
  if (out->capacity < 0 || out->capacity > (int64_t)0xFFFFFFFFll)
    return fail(EMR_E_INVAL, "capacity %lld outside [0, 2^32 - 1]", (long long)out->capacity);
  if (!out->pair_offset) return fail(EMR_E_INVAL, "pair_offset is NULL");
  if (P.n_pairs > 0 && !out->pair_count) return fail(EMR_E_INVAL, "pair_count is NULL");
  if (out->capacity > 0 && (!out->parent || !out->w4))
    return fail(EMR_E_INVAL, "parent/w4 is NULL with capacity > 0");
  return run_plan(pop, P, theta, out, nullptr, out->workspace, out->workspace_bytes,
                  (hipStream_t)stream);
}

emr_status emr_call_check(const void* workspace, int64_t capacity, int64_t* total,
                          int64_t* max_count, void* stream) {
  (void)stream;
  if (!workspace) return fail(EMR_E_INVAL, "workspace is NULL");
  // the flag slot of the latest call with this workspace
  hipEvent_t ev = nullptr;
  const uint32_t* host = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_ring_mu);
    FlagRing* R = nullptr;
    emr_status st = flag_ring(&R);
    if (st != EMR_OK) return st;
    uint64_t latest = 0;
    for (int k = 0; k < kFlagSlots; ++k)
      if (R->ws[k] == workspace && R->seq[k] > latest) {
        latest = R->seq[k];
        ev = R->done[k];
        host = R->host + (size_t)k * kSlotWords;
      }
  }
  if (!ev)
    return fail(EMR_E_INVAL, "no call with this workspace among the last %d calls on this device",
                kFlagSlots);
  HIP_OR_FAIL(hipEventSynchronize(ev));
  const uint32_t err = host[emr::kFlagErr];
  const int64_t mx = host[emr::kFlagMax];
  const int64_t found = (int64_t)(((uint64_t)host[emr::kFlagTotal + 1] << 32) |
                                  host[emr::kFlagTotal]);
  if (max_count) *max_count = mx;
  if (total) *total = found;
  if (err)
    return fail(EMR_E_DEVICE, "kernel reported error flags 0x%x (2: a table entry out of range)",
                err);
  if (found > capacity)
    return fail(EMR_E_CAPACITY, "the call found %lld entries; the capacity is %lld",
                (long long)found, (long long)capacity);
  return EMR_OK;
}

emr_status emr_result_check(const emr_result* out, int64_t* total, int64_t* max_count,
                            void* stream) {
  if (!out) return fail(EMR_E_INVAL, "out is NULL");
  return emr_call_check(out->workspace, out->capacity, total, max_count, stream);
}

emr_status emr_eval_raw(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                        const int32_t* src_offsets, int32_t n_shared, int32_t depth, float* out_dev,
                        void* workspace, int64_t workspace_bytes, void* stream) {
  std::shared_ptr<const Plan> plan;
  emr_status st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  const Plan& P = *plan;
  if (P.n_pairs > 0 && emr::n_positions(depth) > 0 && !out_dev)
    return fail(EMR_E_INVAL, "out_dev is NULL");
  return run_plan(pop, P, 0.0f, nullptr, out_dev, workspace, workspace_bytes, (hipStream_t)stream);
}

emr_status emr_eval_raw_noalloc(const emr_population* pop, const emr_source* sources,
                                int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                                int32_t depth, float* out_dev, uint32_t* err_dev, void* stream) {
  if (!pop) return fail(EMR_E_INVAL, "population is NULL");
  if (!err_dev) return fail(EMR_E_INVAL, "err_dev is NULL");
  // The plan: one of the population's host-only plans, built on first use for these arguments.
  std::shared_ptr<const Plan> plan;
  {
    std::lock_guard<std::mutex> lock(pop->plan_mu);
    for (const auto& q : pop->noalloc_plans)
      if ((n_sources == 0 || sources) && n_sources >= 0 &&
          plan_matches(*q, sources, n_sources, src_offsets, n_shared, depth, pop->n_genomes)) {
        plan = q;
        break;
      }
  }
  if (!plan) {
    auto P = std::make_shared<Plan>();
    emr_status st = build_plan(pop, sources, n_sources, src_offsets, n_shared, depth, P.get());
    if (st != EMR_OK) return st;
    std::lock_guard<std::mutex> lock(pop->plan_mu);
    pop->noalloc_plans.push_back(P);
    plan = P;
  }
  const Plan& P = *plan;
  if (P.n_pairs > 0 && emr::n_positions(depth) > 0 && !out_dev)
    return fail(EMR_E_INVAL, "out_dev is NULL");
  // Scratch layout: the plan's tables, the tile geometry rows, the bias rows, then the workspace.
  const int64_t geo_rows = P.tiles + emr::kGeoPadRows;
  const size_t off_geo = align256(P.img.size());
  const size_t off_bias = align256(off_geo + (size_t)geo_rows * 16);
  const size_t off_ws = align256(off_bias + P.bias_table_floats() * sizeof(float));
  const size_t need = off_ws + P.total;
  if (need > (size_t)EMR_NOALLOC_SCRATCH_BYTES)
    return fail(EMR_E_LIMIT, "the call needs %zu bytes of scratch; the allocation-free scratch "
                "holds %d", need, EMR_NOALLOC_SCRATCH_BYTES);
  void* base = nullptr;
  HIP_OR_FAIL(emr_noalloc_scratch(&base));
  char* scr = (char*)base;
  const hipStream_t s = (hipStream_t)stream;
  CallTables T;
  T.tables = scr;
  T.geo = (const uint32_t*)(scr + off_geo);
  T.geo_rows = (uint32_t)geo_rows;
  T.bias = (const float*)(scr + off_bias);
  char* ws = scr + off_ws;
  // The call's first kernel clears the caller's error word; then the tables, the geometry and the
  // bias rows (the bind kernel, each call: they live in the shared scratch).
  HIP_OR_FAIL(emr_launch_fill(err_dev, 1, 0u, s));
  HIP_OR_FAIL(hipMemcpyAsync(scr, P.img.data(), P.img.size(), hipMemcpyHostToDevice, s));
  HIP_OR_FAIL(emr_launch_tile_geo((uint32_t*)(scr + off_geo), (uint32_t)P.tiles,
                                  (uint32_t)geo_rows, s));
  const emr::BindArgs bind = bind_args(pop, P, scr, (float*)(scr + off_bias), err_dev);
  HIP_OR_FAIL(emr_launch_bind(&bind, s));
  return launch_range(pop, P, T, 0.0f, nullptr, out_dev, ws, s, 0, P.tiles, false, err_dev,
                      nullptr, false, false, false);
}

emr_status emr_discover_cost(const emr_population* pop, const emr_source* sources,
                             int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                             int32_t depth, double transcendental_slots, double* slots,
                             double* queries, double* evaluated, double* flops) {
  std::shared_ptr<const Plan> plan;
  emr_status st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  const Plan& P = *plan;
  const double npos = (double)emr::n_positions(depth);
  double total = 0.0, varying = 0.0, fl = 0.0;
  for (const Plan::Bucket& b : P.buckets)
    for (uint32_t g = b.first; g < b.first + b.count; ++g) {
      // the group's S sources, walked together (members of one program)
      const emr::GenomeInfo& inf = pop->info[P.members[P.group_member0[g]].desc];
      total += b.S * query_slots(inf, transcendental_slots, b.S) * npos;
      if (inf.out_varying) {
        varying += b.S * npos;
        fl += b.S * query_flops(inf, b.S) * npos;
      }
    }
  if (slots) *slots = total;
  if (queries) *queries = (double)P.n_pairs * npos;
  if (evaluated) *evaluated = varying;
  if (flops) *flops = fl;
  return EMR_OK;
}

emr_status emr_set_jit(int32_t policy) {
  if (policy != EMR_JIT_OFF && policy != EMR_JIT_AUTO && policy != EMR_JIT_ALWAYS)
    return fail(EMR_E_INVAL, "compiled-tier policy %d (0 off, 1 auto, 2 always)", policy);
  g_jit_policy.store(policy);
  return EMR_OK;
}

emr_status emr_jit_info(const emr_population* pop, int32_t* state, int64_t* programs,
                        int64_t* code_bytes, double* compile_ms, double* load_ms) {
  if (!pop) return fail(EMR_E_INVAL, "population is NULL");
  std::shared_ptr<const Plan> plan;
  {
    std::lock_guard<std::mutex> lock(pop->plan_mu);
    plan = pop->plan;
  }
  int32_t st = 0;
  int64_t np = 0, nb = 0;
  double cm = 0.0, lm = 0.0;
  if (plan) {
    std::lock_guard<std::mutex> lock(plan->jit_mu);
    st = plan->jit_state;
    if (st == 1) {
      np = (int64_t)plan->jit->programs;
      nb = (int64_t)plan->jit->program_bytes;
      cm = plan->jit->compile_ms;
      lm = plan->jit->load_ms;
    } else if (st == -1) {
      g_err = plan->jit_error;
    }
  }
  if (state) *state = st;
  if (programs) *programs = np;
  if (code_bytes) *code_bytes = nb;
  if (compile_ms) *compile_ms = cm;
  if (load_ms) *load_ms = lm;
  return EMR_OK;
}

emr_status emr_profile_enable(int32_t on, int32_t every, double transcendental_slots) {
  if (on < 0 || on > 2) return fail(EMR_E_INVAL, "profile mode %d (0 off, 1 every launch, 2 first)", on);
  if (every < 1) return fail(EMR_E_INVAL, "profile every %d calls", every);
  g_prof.on = on != 0;
  g_prof.first_only = on == 2;
  g_prof.every = every;
  g_prof.seen = 0;
  g_prof.rT = transcendental_slots;
  g_prof.recs.clear();
  g_prof.calls = 0;
  return EMR_OK;
}

emr_status emr_profile_read(emr_launch_profile* out, int32_t cap, int32_t* n) {
  Profiler& prof = g_prof;
  if (n) *n = (int32_t)prof.recs.size();
  if (!out) return EMR_OK;
  for (size_t i = 0; i < prof.recs.size(); ++i) {
    HIP_OR_FAIL(hipEventSynchronize(prof.events[2 * i + 1]));
    float ms = 0.0f;
    HIP_OR_FAIL(hipEventElapsedTime(&ms, prof.events[2 * i], prof.events[2 * i + 1]));
    prof.recs[i].ms = ms;
    if ((int32_t)i < cap) out[i] = prof.recs[i];
  }
  prof.recs.clear();
  prof.calls = 0;
  return EMR_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ streaming
namespace {

// The buffers, side stream and events of one streamed call. A call takes an idle set of its
// device from a process-wide cache (or a new one), grows what is too small, and gives the set back
// when it is done with it, so repeated streamed calls allocate nothing (a set is kept until the
// process ends: at most the largest call's buffers per concurrent streamed call). The destructor
// drains both streams first, so an early return (an error, or a sink that stops the run) never
// hands over memory that a queued kernel or copy still uses.
struct StreamSet {
  int device = -1;
  hipStream_t side = nullptr;
  hipEvent_t ev_count[2] = {}, ev_copy[2] = {};
  void* ws = nullptr;               // workspace, with the chunk's record pool
  int64_t* counts = nullptr;        // per-pair counts and offsets of the current chunk
  int64_t* offsets = nullptr;
  uint32_t* g_parent[2] = {};       // each chunk's records (CSR), double buffered
  float* g_w4[2] = {};
  int64_t* counts_h[2] = {};        // pinned: a chunk's counts, then its error flags (one word)
  int64_t* counts_h_dev[2] = {};    // the same words, device view (k_scan writes them)
  uint32_t* stage_parent[2] = {};   // pinned staging of a chunk's records
  float* stage_w4[2] = {};
  int64_t stage_cap[2] = {0, 0};
  int64_t ws_bytes = 0, count_pairs = 0, g_records = 0, counts_h_pairs = 0;
};
std::mutex g_stream_sets_mu;
std::vector<StreamSet*> g_stream_sets;  // idle sets

struct StreamRun : StreamSet {
  hipStream_t s = nullptr;
  bool copy_pending[2] = {false, false};
  StreamRun() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return;
    std::lock_guard<std::mutex> lock(g_stream_sets_mu);
    for (size_t k = 0; k < g_stream_sets.size(); ++k)
      if (g_stream_sets[k]->device == dev) {
        static_cast<StreamSet&>(*this) = *g_stream_sets[k];
        delete g_stream_sets[k];
        g_stream_sets.erase(g_stream_sets.begin() + (ptrdiff_t)k);
        return;
      }
    device = dev;
  }
  ~StreamRun() {
    // nothing queued may still use the set when the next call takes it
    if (s) (void)hipStreamSynchronize(s);
    if (side) (void)hipStreamSynchronize(side);
    std::lock_guard<std::mutex> lock(g_stream_sets_mu);
    g_stream_sets.push_back(new StreamSet(static_cast<const StreamSet&>(*this)));
  }
};

// Device buffer *p of at least `bytes` (256 or more), keeping the current one when it is large
// enough; *have is its size.
bool reserve_device(void** p, int64_t* have, int64_t bytes) {
  bytes = std::max<int64_t>(bytes, 256);
  if (*p && *have >= bytes) return true;
  if (*p) (void)hipFree(*p);
  *p = nullptr;
  *have = 0;
  if (hipMalloc(p, (size_t)bytes) != hipSuccess) {
    *p = nullptr;
    return false;
  }
  *have = bytes;
  return true;
}

// Largest device footprint of one streamed call's record buffers (the pool + two chunk outputs).
constexpr int64_t kStreamBufferLimit = int64_t(48) << 30;

}  // namespace

extern "C" {

emr_status emr_stream_chunks(int32_t depth, int64_t chunk_positions, int64_t* n_chunks) {
  if (depth < 0 || depth > EMR_MAX_DEPTH)
    return fail(EMR_E_INVAL, "depth %d outside [0, %d]", depth, EMR_MAX_DEPTH);
  if (chunk_positions < emr::kTile || chunk_positions % emr::kTile != 0)
    return fail(EMR_E_INVAL, "chunk_positions=%lld must be a positive multiple of %d",
                (long long)chunk_positions, emr::kTile);
  if (!n_chunks) return fail(EMR_E_INVAL, "n_chunks is NULL");
  const int64_t tpc = chunk_positions / emr::kTile, tiles = emr::tiles_per_pair(depth);
  *n_chunks = (tiles + tpc - 1) / tpc;
  return EMR_OK;
}

emr_status emr_discover_stream(const emr_population* pop, const emr_source* sources,
                               int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                               int32_t depth, float theta, int64_t chunk_positions, int64_t start,
                               emr_sink sink, void* user, int64_t* next, void* stream) {
  if (next) *next = start;
  if (!sink) return fail(EMR_E_INVAL, "sink is NULL");
  int64_t n_chunks = 0;
  emr_status st = emr_stream_chunks(depth, chunk_positions, &n_chunks);
  if (st != EMR_OK) return st;
  std::shared_ptr<const Plan> plan;
  st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  const Plan& P = *plan;
  const int64_t n_pairs = P.n_pairs, tpc = chunk_positions / emr::kTile;
  const int64_t total = n_chunks * n_pairs;
  if (start < 0 || start > total)
    return fail(EMR_E_INVAL, "start=%lld outside [0, %lld]", (long long)start, (long long)total);
  if (start == total) {
    if (next) *next = total;
    return EMR_OK;
  }
  // A chunk keeps at most 64 parents per tile of each pair, and never more than Q(D) per pair.
  const int64_t per_pair = std::min<int64_t>(tpc * (emr::kTile / 4), emr::n_parents(depth));
  const int64_t records = n_pairs * per_pair;  // the pool's and each chunk output's capacity
  const int64_t set_bytes = records * 20;
  if (records > (int64_t)0xFFFFFFFFll || set_bytes > kStreamBufferLimit / 3)
    return fail(EMR_E_LIMIT, "%lld pairs x %lld-position chunks need %lld bytes of record buffers; "
                "use smaller chunks", (long long)n_pairs, (long long)chunk_positions,
                (long long)(3 * set_bytes));

  StreamRun R;
  R.s = (hipStream_t)stream;
  if (!R.side) HIP_OR_FAIL(hipStreamCreateWithFlags(&R.side, hipStreamNonBlocking));
  for (int b = 0; b < 2; ++b) {
    if (!R.ev_count[b]) HIP_OR_FAIL(hipEventCreateWithFlags(&R.ev_count[b], hipEventDisableTiming));
    if (!R.ev_copy[b]) HIP_OR_FAIL(hipEventCreateWithFlags(&R.ev_copy[b], hipEventDisableTiming));
  }
  const int64_t ws_need = (int64_t)workspace_need(P, records);
  int64_t have = 0;
  bool ok = reserve_device(&R.ws, &R.ws_bytes, ws_need);
  if (ok && R.count_pairs < n_pairs + 1) {
    have = R.count_pairs * 8;
    ok = reserve_device((void**)&R.counts, &have, (n_pairs + 1) * 8);
    have = R.count_pairs * 8;
    ok = ok && reserve_device((void**)&R.offsets, &have, (n_pairs + 1) * 8);
    R.count_pairs = ok ? n_pairs + 1 : 0;
  }
  if (!ok)
    return fail(EMR_E_NOMEM, "device buffers of a streamed call (%lld bytes of workspace)",
                (long long)ws_need);
  if (R.g_records < records) {
    for (int b = 0; b < 2 && ok; ++b) {
      have = R.g_records * 4;
      ok = reserve_device((void**)&R.g_parent[b], &have, records * 4);
      have = R.g_records * 16;
      ok = ok && reserve_device((void**)&R.g_w4[b], &have, records * 16);
    }
    R.g_records = ok ? records : 0;
    if (!ok) return fail(EMR_E_NOMEM, "record buffers of a streamed call");
  }
  if (R.counts_h_pairs < n_pairs + 1) {
    for (int b = 0; b < 2; ++b) {
      if (R.counts_h[b]) (void)hipHostFree(R.counts_h[b]);
      R.counts_h[b] = nullptr;
      R.counts_h_dev[b] = nullptr;
    }
    R.counts_h_pairs = 0;
    for (int b = 0; b < 2; ++b)
      if (hipHostMalloc((void**)&R.counts_h[b], (size_t)(n_pairs + 1) * 8, hipHostMallocDefault) !=
              hipSuccess ||
          hipHostGetDevicePointer((void**)&R.counts_h_dev[b], R.counts_h[b], 0) != hipSuccess)
        return fail(EMR_E_NOMEM, "pinned counts of a streamed call");
    R.counts_h_pairs = n_pairs + 1;
  }

  CallTables T;
  st = call_tables(pop, P, &T);
  if (st != EMR_OK) return st;
  if ((st = check_call_workspace(R.ws, R.ws_bytes, ws_need)) != EMR_OK) return st;
  CallFlags f;  // the chunks raise into its words, handed over once at the end
  st = take_flags(nullptr, R.s, &f);
  if (st != EMR_OK) return st;
  bool jit = false;
  st = jit_use(pop, P, plan_slots(P) * (double)(total - start) / (double)total, &jit);
  if (st != EMR_OK) return st;

  // Chunk c on the compute stream: discover + compact over its tiles into buffer c & 1, then its
  // counts and the call's error word to pinned memory.
  auto enqueue = [&](int64_t c) -> emr_status {
    const int b = (int)(c & 1);
    if (R.copy_pending[b]) HIP_OR_FAIL(hipStreamWaitEvent(R.s, R.ev_copy[b], 0));
    const int64_t tile_lo = c * tpc, n = std::min<int64_t>(tpc, P.tiles - tile_lo);
    emr_result chunk_out{R.g_parent[b], R.g_w4[b], records, R.counts, R.offsets, R.ws,
                         R.ws_bytes};
    // k_scan also writes the chunk's counts and the call's error bits to the pinned words
    emr_status e = launch_range(pop, P, T, theta, &chunk_out, nullptr, R.ws, R.s, tile_lo, n, jit,
                                f.dev, f.host_dev, false, true, true, R.counts_h_dev[b]);
    if (e != EMR_OK) return e;
    HIP_OR_FAIL(hipEventRecord(R.ev_count[b], R.s));
    return EMR_OK;
  };

  const int64_t c0 = start / n_pairs, skip = start % n_pairs;
  st = enqueue(c0);
  if (st != EMR_OK) return st;
  for (int64_t c = c0; c < n_chunks; ++c) {
    const int b = (int)(c & 1);
    if (c + 1 < n_chunks) {
      st = enqueue(c + 1);  // the GPU computes the next chunk while this one is delivered
      if (st != EMR_OK) return st;
    }
    HIP_OR_FAIL(hipEventSynchronize(R.ev_count[b]));
    // a kernel error raised up to this chunk stops the run before its records are delivered
    const uint32_t err = (uint32_t)R.counts_h[b][n_pairs];
    if (err) {
      if (next) *next = c * n_pairs + (c == c0 ? skip : 0);
      return fail(EMR_E_DEVICE, "kernel reported error flags 0x%x at chunk %lld (2: a table entry "
                  "out of range)", err, (long long)c);
    }
    int64_t n_rec = 0;
    for (int64_t r = 0; r < n_pairs; ++r) n_rec += std::max<int64_t>(R.counts_h[b][r], 0);
    if (n_rec > records)
      return fail(EMR_E_DEVICE, "chunk %lld reports %lld records for a pool of %lld",
                  (long long)c, (long long)n_rec, (long long)records);
    if (n_rec > R.stage_cap[b]) {
      if (R.stage_parent[b]) (void)hipHostFree(R.stage_parent[b]);
      if (R.stage_w4[b]) (void)hipHostFree(R.stage_w4[b]);
      R.stage_parent[b] = nullptr;
      R.stage_w4[b] = nullptr;
      R.stage_cap[b] = 0;
      const int64_t want = std::max<int64_t>(n_rec, int64_t(1) << 16);
      if (hipHostMalloc((void**)&R.stage_parent[b], (size_t)want * 4, hipHostMallocDefault) !=
              hipSuccess ||
          hipHostMalloc((void**)&R.stage_w4[b], (size_t)want * 16, hipHostMallocDefault) !=
              hipSuccess)
        return fail(EMR_E_NOMEM, "pinned staging of %lld records", (long long)want);
      R.stage_cap[b] = want;
    }
    if (n_rec > 0) {
      HIP_OR_FAIL(hipStreamWaitEvent(R.side, R.ev_count[b], 0));
      HIP_OR_FAIL(hipMemcpyAsync(R.stage_parent[b], R.g_parent[b], (size_t)n_rec * 4,
                                 hipMemcpyDeviceToHost, R.side));
      HIP_OR_FAIL(hipMemcpyAsync(R.stage_w4[b], R.g_w4[b], (size_t)n_rec * 16,
                                 hipMemcpyDeviceToHost, R.side));
      HIP_OR_FAIL(hipEventRecord(R.ev_copy[b], R.side));
      R.copy_pending[b] = true;
      HIP_OR_FAIL(hipEventSynchronize(R.ev_copy[b]));
    }
    int64_t off = 0;
    for (int64_t r = 0; r < n_pairs; ++r) {
      const int64_t nr = std::max<int64_t>(R.counts_h[b][r], 0);
      if (nr > 0 && !(c == c0 && r < skip)) {
        if (sink(r, c, R.stage_parent[b] + off, R.stage_w4[b] + 4 * off, nr, user) != 0) {
          if (next) *next = c * n_pairs + r;
          return fail(EMR_E_ABORTED, "the sink stopped the run at chunk %lld, pair %lld",
                      (long long)c, (long long)r);
        }
      }
      off += nr;
    }
    if (next) *next = (c + 1) * n_pairs;
  }
  HIP_OR_FAIL(emr_launch_finalize(f.dev, f.host_dev, R.s));
  HIP_OR_FAIL(hipStreamSynchronize(R.s));
  f.ok = true;
  const uint32_t err = f.host[emr::kFlagErr];
  if (err)
    return fail(EMR_E_DEVICE, "kernel reported error flags 0x%x (2: a table entry out of "
                "range)", err);
  return EMR_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ after discovery
namespace {

// The records of a checked discover call as the phase-2 kernels read them.
emr_status records_in(const emr_result* rec, int64_t n_pairs, int32_t depth, emr::RecordsIn* R) {
  if (!rec) return fail(EMR_E_INVAL, "rec is NULL");
  if (n_pairs < 0 || n_pairs > 0xFFFFFFFFll) return fail(EMR_E_INVAL, "n_pairs %lld", (long long)n_pairs);
  if (depth < 0 || depth > EMR_MAX_DEPTH)
    return fail(EMR_E_INVAL, "depth %d outside [0, %d]", depth, EMR_MAX_DEPTH);
  if (!rec->pair_offset || (n_pairs > 0 && !rec->pair_count))
    return fail(EMR_E_INVAL, "rec has no pair_count / pair_offset");
  if (rec->capacity < 0 || (rec->capacity > 0 && (!rec->parent || !rec->w4)))
    return fail(EMR_E_INVAL, "rec has no records");
  *R = emr::RecordsIn{};
  R->parent = rec->parent;
  R->w4 = rec->w4;
  R->count = rec->pair_count;
  R->offset = rec->pair_offset;
  R->cap = rec->capacity;
  R->n_pairs = (uint32_t)n_pairs;
  R->depth = depth;
  return EMR_OK;
}

// A workspace of at least `need` bytes, 256-byte aligned.
emr_status check_workspace(const void* ws, int64_t bytes, int64_t need) {
  if (!ws || bytes < need)
    return fail(EMR_E_INVAL, "workspace of %lld bytes is smaller than the %lld needed",
                (long long)bytes, (long long)need);
  if (((uintptr_t)ws & 255) != 0) return fail(EMR_E_INVAL, "workspace not 256-byte aligned");
  return EMR_OK;
}

int64_t cell_words(int32_t depth) { return (emr::n_positions(depth) + 31) / 32; }

// Workspace layouts: hidden nodes (fresh bitmap, per-genome totals and counts), expression (per-pair
// totals), chain (membership bitmap, per-pair totals).
struct HiddenLayout {
  size_t fresh = 0, totals = 0, counts = 0, bytes = 0;
  HiddenLayout(int64_t G, int32_t depth) {
    fresh = 0;
    totals = align256((size_t)G * (size_t)cell_words(depth) * 4);
    counts = align256(totals + (size_t)G * 4);
    bytes = align256(counts + (size_t)G * 8);
  }
};
struct ChainLayout {
  size_t member = 0, totals = 0, bytes = 0;
  int64_t qwords = 0;
  ChainLayout(int64_t n_pairs, int32_t depth) {
    qwords = (emr::n_parents(depth) + 31) / 32;
    totals = align256((size_t)n_pairs * (size_t)qwords * 4);
    bytes = align256(totals + (size_t)n_pairs * 4);
  }
};

// The offsets of a phase-2 output (k_scan over per-pair or per-genome totals), which also hands the
// call's flags over.
emr_status scan_totals(uint32_t* totals, int64_t* counts, int64_t* offsets, int64_t n,
                       const CallFlags& f, hipStream_t s) {
  if (n == 0) {
    HIP_OR_FAIL(emr_launch_fill(offsets, 2, 0u, s));
    HIP_OR_FAIL(emr_launch_finalize(f.dev, f.host_dev, s));
    return EMR_OK;
  }
  emr::ScanArgs S{};
  S.pair_total = totals;
  S.pair_count = counts;
  S.pair_offset = offsets;
  S.flags = f.dev;
  S.host = f.host_dev;
  S.n_pairs = (uint32_t)n;
  HIP_OR_FAIL(emr_launch_scan(&S, s));
  return EMR_OK;
}

}  // namespace

extern "C" {

emr_status emr_cell_words(int32_t depth, int64_t* words) {
  if (depth < 0 || depth > EMR_MAX_DEPTH)
    return fail(EMR_E_INVAL, "depth %d outside [0, %d]", depth, EMR_MAX_DEPTH);
  if (!words) return fail(EMR_E_INVAL, "words is NULL");
  *words = cell_words(depth);
  return EMR_OK;
}

emr_status emr_hidden_workspace_bytes(int32_t n_genomes, int32_t depth, int64_t* bytes) {
  if (n_genomes < 0 || depth < 0 || depth > EMR_MAX_DEPTH || !bytes)
    return fail(EMR_E_INVAL, "bad arguments");
  *bytes = (int64_t)HiddenLayout(n_genomes, depth).bytes;
  return EMR_OK;
}

emr_status emr_hidden_sources(const emr_population* pop, const emr_source* sources,
                              int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                              int32_t depth, const emr_result* rec, const emr_hidden* out,
                              void* stream) {
  if (!out) return fail(EMR_E_INVAL, "out is NULL");
  std::shared_ptr<const Plan> plan;
  emr_status st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  const Plan& P = *plan;
  const int64_t G = pop->n_genomes;
  emr::RecordsIn R;
  if ((st = records_in(rec, P.n_pairs, depth, &R)) != EMR_OK) return st;
  if (out->capacity < 0 || out->capacity > 0xFFFFFFFFll || !out->offsets ||
      (out->capacity > 0 && !out->sources))
    return fail(EMR_E_INVAL, "bad hidden-node output buffers");
  const HiddenLayout L(G, depth);
  if ((st = check_workspace(out->workspace, out->workspace_bytes, (int64_t)L.bytes)) != EMR_OK)
    return st;
  CallTables T;
  if ((st = call_tables(pop, P, &T)) != EMR_OK) return st;
  R.pair_info = (const uint32_t*)(T.tables + P.t_pairinfo);
  R.src_xy = (const float*)(T.tables + P.t_srcxy);
  const hipStream_t s = (hipStream_t)stream;
  CallFlags f;
  if ((st = take_flags(out->workspace, s, &f)) != EMR_OK) return st;
  char* ws = (char*)out->workspace;
  emr::HiddenArgs A{};
  A.rec = R;
  A.fresh = (uint32_t*)(ws + L.fresh);
  A.known = out->known;
  A.totals = (uint32_t*)(ws + L.totals);
  A.offsets = out->offsets;
  A.out_src = (uint32_t*)out->sources;
  A.out_cell = out->cell;
  A.cap = out->capacity;
  A.words = cell_words(depth);
  A.n_genomes = (uint32_t)G;
  HIP_OR_FAIL(emr_launch_fill(A.fresh, G * A.words, 0u, s));
  HIP_OR_FAIL(emr_launch_hidden(&A, 0, s));
  HIP_OR_FAIL(emr_launch_hidden(&A, 1, s));
  if ((st = scan_totals(A.totals, (int64_t*)(ws + L.counts), out->offsets, G, f, s)) != EMR_OK)
    return st;
  HIP_OR_FAIL(emr_launch_hidden(&A, 2, s));
  f.ok = true;
  return EMR_OK;
}

emr_status emr_express_workspace_bytes(int64_t n_pairs, int64_t* bytes) {
  if (n_pairs < 0 || !bytes) return fail(EMR_E_INVAL, "bad arguments");
  *bytes = (int64_t)align256((size_t)n_pairs * 4);
  return EMR_OK;
}

emr_status emr_express(const emr_population* pop, const emr_source* sources, int32_t n_sources,
                       const int32_t* src_offsets, int32_t n_shared, int32_t depth,
                       const emr_result* rec, int32_t type_mask, float w_min,
                       const emr_connections* out, void* stream) {
  if (!out) return fail(EMR_E_INVAL, "out is NULL");
  if (type_mask < 0 || type_mask > EMR_CONN_ALL)
    return fail(EMR_E_INVAL, "type_mask 0x%x (bits of EMR_CONN_ALL)", type_mask);
  std::shared_ptr<const Plan> plan;
  emr_status st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  const Plan& P = *plan;
  emr::RecordsIn R;
  if ((st = records_in(rec, P.n_pairs, depth, &R)) != EMR_OK) return st;
  if (out->capacity < 0 || !out->pair_offset || (P.n_pairs > 0 && !out->pair_count) ||
      (out->capacity > 0 && (!out->cell || !out->w)))
    return fail(EMR_E_INVAL, "bad connection output buffers");
  if ((st = check_workspace(out->workspace, out->workspace_bytes,
                            (int64_t)align256((size_t)P.n_pairs * 4))) != EMR_OK)
    return st;
  CallTables T;
  if ((st = call_tables(pop, P, &T)) != EMR_OK) return st;
  R.pair_info = (const uint32_t*)(T.tables + P.t_pairinfo);
  R.src_xy = (const float*)(T.tables + P.t_srcxy);
  const hipStream_t s = (hipStream_t)stream;
  CallFlags f;
  if ((st = take_flags(out->workspace, s, &f)) != EMR_OK) return st;
  emr::ExpressArgs A{};
  A.rec = R;
  A.type_mask = (uint32_t)type_mask;
  A.w_min = w_min;
  A.totals = (uint32_t*)out->workspace;
  A.out_offset = out->pair_offset;
  A.out_cell = out->cell;
  A.out_w = out->w;
  A.cap = out->capacity;
  if (P.n_pairs > 0) HIP_OR_FAIL(emr_launch_express(&A, 0, s));
  if ((st = scan_totals(A.totals, out->pair_count, out->pair_offset, P.n_pairs, f, s)) != EMR_OK)
    return st;
  if (P.n_pairs > 0) HIP_OR_FAIL(emr_launch_express(&A, 1, s));
  f.ok = true;
  return EMR_OK;
}

emr_status emr_band_workspace_bytes(int64_t n_pairs, int64_t* bytes) {
  if (n_pairs < 0 || !bytes) return fail(EMR_E_INVAL, "bad arguments");
  *bytes = (int64_t)align256((size_t)n_pairs * sizeof(emr::BandPair));
  return EMR_OK;
}

emr_status emr_band_values(const emr_population* pop, const emr_source* sources,
                           int32_t n_sources, const int32_t* src_offsets, int32_t n_shared,
                           int32_t depth, const emr_connections* conn, float* band,
                           void* workspace, int64_t workspace_bytes, void* stream) {
  if (!conn) return fail(EMR_E_INVAL, "conn is NULL");
  std::shared_ptr<const Plan> plan;
  emr_status st = plan_for(pop, sources, n_sources, src_offsets, n_shared, depth, &plan);
  if (st != EMR_OK) return st;
  const Plan& P = *plan;
  if (P.n_pairs > 0xFFFFFFFFll) return fail(EMR_E_LIMIT, "%lld pairs", (long long)P.n_pairs);
  if (conn->capacity < 0 || !conn->pair_offset ||
      (conn->capacity > 0 && (!conn->cell || !conn->w || !band)))
    return fail(EMR_E_INVAL, "bad connection buffers");
  if ((st = check_workspace(workspace, workspace_bytes,
                            (int64_t)align256((size_t)P.n_pairs * sizeof(emr::BandPair)))) != EMR_OK)
    return st;
  // each pair's program, window and bias rows, from the group that holds it
  std::vector<emr::BandPair> bp((size_t)P.n_pairs, emr::BandPair{0u, 0u, 0u, 0u});
  for (const auto& bk : P.buckets)
    for (uint32_t gi = bk.first; gi < bk.first + bk.count; ++gi) {
      const emr::Group& G = P.groups[gi];
      for (int k = 0; k < bk.S; ++k) {
        const uint32_t pair = G.pair[k];
        if ((int64_t)pair >= P.n_pairs) return fail(EMR_E_DEVICE, "plan: pair %u", pair);
        if (k > 0 && pair == G.pair[k - 1]) break;  // (an unused slot repeats the last pair)
        bp[pair] = emr::BandPair{G.var_off, (G.flags & 1u) ? G.n_rec : 0u, (uint32_t)bk.window,
                                 G.bias_off + (uint32_t)k};
      }
    }
  CallTables T;
  if ((st = call_tables(pop, P, &T)) != EMR_OK) return st;
  const hipStream_t s = (hipStream_t)stream;
  CallFlags f;
  if ((st = take_flags(workspace, s, &f)) != EMR_OK) return st;
  if (P.n_pairs > 0) {
    HIP_OR_FAIL(hipMemcpyAsync(workspace, bp.data(), bp.size() * sizeof(emr::BandPair),
                               hipMemcpyHostToDevice, s));
    HIP_OR_FAIL(hipStreamSynchronize(s));  // (bp is a host temporary)
    emr::BandArgs A{};
    A.blob = pop->d_blob;
    A.bias = T.bias;
    A.pairs = (const emr::BandPair*)workspace;
    A.conn_offset = conn->pair_offset;
    A.conn_cell = conn->cell;
    A.conn_w = conn->w;
    A.band = band;
    A.err = f.dev + emr::kFlagErr;
    A.cap = conn->capacity;
    A.n_pairs = (uint32_t)P.n_pairs;
    A.depth = depth;
    A.blob_words = (uint32_t)pop->blob_words;
    A.bias_floats = (uint32_t)P.bias_table_floats();
    HIP_OR_FAIL(emr_launch_band(&A, s));
  }
  HIP_OR_FAIL(emr_launch_finalize(f.dev, f.host_dev, s));
  f.ok = true;
  return EMR_OK;
}

emr_status emr_band_filter(const emr_connections* in, const float* band, int64_t n_pairs,
                           float theta_band, const emr_connections* out, void* stream) {
  if (!in || !out) return fail(EMR_E_INVAL, "in or out is NULL");
  if (n_pairs < 0 || n_pairs > 0xFFFFFFFFll) return fail(EMR_E_INVAL, "n_pairs %lld", (long long)n_pairs);
  if (std::isnan(theta_band)) return fail(EMR_E_INVAL, "theta_band is NaN");
  if (in->capacity < 0 || !in->pair_offset ||
      (in->capacity > 0 && (!in->cell || !in->w || !band)))
    return fail(EMR_E_INVAL, "bad input connections");
  if (out->capacity < 0 || !out->pair_offset || (n_pairs > 0 && !out->pair_count) ||
      (out->capacity > 0 && (!out->cell || !out->w)))
    return fail(EMR_E_INVAL, "bad output connections");
  emr_status st = check_workspace(out->workspace, out->workspace_bytes,
                                  (int64_t)align256((size_t)n_pairs * 4));
  if (st != EMR_OK) return st;
  const hipStream_t s = (hipStream_t)stream;
  CallFlags f;
  if ((st = take_flags(out->workspace, s, &f)) != EMR_OK) return st;
  emr::BandSelectArgs A{};
  A.in_offset = in->pair_offset;
  A.in_cell = in->cell;
  A.in_w = in->w;
  A.band = band;
  A.in_cap = in->capacity;
  A.theta_band = theta_band;
  A.totals = (uint32_t*)out->workspace;
  A.out_offset = out->pair_offset;
  A.out_cell = out->cell;
  A.out_w = out->w;
  A.out_cap = out->capacity;
  A.n_pairs = (uint32_t)n_pairs;
  if (n_pairs > 0) HIP_OR_FAIL(emr_launch_band_select(&A, 0, s));
  if ((st = scan_totals(A.totals, out->pair_count, out->pair_offset, n_pairs, f, s)) != EMR_OK)
    return st;
  if (n_pairs > 0) HIP_OR_FAIL(emr_launch_band_select(&A, 1, s));
  f.ok = true;
  return EMR_OK;
}

emr_status emr_chain_workspace_bytes(int64_t n_pairs, int32_t depth, int64_t* bytes) {
  if (n_pairs < 0 || depth < 0 || depth > EMR_MAX_DEPTH || !bytes)
    return fail(EMR_E_INVAL, "bad arguments");
  *bytes = (int64_t)ChainLayout(n_pairs, depth).bytes;
  return EMR_OK;
}

emr_status emr_chain_filter(const emr_result* rec, int64_t n_pairs, int32_t depth,
                            const emr_result* out, void* stream) {
  if (!out) return fail(EMR_E_INVAL, "out is NULL");
  emr::RecordsIn R;
  emr_status st = records_in(rec, n_pairs, depth, &R);
  if (st != EMR_OK) return st;
  if (out->capacity < 0 || out->capacity > 0xFFFFFFFFll || !out->pair_offset ||
      (n_pairs > 0 && !out->pair_count) || (out->capacity > 0 && (!out->parent || !out->w4)))
    return fail(EMR_E_INVAL, "bad output buffers");
  const ChainLayout L(n_pairs, depth);
  if ((st = check_workspace(out->workspace, out->workspace_bytes, (int64_t)L.bytes)) != EMR_OK)
    return st;
  const hipStream_t s = (hipStream_t)stream;
  CallFlags f;
  if ((st = take_flags(out->workspace, s, &f)) != EMR_OK) return st;
  char* ws = (char*)out->workspace;
  emr::ChainArgs A{};
  A.rec = R;
  A.member = (uint32_t*)(ws + L.member);
  A.qwords = L.qwords;
  A.totals = (uint32_t*)(ws + L.totals);
  A.out_offset = out->pair_offset;
  A.out_parent = out->parent;
  A.out_w4 = out->w4;
  A.cap = out->capacity;
  if (n_pairs > 0) {
    HIP_OR_FAIL(emr_launch_fill(A.member, n_pairs * L.qwords, 0u, s));
    HIP_OR_FAIL(emr_launch_chain(&A, 0, s));
    HIP_OR_FAIL(emr_launch_chain(&A, 1, s));
  }
  if ((st = scan_totals(A.totals, out->pair_count, out->pair_offset, n_pairs, f, s)) != EMR_OK)
    return st;
  if (n_pairs > 0) HIP_OR_FAIL(emr_launch_chain(&A, 2, s));
  f.ok = true;
  return EMR_OK;
}

}  // extern "C"
