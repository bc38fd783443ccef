// The host side of discovery: packing a population into one table of program words, a call's plan
// (which sources walk together, the launch's buckets, the table image the kernels read, the
// workspace layout) and the bounds check of those tables. No HIP here: the library uploads what
// this file builds, and the CPU tests build and check it through the test shim.
#include "plan.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>

namespace emr {
namespace {

emr_status fail_msg(std::string* msg, emr_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (msg) *msg = buf;
  return st;
}

bool check_fail(std::string* msg, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (msg) *msg = buf;
  return false;
}

}  // namespace

namespace {
// Per query of a source, the work of the nodes shared by the S sources of a walk is paid once
// for all of them: (S - 1) / S of it is left out of each query's count.
double unshared(int S) { return S > 1 ? 1.0 - 1.0 / S : 0.0; }
const double kActOther[6] = {0.0, 1.0, 2.0, 1.0, 1.0, 1.0};  // non-transcendental operations
const double kActTrans[6] = {0.0, 2.0, 2.0, 1.0, 1.0, 0.0};  // transcendental instructions
}  // namespace

double query_base(const GenomeInfo& inf, int S) {
  if (!inf.out_varying) return 0.0;
  double c = inf.fma_xy + inf.fma_node + 2.5, sh = inf.shared_edges;
  for (int a = 0; a < 6; ++a) {
    c += inf.act_count[a] * kActOther[a];
    sh += inf.shared_act_count[a] * kActOther[a];
  }
  return c - unshared(S) * sh;
}

double query_trans(const GenomeInfo& inf, int S) {
  if (!inf.out_varying) return 0.0;
  double c = 0.0, sh = 0.0;
  for (int a = 0; a < 6; ++a) {
    c += inf.act_count[a] * kActTrans[a];
    sh += inf.shared_act_count[a] * kActTrans[a];
  }
  return c - unshared(S) * sh;
}

double query_slots(const GenomeInfo& inf, double rT, int S) {
  return query_base(inf, S) + rT * query_trans(inf, S);
}

double query_flops(const GenomeInfo& inf, int S) {
  if (!inf.out_varying) return 0.0;
  // a multiply-add per edge counts 2, every other operation 1
  double c = 2.0 * (inf.fma_xy + inf.fma_node) + 2.5, sh = 2.0 * inf.shared_edges;
  for (int a = 0; a < 6; ++a) {
    c += inf.act_count[a] * (kActOther[a] + kActTrans[a]);
    sh += inf.shared_act_count[a] * (kActOther[a] + kActTrans[a]);
  }
  return c - unshared(S) * sh;
}

int window_bucket(int window) {
  for (int w : kWindows)
    if (window <= w) return w;
  return -1;
}

emr_status pack_genomes(int32_t n, const std::function<emr_genome(int32_t)>& genome_at,
                        int n_parts, const std::function<void(int, const std::function<void(int)>&)>& run,
                        std::vector<ProgDesc>* desc, std::vector<GenomeInfo>* info,
                        std::vector<uint32_t>* words, int32_t* bad, std::string* msg) {
  if (n < 0) return fail_msg(msg, EMR_E_INVAL, "n_genomes %d", n);
  n_parts = std::max(1, n_parts);
  desc->assign(2 * (size_t)n, ProgDesc{});
  info->assign(2 * (size_t)n, GenomeInfo{});
  struct Part {
    std::vector<uint32_t> words;
    int32_t bad = -1;
    emr_status st = EMR_OK;
    std::string msg;
  };
  std::vector<Part> parts((size_t)n_parts);
  auto range = [&](int t, int32_t* lo, int32_t* hi) {
    *lo = (int32_t)((int64_t)n * t / n_parts);
    *hi = (int32_t)((int64_t)n * (t + 1) / n_parts);
  };
  run(n_parts, [&](int t) {
    int32_t lo, hi;
    range(t, &lo, &hi);
    Part& p = parts[(size_t)t];
    for (int32_t g = lo; g < hi; ++g) {
      emr_status st = EMR_OK;
      std::string m;
      if (!pack_genome(genome_at(g), p.words, &(*desc)[2 * (size_t)g], &(*info)[2 * (size_t)g], &st,
                       &m)) {
        p.bad = g;
        p.st = st;
        p.msg = m;
        return;
      }
      if (p.words.size() > 0xF0000000ull) {
        p.bad = g;
        p.st = EMR_E_LIMIT;
        p.msg = "population too large";
        return;
      }
    }
    while (p.words.size() % kRecWords) p.words.push_back(0u);  // keep bases aligned
  });
  for (const Part& p : parts)
    if (p.bad >= 0) {  // the parts cover increasing genome ranges: the first is the lowest
      if (bad) *bad = p.bad;
      return fail_msg(msg, p.st, "genome %d: %s", p.bad, p.msg.c_str());
    }
  // concatenate, moving each part's descriptors by its base
  size_t total = 16;  // the kernels may read a few words past a program's end
  for (const Part& p : parts) total += p.words.size();
  if (total > 0xF0000000ull) return fail_msg(msg, EMR_E_LIMIT, "population too large");
  words->assign(total, 0u);
  size_t base = 0;
  for (int t = 0; t < n_parts; ++t) {
    int32_t lo, hi;
    range(t, &lo, &hi);
    for (size_t d = 2 * (size_t)lo; d < 2 * (size_t)hi; ++d) {
      (*desc)[d].var_off += (uint32_t)base;
      (*desc)[d].uni_off += (uint32_t)base;
      (*desc)[d].uni_end += (uint32_t)base;
    }
    const std::vector<uint32_t>& w = parts[(size_t)t].words;
    if (!w.empty()) std::memcpy(words->data() + base, w.data(), w.size() * 4);
    base += w.size();
  }
  return EMR_OK;
}

emr_status build_plan_tables(const ProgDesc* desc, const GenomeInfo* info, int32_t n_genomes,
                             const emr_source* sources, int32_t n_sources, const int32_t* offs,
                             int32_t n_shared, int32_t depth, PlanTables* plan, std::string* msg) {
  if (depth < 0 || depth > EMR_MAX_DEPTH)
    return fail_msg(msg, EMR_E_INVAL, "depth %d outside [0, %d]", depth, EMR_MAX_DEPTH);
  if (n_sources < 0 || (n_sources > 0 && !sources))
    return fail_msg(msg, EMR_E_INVAL, "bad sources");
  const int32_t G = n_genomes;
  if (offs) {
    if (offs[0] != 0) return fail_msg(msg, EMR_E_INVAL, "src_offsets[0] must be 0");
    for (int32_t g = 0; g < G; ++g)
      if (offs[g + 1] < offs[g])
        return fail_msg(msg, EMR_E_INVAL, "src_offsets not ascending at %d", g);
    if (offs[G] != n_sources)
      return fail_msg(msg, EMR_E_INVAL, "src_offsets[n_genomes]=%d but n_sources=%d", offs[G],
                      n_sources);
  } else {
    if (n_shared < 0 || n_shared != n_sources)
      return fail_msg(msg, EMR_E_INVAL, "n_shared=%d must equal n_sources=%d", n_shared,
                      n_sources);
  }
  for (int32_t i = 0; i < n_sources; ++i)
    if (sources[i].dir != EMR_DIR_OUT && sources[i].dir != EMR_DIR_IN)
      return fail_msg(msg, EMR_E_INVAL, "source %d has direction %d", i, sources[i].dir);

  PlanTables& P = *plan;  // a freshly made plan
  P.depth = depth;
  P.n_genomes = G;
  P.n_sources = n_sources;
  P.n_pairs = offs ? (int64_t)n_sources : (int64_t)G * n_shared;
  P.tiles = tiles_per_pair(depth);
  if (P.n_pairs > 0xFFFFFFFFll) return fail_msg(msg, EMR_E_LIMIT, "too many pairs");

  // Group each genome's sources by direction, in source order, into sets of <= max_group(window).
  struct TmpGroup {
    Group g;
    int S, window;
    uint32_t desc;
    uint32_t src[kMaxGroup];
    double cost;
  };
  std::vector<TmpGroup> tmp;
  for (int32_t g = 0; g < G; ++g) {
    const int32_t lo = offs ? offs[g] : 0, hi = offs ? offs[g + 1] : n_shared;
    for (int dir = 0; dir < 2; ++dir) {
      const uint32_t di = 2u * (uint32_t)g + (uint32_t)dir;
      const ProgDesc& d = desc[di];
      const int wb = window_bucket(info[di].window);
      if (wb < 0)
        return fail_msg(msg, EMR_E_LIMIT, "genome %d needs a value window of %d", g,
                        info[di].window);
      const int gmax = max_group(wb);
      TmpGroup cur{};
      int n = 0;
      auto flush = [&]() {
        if (n == 0) return;
        cur.S = n;
        cur.window = wb;
        cur.desc = di;
        for (int s = n; s < kMaxGroup; ++s) cur.g.pair[s] = cur.g.pair[n - 1];
        cur.g.var_off = d.var_off;
        cur.g.n_rec = d.n_rec;
        cur.g.n_steps = d.n_steps;
        cur.g.flags = d.flags;
        tmp.push_back(cur);
        cur = TmpGroup{};
        n = 0;
      };
      for (int32_t j = lo; j < hi; ++j) {
        if (sources[j].dir != dir) continue;
        const int64_t pair = offs ? (int64_t)j : (int64_t)g * n_shared + j;
        cur.g.pair[n] = (uint32_t)pair;
        cur.src[n] = (uint32_t)j;
        if (++n == gmax) flush();
      }
      flush();
    }
  }
  // Order groups by bucket; assign bias-table offsets and members. Within a bucket the most
  // expensive programs come first (the round-robin chunk shares of a first call then end with the
  // cheapest); output order does not depend on this order (each pair has its own totals and
  // offsets).
  // per query of a group's source, its S sources walked together
  for (TmpGroup& t : tmp) t.cost = query_slots(info[t.desc], 4.0, t.S);
  auto cost = [](const TmpGroup& t) { return t.cost; };
  std::stable_sort(tmp.begin(), tmp.end(), [&](const TmpGroup& a, const TmpGroup& b) {
    if (a.S != b.S) return a.S < b.S;
    if (a.window != b.window) return a.window < b.window;
    return cost(a) > cost(b);
  });
  P.groups.reserve(tmp.size());
  uint64_t bias = 0;
  for (size_t i = 0; i < tmp.size(); ++i) {
    TmpGroup& t = tmp[i];
    if (P.buckets.empty() || P.buckets.back().S != t.S || P.buckets.back().window != t.window)
      P.buckets.push_back({t.S, t.window, (uint32_t)i, 0, 0.0, 0});
    P.buckets.back().count++;
    if (t.g.flags & 1u) P.buckets.back().varying = P.buckets.back().count;
    P.buckets.back().cost += t.S * cost(t);
    t.g.bias_off = (uint32_t)bias;
    P.group_member0.push_back((uint32_t)P.members.size());
    const uint32_t rows = t.g.n_rec + 2;  // output row, one per record at most, prefetch row
    for (int s = 0; s < t.S; ++s) P.members.push_back({t.desc, t.src[s], (uint32_t)(bias + s), rows});
    bias += 4ull * rows;
    if (bias > 0xFFFFFFFFull) return fail_msg(msg, EMR_E_LIMIT, "bias table too large");
    P.groups.push_back(t.g);
    P.group_cost.push_back((float)cost(t));
  }
  // Part order within the launch: the costliest bucket first (its chunks are handed out first).
  std::stable_sort(P.buckets.begin(), P.buckets.end(),
                   [](const PlanTables::Bucket& a, const PlanTables::Bucket& b) {
                     return a.cost > b.cost;
                   });
  // One launch with every bucket as a part, in cost order.
  if ((int)P.buckets.size() > kMaxBuckets) return fail_msg(msg, EMR_E_LIMIT, "too many buckets");
  if (!P.buckets.empty()) {
    PlanTables::Launch L{};
    for (size_t bi = 0; bi < P.buckets.size(); ++bi) {
      const PlanTables::Bucket& b = P.buckets[bi];
      L.part[L.n_parts++] = (int)bi;
      L.cost += b.cost;
      for (uint32_t g = 0; g < b.count; ++g) {
        const GenomeInfo& inf = info[P.members[P.group_member0[b.first + g]].desc];
        L.slots_base += b.S * query_base(inf, b.S);
        L.slots_trans += b.S * query_trans(inf, b.S);
      }
      L.sources += (double)b.S * b.count;
    }
    P.launches.push_back(L);
  }
  for (const auto& b : P.buckets)
    if ((uint64_t)b.count * (uint64_t)P.tiles > 0xFFFFFFFFull)
      return fail_msg(msg, EMR_E_LIMIT, "too many tiles in one launch");
  P.bias_floats = bias;
  P.src_xy.resize(2 * (size_t)n_sources);
  for (int32_t i = 0; i < n_sources; ++i) {
    P.src_xy[2 * i] = sources[i].x;
    P.src_xy[2 * i + 1] = sources[i].y;
  }

  // workspace: tile status words, group marks, per-pair totals
  P.off_status = 0;
  P.status_bytes = (size_t)P.n_pairs * P.tiles * 8;
  P.off_nz = align256(P.off_status + P.status_bytes);
  P.nz_bytes = (size_t)P.n_pairs * nz_words((uint32_t)P.tiles) * 8;
  P.off_ptotal = align256(P.off_nz + P.nz_bytes);
  P.total = align256(P.off_ptotal + (size_t)P.n_pairs * 4);
  P.clear_words = (int64_t)((P.off_ptotal + (size_t)P.n_pairs * 4 - P.off_nz + 3) / 4);
  // tables
  P.t_groups = 0;
  P.t_members = align256(P.groups.size() * sizeof(Group));
  P.t_srcxy = align256(P.t_members + P.members.size() * sizeof(Member));
  P.t_uniform = align256(P.t_srcxy + P.src_xy.size() * sizeof(float));
  P.t_pairinfo = align256(P.t_uniform + (size_t)P.n_pairs);
  P.img.assign(align256(P.t_pairinfo + (size_t)P.n_pairs * 8) + 256, 0);
  {
    uint32_t* pinfo = (uint32_t*)(P.img.data() + P.t_pairinfo);
    for (int32_t g = 0; g < G; ++g) {
      const int32_t lo = offs ? offs[g] : 0, hi = offs ? offs[g + 1] : n_shared;
      for (int32_t j = lo; j < hi; ++j) {
        const int64_t pair = offs ? (int64_t)j : (int64_t)g * n_shared + j;
        pinfo[2 * pair] = ((uint32_t)g << 1) | (uint32_t)sources[j].dir;
        pinfo[2 * pair + 1] = (uint32_t)j;
      }
    }
  }
  for (const Group& g : P.groups)
    if (!(g.flags & 1u))
      for (int s = 0; s < kMaxGroup; ++s) P.img[P.t_uniform + g.pair[s]] = 1;
  if (!P.groups.empty())
    std::memcpy(P.img.data() + P.t_groups, P.groups.data(), P.groups.size() * sizeof(Group));
  if (!P.members.empty())
    std::memcpy(P.img.data() + P.t_members, P.members.data(), P.members.size() * sizeof(Member));
  if (!P.src_xy.empty())
    std::memcpy(P.img.data() + P.t_srcxy, P.src_xy.data(), P.src_xy.size() * sizeof(float));
  P.key_sources.assign(sources, sources + n_sources);
  P.key_has_offs = offs != nullptr;
  if (offs) P.key_offs.assign(offs, offs + G + 1);
  P.key_n_shared = n_shared;
  return EMR_OK;
}

bool check_plan_tables(const PlanTables& P, const ProgDesc* desc, uint64_t blob_words,
                       std::string* msg) {
  const uint64_t n_desc = 2ull * (uint64_t)P.n_genomes;
  const uint64_t n_pairs = (uint64_t)P.n_pairs;
  // The population's descriptors: the record stream (with the one-record prefetch past its end)
  // and the uniform program inside the program words (what the discover and bind kernels read).
  for (uint64_t d = 0; d < n_desc; ++d) {
    const ProgDesc& x = desc[d];
    if (x.n_rec > kMaxRecords || x.n_steps > x.n_rec || x.var_off % kRecWords != 0 ||
        (uint64_t)x.var_off + (uint64_t)kRecWords * (x.n_rec + 1) > blob_words)
      return check_fail(msg, "descriptor %llu: records %u at word %u (%u steps) outside %llu words",
                        (unsigned long long)d, x.n_rec, x.var_off, x.n_steps,
                        (unsigned long long)blob_words);
    if ((uint64_t)x.uni_off + 4 > x.uni_end || x.uni_end > blob_words)
      return check_fail(msg, "descriptor %llu: uniform program [%u, %u) outside %llu words",
                        (unsigned long long)d, x.uni_off, x.uni_end,
                        (unsigned long long)blob_words);
  }
  // Groups: the same records as their descriptor, their bias rows inside the bias table, their
  // pairs inside the call.
  if (P.group_member0.size() != P.groups.size() || P.group_cost.size() != P.groups.size())
    return check_fail(msg, "group side tables of %zu / %zu entries for %zu groups",
                      P.group_member0.size(), P.group_cost.size(), P.groups.size());
  std::vector<uint8_t> pair_seen(n_pairs, 0);
  for (size_t gi = 0; gi < P.groups.size(); ++gi) {
    const Group& g = P.groups[gi];
    const uint32_t m0 = P.group_member0[gi];
    const uint32_t m1 = gi + 1 < P.groups.size() ? P.group_member0[gi + 1]
                                                 : (uint32_t)P.members.size();
    if (m0 >= m1 || m1 > P.members.size() || m1 - m0 > (uint32_t)kMaxGroup)
      return check_fail(msg, "group %zu: members [%u, %u)", gi, m0, m1);
    const uint32_t S = m1 - m0;
    const uint32_t di = P.members[m0].desc;
    if (di >= n_desc) return check_fail(msg, "group %zu: descriptor %u", gi, di);
    const ProgDesc& x = desc[di];
    if (g.var_off != x.var_off || g.n_rec != x.n_rec || g.n_steps != x.n_steps ||
        g.flags != x.flags)
      return check_fail(msg, "group %zu: records differ from descriptor %u", gi, di);
    if (g.bias_off % 4 != 0 || (uint64_t)g.bias_off + 4ull * (g.n_rec + 2) > P.bias_floats)
      return check_fail(msg, "group %zu: bias rows at %u (%u records) outside %llu floats", gi,
                        g.bias_off, g.n_rec, (unsigned long long)P.bias_floats);
    for (int s = 0; s < kMaxGroup; ++s)
      if (g.pair[s] >= n_pairs)
        return check_fail(msg, "group %zu: pair %u of %llu", gi, g.pair[s],
                          (unsigned long long)n_pairs);
    for (uint32_t s = S; s < (uint32_t)kMaxGroup; ++s)
      if (g.pair[s] != g.pair[S - 1])
        return check_fail(msg, "group %zu: unused slot %u names another pair", gi, s);
    // members: one per source slot, the group's genome and direction, their slot's bias column
    const uint32_t* pinfo = (const uint32_t*)(P.img.data() + P.t_pairinfo);
    for (uint32_t s = 0; s < S; ++s) {
      const Member& m = P.members[m0 + s];
      if (m.desc != di || m.source >= (uint32_t)P.n_sources || m.bias_base != g.bias_off + s ||
          m.bias_rows != g.n_rec + 2)
        return check_fail(msg, "group %zu: member %u (descriptor %u, source %u, bias %u, rows %u)",
                          gi, m0 + s, m.desc, m.source, m.bias_base, m.bias_rows);
      const uint32_t pair = g.pair[s];
      if (pinfo[2 * (size_t)pair] != di || pinfo[2 * (size_t)pair + 1] != m.source)
        return check_fail(msg, "group %zu: pair %u is genome/dir %u source %u, member says %u / %u",
                          gi, pair, pinfo[2 * (size_t)pair], pinfo[2 * (size_t)pair + 1], di,
                          m.source);
      if (pair_seen[pair]++) return check_fail(msg, "pair %u in two groups", pair);
      const uint8_t uniform = (uint8_t)P.img[P.t_uniform + pair];
      if (uniform != ((g.flags & 1u) ? 0 : 1))
        return check_fail(msg, "pair %u: uniform mark %u for flags %u", pair, uniform, g.flags);
    }
  }
  for (uint64_t p = 0; p < n_pairs; ++p)
    if (!pair_seen[p]) return check_fail(msg, "pair %llu in no group", (unsigned long long)p);
  // Buckets and the launch's parts cover the groups in order.
  uint64_t covered = 0;
  for (size_t bi = 0; bi < P.buckets.size(); ++bi) {
    const PlanTables::Bucket& b = P.buckets[bi];
    if ((uint64_t)b.first + b.count > P.groups.size() || b.varying > b.count ||
        max_group(b.window) < b.S)
      return check_fail(msg, "bucket %zu: groups [%u, +%u) of %zu", bi, b.first, b.count,
                        P.groups.size());
    for (uint32_t g = 0; g < b.count; ++g) {
      const Group& x = P.groups[b.first + g];
      const uint32_t m0 = P.group_member0[b.first + g];
      const uint32_t m1 = b.first + g + 1 < P.groups.size() ? P.group_member0[b.first + g + 1]
                                                            : (uint32_t)P.members.size();
      if ((int)(m1 - m0) != b.S || ((x.flags & 1u) != 0) != (g < b.varying))
        return check_fail(msg, "bucket %zu: group %u does not fit it", bi, b.first + g);
    }
    covered += b.count;
  }
  if (covered != P.groups.size())
    return check_fail(msg, "buckets cover %llu of %zu groups", (unsigned long long)covered,
                      P.groups.size());
  for (const PlanTables::Launch& L : P.launches)
    for (int k = 0; k < L.n_parts; ++k)
      if (L.part[k] < 0 || (size_t)L.part[k] >= P.buckets.size())
        return check_fail(msg, "launch part %d names bucket %d", k, L.part[k]);
  // The image's tables follow each other inside it.
  const size_t ends[5][2] = {{P.t_groups, P.groups.size() * sizeof(Group)},
                             {P.t_members, P.members.size() * sizeof(Member)},
                             {P.t_srcxy, P.src_xy.size() * sizeof(float)},
                             {P.t_uniform, (size_t)n_pairs},
                             {P.t_pairinfo, (size_t)n_pairs * 8}};
  for (int k = 0; k < 5; ++k) {
    if (ends[k][0] + ends[k][1] > P.img.size() || (k < 4 && ends[k][0] + ends[k][1] > ends[k + 1][0]))
      return check_fail(msg, "table %d of the image at %zu (+%zu) overlaps or overflows", k,
                        ends[k][0], ends[k][1]);
  }
  // The workspace regions follow each other, and the cleared words cover the marks and totals.
  if (P.off_status + P.status_bytes > P.off_nz || P.off_nz + P.nz_bytes > P.off_ptotal ||
      P.off_ptotal + n_pairs * 4 > P.total ||
      (uint64_t)P.clear_words * 4 < P.off_ptotal + n_pairs * 4 - P.off_nz ||
      P.off_nz + (uint64_t)P.clear_words * 4 > P.total)
    return check_fail(msg, "workspace regions overlap or overflow");
  if (P.status_bytes != n_pairs * (uint64_t)P.tiles * 8)
    return check_fail(msg, "status words for %llu pairs x %lld tiles", (unsigned long long)n_pairs,
                      (long long)P.tiles);
  return true;
}

}  // namespace emr
