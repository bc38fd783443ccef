// Longest-processing-time-first placement of a discover launch's chunks on its waves.
//
// A launch runs a fixed number of resident waves, each walking its share of the chunks (runs of
// consecutive tiles of one group of sources). Chunk costs differ by two orders of magnitude (the
// programs' lengths and activations differ), and with only a few chunks per wave, handing them out
// round-robin leaves some waves with several times the mean work: the launch lasts as long as its
// busiest wave. The host knows every chunk's cost from the cost model, so it places them once per
// plan and grid with the classical greedy rule, and the kernel reads each wave's list.
//
// The device's workgroups are spread over its XCDs round-robin, each XCD with its own L2. A
// group's chunks run the same program (machine code or records) over the same bias rows, so the
// placement first gives every group one XCD (a domain of waves), balanced by the groups' total
// cost, and then balances that XCD's chunks over its waves: each program is fetched into one L2.
#include "sched.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <queue>
#include <utility>

#include "emr_internal.h"

namespace emr {
namespace {

using Slot = std::pair<double, uint32_t>;  // (load, index): the least load, then the lowest index
// Domains are used only when no key holds more than this share of a domain's mean load.
constexpr double kMaxKeyShare = 0.1;
using MinHeap = std::priority_queue<Slot, std::vector<Slot>, std::greater<Slot>>;

// Chunks `order` (already in decreasing cost) onto the waves `ws`, appending to lists[w].
void place(const float* cost, const std::vector<uint32_t>& order, const std::vector<uint32_t>& ws,
           std::vector<std::vector<uint32_t>>* lists) {
  MinHeap heap;
  for (uint32_t i = 0; i < ws.size(); ++i) heap.push({0.0, i});
  for (uint32_t c : order) {
    Slot s = heap.top();
    heap.pop();
    (*lists)[ws[s.second]].push_back(c);
    s.first += (double)cost[c];
    heap.push(s);
  }
}

}  // namespace

bool lpt_schedule(const float* cost, const uint32_t* key, uint32_t n_keys, uint32_t n,
                  uint32_t waves, uint32_t domain_waves, uint32_t domains,
                  std::vector<uint32_t>* table, uint32_t* stride) {
  table->clear();
  *stride = 0;
  if (waves == 0 || (n > 0 && !cost)) return false;
  for (uint32_t c = 0; c < n; ++c)
    if (!std::isfinite(cost[c]) || cost[c] < 0.0f) return false;
  if (domains <= 1) domains = 1;
  if (domains > 1) {
    if (!key || domain_waves == 0 || (uint64_t)domain_waves * domains > waves) return false;
    for (uint32_t c = 0; c < n; ++c)
      if (key[c] >= n_keys) return false;
  }
  std::vector<uint32_t> order(n);
  for (uint32_t c = 0; c < n; ++c) order[c] = c;
  std::stable_sort(order.begin(), order.end(),
                   [&](uint32_t a, uint32_t b) { return cost[a] > cost[b]; });
  std::vector<std::vector<uint32_t>> lists(waves);
  if (domains == 1) {
    std::vector<uint32_t> all(waves);
    for (uint32_t w = 0; w < waves; ++w) all[w] = w;
    place(cost, order, all, &lists);
  } else {
    // the domains' waves
    std::vector<std::vector<uint32_t>> dw(domains);
    for (uint32_t w = 0; w < waves; ++w) dw[(w / domain_waves) % domains].push_back(w);
    // keys onto domains by total cost, per wave of the domain
    std::vector<double> total(n_keys, 0.0);
    for (uint32_t c = 0; c < n; ++c) total[key[c]] += (double)cost[c];
    std::vector<uint32_t> korder;
    for (uint32_t k = 0; k < n_keys; ++k)
      if (total[k] > 0.0) korder.push_back(k);
    std::stable_sort(korder.begin(), korder.end(),
                     [&](uint32_t a, uint32_t b) { return total[a] > total[b]; });
    // Keys too large to balance over the domains (a call with few groups) would leave domains
    // idle: then the chunks are placed over all waves as one domain.
    double sum = 0.0, biggest = 0.0;
    for (uint32_t k : korder) {
      sum += total[k];
      biggest = std::max(biggest, total[k]);
    }
    if (biggest > kMaxKeyShare * sum / domains)
      return lpt_schedule(cost, key, n_keys, n, waves, domain_waves, 1u, table, stride);
    std::vector<uint32_t> dom(n_keys, 0u);
    std::vector<double> load(domains, 0.0);
    for (uint32_t k : korder) {
      uint32_t best = 0;
      for (uint32_t d = 1; d < domains; ++d)
        if (load[d] / (double)dw[d].size() < load[best] / (double)dw[best].size()) best = d;
      dom[k] = best;
      load[best] += total[k];
    }
    // each domain's chunks (zero-cost keys stay in domain 0), in decreasing cost, onto its waves
    std::vector<std::vector<uint32_t>> dorder(domains);
    for (uint32_t c : order) dorder[dom[key[c]]].push_back(c);
    for (uint32_t d = 0; d < domains; ++d) place(cost, dorder[d], dw[d], &lists);
  }
  size_t most = 0;
  for (const auto& l : lists) most = std::max(most, l.size());
  const uint32_t st = (uint32_t)std::max<size_t>(kWave, (most + kWave - 1) / kWave * kWave);
  table->assign((size_t)waves * st, kNoChunk);
  for (uint32_t w = 0; w < waves; ++w)
    std::copy(lists[w].begin(), lists[w].end(), table->begin() + (size_t)w * st);
  *stride = st;
  return true;
}

}  // namespace emr

extern "C" int emr_lpt_schedule(const float* cost, const uint32_t* key, uint32_t n_keys,
                                uint32_t n, uint32_t waves, uint32_t domain_waves,
                                uint32_t domains, uint32_t* table, uint64_t table_cap,
                                uint32_t* stride) {
  std::vector<uint32_t> t;
  uint32_t st = 0;
  if (!stride ||
      !emr::lpt_schedule(cost, key, n_keys, n, waves, domain_waves, domains, &t, &st))
    return -1;
  *stride = st;
  if (!table || table_cap < t.size()) return 1;
  std::memcpy(table, t.data(), t.size() * sizeof(uint32_t));
  return 0;
}
