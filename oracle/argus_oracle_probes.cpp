// argus_oracle_probes.cpp -- CPU oracle for joining forced-completion probe
// intervals to the reference trace and summarising their exposed latency.
//
// TEST INFRASTRUCTURE ONLY, like argus_oracle.cpp: single-threaded, plain
// C++17, sharing nothing with the GPU library.
//
// Section 3.3 of the paper: a probe forces one asynchronous operation of one
// selected iteration to complete right after it is issued and records that
// interval (the exposed latency); only this interval is kept, and it is
// joined to the same operation's issue in the same iteration of the
// reference trace through the operation's stable id and the dynamic scope,
// not by comparing timestamps across runs (Section 3.5).  Appendix B shows
// the mean and the 0th/20th/40th/60th/80th percentiles per operation and
// iteration.  Readings:
//   * The reference issue event of (context, operation, iteration i) is the
//     reference instance of that context whose BEGIN region is the
//     operation's region and whose iteration ordinal is i.
//   * Percentiles are nearest-rank: the k-th smallest latency with
//     k = max(1, ceil(q n / 100)), so p0 is the minimum and p100 the
//     maximum; they are integers.  The mean is the exact sum divided once.

#include "argus_oracle.h"

#include <algorithm>
#include <cstring>
#include <map>
#include <utility>
#include <vector>

namespace {

struct Instance {
  uint64_t t_begin;
  uint64_t t_end;
  uint32_t ctx;
  uint32_t parent;
  uint32_t level;
  uint16_t region;
  uint16_t end_region;
};
static_assert(sizeof(Instance) == 32, "instance is 32 bytes");

struct Probe {
  uint64_t t_start;
  uint64_t t_end;
  uint32_t ctx;
  uint32_t iteration;
  uint16_t op_region;
  uint16_t pad0;
  uint32_t pad1;
};
static_assert(sizeof(Probe) == 32, "probe is 32 bytes");

const uint32_t kNone = 0xFFFFFFFFu;

}  // namespace

extern "C" int argus_oracle_probes(const void* instances_v, uint64_t n_inst,
                                   uint32_t num_regions, const void* probes_v,
                                   uint64_t n_probes, uint32_t* ref, uint64_t* completion,
                                   uint64_t* groups, double* mean, uint64_t group_cap,
                                   uint64_t* counters) {
  if (!counters || (n_probes > 0 && (!probes_v || !ref || !completion))) return -1;
  if (num_regions < 1 || num_regions > 65535) return -1;
  if (n_inst > 0 && !instances_v) return -1;
  const Instance* inst = static_cast<const Instance*>(instances_v);
  const Probe* pr = static_cast<const Probe*>(probes_v);
  std::memset(counters, 0, sizeof(uint64_t) * ORC_PR_NUM_COUNTERS);

  // The reference instances of each (context, region), in canonical order:
  // the i-th of them is iteration i.
  std::map<std::pair<uint32_t, uint16_t>, std::vector<uint32_t>> by_key;
  for (uint64_t x = 0; x < n_inst; ++x)
    by_key[{inst[x].ctx, inst[x].region}].push_back(static_cast<uint32_t>(x));

  std::map<uint32_t, std::vector<uint64_t>> lat_of;  // instance -> latencies
  for (uint64_t j = 0; j < n_probes; ++j) {
    counters[ORC_PR_N_PROBES] += 1;
    ref[j] = kNone;
    completion[j] = ~uint64_t(0);
    const Probe& p = pr[j];
    if (p.t_end < p.t_start || p.op_region >= num_regions) {
      counters[ORC_PR_N_BAD] += 1;
      continue;
    }
    auto it = by_key.find({p.ctx, p.op_region});
    if (it == by_key.end() || p.iteration >= it->second.size()) {
      counters[ORC_PR_N_UNJOINED] += 1;
      continue;
    }
    const uint32_t x = it->second[p.iteration];
    const uint64_t lat = p.t_end - p.t_start;
    counters[ORC_PR_N_JOINED] += 1;
    ref[j] = x;
    completion[j] = inst[x].t_begin + lat;
    lat_of[x].push_back(lat);
  }

  uint64_t g = 0;
  for (auto& kv : lat_of) {
    if (g >= group_cap) return -2;
    std::vector<uint64_t>& v = kv.second;
    std::sort(v.begin(), v.end());
    const uint64_t n = v.size();
    uint64_t sum = 0;
    for (uint64_t x : v) sum += x;
    uint64_t* row = groups + g * ORC_PG_WIDTH;
    row[ORC_PG_INSTANCE] = kv.first;
    row[ORC_PG_COUNT] = n;
    row[ORC_PG_SUM] = sum;
    row[ORC_PG_ISSUE] = inst[kv.first].t_begin;
    const int q[6] = {0, 20, 40, 60, 80, 100};
    for (int k = 0; k < 6; ++k) {
      uint64_t rank = (uint64_t(q[k]) * n + 99) / 100;  // ceil(q n / 100)
      if (rank < 1) rank = 1;
      row[ORC_PG_P0 + k] = v[rank - 1];
    }
    mean[g] = double(sum) / double(n);
    g += 1;
  }
  counters[ORC_PR_N_GROUPS] = g;
  return 0;
}
