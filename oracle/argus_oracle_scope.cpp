// argus_oracle_scope.cpp -- CPU oracle for iteration ordinals and scoped
// per-region statistics.
//
// TEST INFRASTRUCTURE ONLY, like argus_oracle.cpp: single-threaded, plain
// C++17, sharing nothing with the GPU library.
//
// Section 3.2 of the paper separates a region (the code) from its scope
// (which dynamic executions are reported: a warp role, an iteration window
// or a subset of SMs); Section 3.3 specialises probes to one iteration of a
// loop region.  Readings:
//   * The iteration of an instance is its 0-based ordinal among the
//     instances of the same context with the same BEGIN region, counted in
//     canonical order (every status counts: a malformed occurrence still
//     took an iteration).
//   * A warp role is a range of (ctx_key & role_mask); an SM subset is a
//     range of groups (ctx_key >> group_shift); an iteration window is a
//     range of ordinals; optionally a set of regions.
//   * Scoped statistics are the observed per-region statistics over the
//     in-scope instances (Section 3.5), in the same layout as the unscoped
//     ones.

#include "argus_oracle.h"

#include <algorithm>
#include <cstring>
#include <map>
#include <utility>

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

const uint16_t kNoEnd = 0xFFFF;
const uint32_t kNone = 0xFFFFFFFFu;

unsigned bit_width(uint64_t d) {
  unsigned b = 0;
  while (d != 0) {
    ++b;
    d >>= 1;
  }
  return b;
}

bool in_range(uint64_t v, uint64_t lo, uint64_t hi) { return lo <= v && v <= hi; }

}  // namespace

extern "C" int argus_oracle_scope(const void* instances_v, const uint64_t* excl, uint64_t n_inst,
                                  uint32_t num_regions, const orc_scope* sc,
                                  const uint8_t* region_mask, uint32_t* ordinal,
                                  uint64_t* stats, uint64_t* counters) {
  if (!sc || !ordinal || !stats || !counters) return -1;
  if (num_regions < 1 || num_regions > 65535) return -1;
  if (n_inst > 0 && (!instances_v || !excl)) return -1;
  const Instance* inst = static_cast<const Instance*>(instances_v);
  const uint64_t R = num_regions;

  std::memset(counters, 0, sizeof(uint64_t) * ORC_SC_NUM_COUNTERS);
  for (uint64_t r = 0; r < R; ++r) {
    uint64_t* row = stats + r * ORC_RS_WIDTH;
    std::memset(row, 0, sizeof(uint64_t) * ORC_RS_WIDTH);
    row[ORC_RS_INCL_MIN] = ~uint64_t(0);
    row[ORC_RS_EXCL_MIN] = ~uint64_t(0);
  }

  // Ordinals: a counter per (context, region), in canonical order.
  std::map<std::pair<uint32_t, uint16_t>, uint32_t> seen;
  uint64_t iterations = 0;
  for (uint64_t x = 0; x < n_inst; ++x) {
    uint32_t& c = seen[{inst[x].ctx, inst[x].region}];
    ordinal[x] = c;
    c += 1;
    iterations = std::max<uint64_t>(iterations, uint64_t(ordinal[x]) + 1);
  }
  counters[ORC_SC_N_INSTANCES] = n_inst;
  counters[ORC_SC_N_ITERATIONS] = iterations;

  for (uint64_t x = 0; x < n_inst; ++x) {
    const Instance& a = inst[x];
    const uint64_t group = sc->group_shift >= 32 ? 0 : (a.ctx >> sc->group_shift);
    const bool in = in_range(a.ctx & sc->role_mask, sc->role_lo, sc->role_hi) &&
                    in_range(group, sc->group_lo, sc->group_hi) &&
                    in_range(ordinal[x], sc->iter_lo, sc->iter_hi) &&
                    a.region < num_regions && (!region_mask || region_mask[a.region] != 0);
    if (!in) continue;
    counters[ORC_SC_N_IN_SCOPE] += 1;
    uint64_t* row = stats + uint64_t(a.region) * ORC_RS_WIDTH;
    if (a.end_region == kNoEnd) {
      counters[ORC_SC_N_UNCLOSED] += 1;
      row[ORC_RS_UNCLOSED] += 1;
      continue;
    }
    if (a.end_region != a.region) {
      counters[ORC_SC_N_MISMATCHED] += 1;
      row[ORC_RS_MISM_AS_BEGIN] += 1;
      if (a.end_region < num_regions)
        stats[uint64_t(a.end_region) * ORC_RS_WIDTH + ORC_RS_MISM_AS_END] += 1;
      continue;
    }
    counters[ORC_SC_N_MATCHED] += 1;
    const uint64_t d = a.t_end - a.t_begin;
    const uint64_t e = excl[x];
    row[ORC_RS_COUNT] += 1;
    row[ORC_RS_INCL_SUM] += d;
    row[ORC_RS_EXCL_SUM] += e;
    row[ORC_RS_INCL_MIN] = std::min(row[ORC_RS_INCL_MIN], d);
    row[ORC_RS_INCL_MAX] = std::max(row[ORC_RS_INCL_MAX], d);
    row[ORC_RS_EXCL_MIN] = std::min(row[ORC_RS_EXCL_MIN], e);
    row[ORC_RS_EXCL_MAX] = std::max(row[ORC_RS_EXCL_MAX], e);
    row[ORC_RS_HIST_INCL + bit_width(d)] += 1;
    row[ORC_RS_HIST_EXCL + bit_width(e)] += 1;
    if (a.parent != kNone && a.parent < n_inst && inst[a.parent].region == a.region) {
      row[ORC_RS_SELF_NESTED] += 1;
      counters[ORC_SC_N_SELF_NESTED] += 1;
    }
  }
  return 0;
}
