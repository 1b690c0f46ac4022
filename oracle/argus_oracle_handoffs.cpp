// argus_oracle_handoffs.cpp -- CPU oracle for the gaps between successive
// phases (sibling regions) of a context.
//
// TEST INFRASTRUCTURE ONLY, like argus_oracle.cpp: single-threaded, plain
// C++17, sharing nothing with the GPU library.
//
// Section 4.2 of the paper reports, from the reference trace of a persistent
// decode kernel, the time per step spent between successive cooperative
// phases, and Section 2 counts a phase handoff among the units a developer
// optimises.  Readings: the phases are the instances of one nesting level;
// two of them are successive when they have the same parent (the same
// context, for top-level phases) and no other child of that parent begins
// between them; the handoff is the time from the end of the first to the
// beginning of the second.  Statistics are kept per (from, to) region pair
// and per parent (the "per step" total when the parent is the step region).

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

unsigned bit_width(uint64_t d) {
  unsigned b = 0;
  while (d != 0) {
    ++b;
    d >>= 1;
  }
  return b;
}

}  // namespace

extern "C" int argus_oracle_handoffs(const void* instances_v, uint64_t n_inst,
                                     uint32_t num_regions, uint32_t level, uint64_t* pairs,
                                     uint64_t* hist, uint64_t* parent_gap, uint64_t* counters) {
  if (!pairs || !hist || !counters) return -1;
  if (num_regions < 1 || num_regions > 4096) return -1;
  if (n_inst > 0 && !instances_v) return -1;
  const Instance* inst = static_cast<const Instance*>(instances_v);
  const uint64_t R = num_regions;
  std::memset(counters, 0, sizeof(uint64_t) * ORC_PH_NUM_COUNTERS);
  std::memset(hist, 0, sizeof(uint64_t) * 65);
  for (uint64_t i = 0; i < R * R; ++i) {
    pairs[4 * i + 0] = 0;
    pairs[4 * i + 1] = 0;
    pairs[4 * i + 2] = ~uint64_t(0);
    pairs[4 * i + 3] = 0;
  }
  if (parent_gap) std::memset(parent_gap, 0, sizeof(uint64_t) * n_inst);

  // The previous level-L child of each (context, parent); a top-level
  // instance's parent is "none" within its context.
  std::map<std::pair<uint32_t, uint32_t>, uint64_t> last;
  for (uint64_t y = 0; y < n_inst; ++y) {
    const Instance& b = inst[y];
    if (b.level != level) continue;
    counters[ORC_PH_N_AT_LEVEL] += 1;
    const std::pair<uint32_t, uint32_t> key{b.ctx, b.parent};
    auto it = last.find(key);
    if (it != last.end()) {
      const Instance& a = inst[it->second];
      // (a phase that never ends has no successor: everything after it in
      // its context is nested inside it)
      if (a.end_region != kNoEnd && a.region < R && b.region < R) {
        const uint64_t gap = b.t_begin - a.t_end;
        uint64_t* row = pairs + 4 * (uint64_t(a.region) * R + b.region);
        row[0] += 1;
        row[1] += gap;
        row[2] = std::min(row[2], gap);
        row[3] = std::max(row[3], gap);
        hist[bit_width(gap)] += 1;
        counters[ORC_PH_N_GAPS] += 1;
        counters[ORC_PH_GAP_SUM] += gap;
        if (parent_gap && b.parent != 0xFFFFFFFFu && b.parent < n_inst) parent_gap[b.parent] += gap;
      }
    }
    last[key] = y;
  }
  return 0;
}
