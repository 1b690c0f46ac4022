// argus_oracle.cpp -- CPU oracle for region attribution over marker traces.
//
// TEST INFRASTRUCTURE ONLY: used by tests, the smoke check and the
// benchmark's CPU-baseline leg.  Single-threaded, plain C++17, no blocking,
// fusion or reordering beyond what each definition below states.  It shares
// nothing with the GPU library.
//
// Every step cites the passage of the paper it follows.  Where the paper is
// silent, the reading adopted is written next to the step ("Reading: ...").
//
// All arithmetic is on unsigned 64-bit integers and wraps modulo 2^64.

#include "argus_oracle.h"

#include <algorithm>
#include <cstring>
#include <vector>

namespace {

const uint32_t kNone = 0xFFFFFFFFu;      // parent of a top-level instance
const uint16_t kNoEnd = 0xFFFF;          // end region of an unclosed instance
const uint64_t kNoTime = ~uint64_t(0);   // t_end of an unclosed instance

struct Record {
  uint64_t ts;
  uint32_t ctx;
  uint16_t region;
  uint8_t kind;
  uint8_t pad;
};
static_assert(sizeof(Record) == 16, "record is 16 bytes");

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

// Number of significant bits: 0 for 0, floor(log2 d) + 1 otherwise.
// Reading: the "log2 histogram" has 65 bins indexed by this value, so every
// u64 duration has exactly one bin and a zero-length region lands in bin 0.
unsigned bit_width(uint64_t d) {
  unsigned b = 0;
  while (d != 0) {
    ++b;
    d >>= 1;
  }
  return b;
}

// Sort key of a valid record: execution context, then timestamp, then the
// record's index in the input ("seq").
struct Key {
  uint32_t ctx;
  uint64_t ts;
  uint64_t seq;
};

}  // namespace

extern "C" int argus_oracle_run(const void* records_v, uint64_t n,
                                uint32_t num_regions, uint32_t num_classes,
                                const uint8_t* region_class,
                                uint32_t group_shift, uint32_t num_groups,
                                uint64_t* counters, uint64_t* region_stats,
                                uint64_t* overlap_group,
                                uint64_t* overlap_global, void* instances_v,
                                uint64_t* instance_excl, uint64_t inst_cap) {
  if (counters == nullptr || region_stats == nullptr) return -1;
  if (n > 0 && records_v == nullptr) return -1;
  if (num_regions < 1 || num_regions > 65535) return -1;
  if (num_classes > 8) return -1;
  if (num_classes > 0 && region_class == nullptr) return -1;
  if (group_shift > 32) return -1;

  const Record* rec = static_cast<const Record*>(records_v);
  const uint64_t R = num_regions;
  const uint64_t K = num_classes;

  std::memset(counters, 0, sizeof(uint64_t) * ORC_NUM_COUNTERS);
  for (uint64_t r = 0; r < R; ++r) {
    uint64_t* row = region_stats + r * ORC_RS_WIDTH;
    std::memset(row, 0, sizeof(uint64_t) * ORC_RS_WIDTH);
    // Reading: a region with no matched instance reports min = UINT64_MAX
    // and max = 0.
    row[ORC_RS_INCL_MIN] = kNoTime;
    row[ORC_RS_EXCL_MIN] = kNoTime;
  }

  // ---- Step 1: validate, in input order.  (Section 3.2: only begin(id)
  // and end(id) transitions of known regions carry region identity.)
  // Reading: kind 1 is BEGIN, kind 2 is END, anything else (0 = an unwritten
  // trace slot) is a bad kind; a region id >= R is a bad region; the pad
  // byte is ignored.  Invalid records take no part in any later step.
  uint64_t ts_min = kNoTime, ts_max = 0;
  uint64_t ctx_min = kNoTime, ctx_max = 0;
  std::vector<Key> keys;
  keys.reserve(n);
  for (uint64_t i = 0; i < n; ++i) {
    const Record& r = rec[i];
    if (r.kind != 1 && r.kind != 2) {
      counters[ORC_N_BAD_KIND] += 1;
      continue;
    }
    if (r.region >= num_regions) {
      counters[ORC_N_BAD_REGION] += 1;
      continue;
    }
    counters[ORC_N_VALID] += 1;
    if (r.kind == 1)
      counters[ORC_N_BEGIN] += 1;
    else
      counters[ORC_N_END] += 1;
    ts_min = std::min(ts_min, r.ts);
    ts_max = std::max(ts_max, r.ts);
    ctx_min = std::min<uint64_t>(ctx_min, r.ctx);
    ctx_max = std::max<uint64_t>(ctx_max, r.ctx);
    keys.push_back(Key{r.ctx, r.ts, i});
  }
  counters[ORC_N_RECORDS] = n;
  counters[ORC_TS_MIN] = ts_min;
  counters[ORC_TS_MAX] = ts_max;
  counters[ORC_CTX_MIN] = ctx_min;
  counters[ORC_CTX_MAX] = ctx_max;

  // ---- Step 2: order each execution context's records by time.
  // (Section 3.2: the region-context stack is kept per warp, i.e. per
  // execution context, and is updated in execution order.)
  // Reading: records with equal (ctx, ts) keep their input order, which is
  // what a stable sort on (ctx, ts) gives.
  std::stable_sort(keys.begin(), keys.end(), [](const Key& a, const Key& b) {
    if (a.ctx != b.ctx) return a.ctx < b.ctx;
    return a.ts < b.ts;
  });

  // ---- Step 3: per-context nested stack.  (Section 3.2: every warp keeps
  // its own stack of open regions; a BEGIN pushes one and an END closes the
  // one opened most recently.)
  // Readings: an END pops the top of the stack whatever its region
  // ("region-blind"); the pair is MATCHED if the regions agree and
  // MISMATCHED otherwise.  An END on an empty stack is an orphan and leaves
  // the stack alone.  A BEGIN still open when its context ends is UNCLOSED.
  // Instances are numbered by the position of their BEGIN in the sorted
  // order, so the numbering does not depend on the input order.
  std::vector<Instance> inst;
  inst.reserve(counters[ORC_N_BEGIN]);
  std::vector<uint32_t> stack;
  uint64_t n_ctx = 0;
  size_t i = 0;
  while (i < keys.size()) {
    const uint32_t ctx = keys[i].ctx;
    n_ctx += 1;
    stack.clear();
    for (; i < keys.size() && keys[i].ctx == ctx; ++i) {
      const Record& r = rec[keys[i].seq];
      if (r.kind == 1) {
        Instance x;
        x.t_begin = r.ts;
        x.t_end = kNoTime;
        x.ctx = ctx;
        x.parent = stack.empty() ? kNone : stack.back();
        x.level = static_cast<uint32_t>(stack.size());
        x.region = r.region;
        x.end_region = kNoEnd;
        stack.push_back(static_cast<uint32_t>(inst.size()));
        inst.push_back(x);
      } else if (stack.empty()) {
        counters[ORC_N_ORPHAN_END] += 1;
        region_stats[uint64_t(r.region) * ORC_RS_WIDTH + ORC_RS_ORPHAN_END] += 1;
      } else {
        const uint32_t id = stack.back();
        stack.pop_back();
        inst[id].t_end = r.ts;
        inst[id].end_region = r.region;
      }
    }
    // Whatever is left on the stack is unclosed (its t_end stays UINT64_MAX
    // and its end region stays 0xFFFF).
  }
  counters[ORC_N_CTX] = n_ctx;

  // Status of an instance, from its fields.
  auto is_closed = [&](const Instance& x) { return x.end_region != kNoEnd; };
  auto is_matched = [&](const Instance& x) {
    return x.end_region != kNoEnd && x.end_region == x.region;
  };

  // ---- Step 4: exclusive time.  (Section 3.2: the innermost active region
  // receives the work.)  Reading: a closed instance's exclusive duration is
  // its inclusive duration minus the inclusive durations of all its closed
  // direct children, matched or mismatched; an unclosed instance gets 0.
  std::vector<uint64_t> child_sum(inst.size(), 0);
  for (size_t id = 0; id < inst.size(); ++id) {
    const Instance& x = inst[id];
    if (is_closed(x) && x.parent != kNone)
      child_sum[x.parent] += x.t_end - x.t_begin;
  }
  std::vector<uint64_t> excl(inst.size(), 0);
  for (size_t id = 0; id < inst.size(); ++id) {
    const Instance& x = inst[id];
    if (is_closed(x)) excl[id] = (x.t_end - x.t_begin) - child_sum[id];
  }

  // ---- Step 5: per-region observed statistics and ambiguity counts.
  // (Section 3.5: duration is an observed field; the report exposes
  // attribution ambiguity.)  Reading: statistics are taken over MATCHED
  // instances only; unclosed, mismatched (by begin and by end region),
  // orphan and self-nested occurrences are counted per region.  A matched
  // instance is self-nested when its parent has the same region.
  uint64_t max_level = 0;
  for (size_t id = 0; id < inst.size(); ++id) {
    const Instance& x = inst[id];
    max_level = std::max<uint64_t>(max_level, x.level);
    uint64_t* row = region_stats + uint64_t(x.region) * ORC_RS_WIDTH;
    if (!is_closed(x)) {
      counters[ORC_N_UNCLOSED] += 1;
      row[ORC_RS_UNCLOSED] += 1;
      continue;
    }
    if (!is_matched(x)) {
      counters[ORC_N_MISMATCHED] += 1;
      row[ORC_RS_MISM_AS_BEGIN] += 1;
      region_stats[uint64_t(x.end_region) * ORC_RS_WIDTH +
                   ORC_RS_MISM_AS_END] += 1;
      continue;
    }
    counters[ORC_N_MATCHED] += 1;
    const uint64_t d = x.t_end - x.t_begin;
    const uint64_t e = excl[id];
    row[ORC_RS_COUNT] += 1;
    row[ORC_RS_INCL_SUM] += d;
    row[ORC_RS_EXCL_SUM] += e;
    row[ORC_RS_INCL_MIN] = std::min(row[ORC_RS_INCL_MIN], d);
    row[ORC_RS_INCL_MAX] = std::max(row[ORC_RS_INCL_MAX], d);
    row[ORC_RS_EXCL_MIN] = std::min(row[ORC_RS_EXCL_MIN], e);
    row[ORC_RS_EXCL_MAX] = std::max(row[ORC_RS_EXCL_MAX], e);
    row[ORC_RS_HIST_INCL + bit_width(d)] += 1;
    row[ORC_RS_HIST_EXCL + bit_width(e)] += 1;
    if (x.parent != kNone && inst[x.parent].region == x.region) {
      row[ORC_RS_SELF_NESTED] += 1;
      counters[ORC_N_SELF_NESTED] += 1;
    }
  }
  counters[ORC_MAX_LEVEL] = max_level;

  // ---- Step 6: overlap between region classes.  (Section 4.3: the
  // overlap of compute and communication regions is the quantity a client
  // optimises; Section 3.2: a scope such as an SM subset selects the
  // executions that count.)  Readings: a region's class is region_class[region]
  // (>= K: unclassified).  Only MATCHED, classified instances whose group
  // (ctx >> group_shift) is below G take part; those with a larger group
  // are counted as skipped.  Intervals are half-open [t_begin, t_end).  For
  // each group, U[A][B] is the time during which at least one class-A and
  // at least one class-B instance are active, and Q[A][B] is the sum over
  // pairs of one class-A and one distinct class-B instance of their
  // intersection length (for A == B each unordered pair counts once).  Both
  // are symmetric.  The global matrices are the sums over groups, because
  // per-SM cycle counters do not share a timebase.
  if (K > 0) {
    std::vector<std::vector<uint32_t>> by_group(num_groups);
    for (size_t id = 0; id < inst.size(); ++id) {
      const Instance& x = inst[id];
      if (!is_matched(x)) continue;
      const uint32_t c = region_class[x.region];
      if (c >= K) continue;
      const uint64_t g = (group_shift >= 32) ? 0 : (x.ctx >> group_shift);
      if (g >= num_groups) {
        counters[ORC_N_OVERLAP_SKIPPED] += 1;
        continue;
      }
      by_group[g].push_back(static_cast<uint32_t>(id));
    }
    const uint64_t KK = K * K;
    if (overlap_global) std::memset(overlap_global, 0, sizeof(uint64_t) * 2 * KK);
    struct Event {
      uint64_t t;
      int delta;
      uint32_t cls;
    };
    std::vector<Event> ev;
    for (uint64_t g = 0; g < num_groups; ++g) {
      std::vector<uint64_t> U(KK, 0), Q(KK, 0);
      ev.clear();
      for (uint32_t id : by_group[g]) {
        const Instance& x = inst[id];
        const uint32_t c = region_class[x.region];
        ev.push_back(Event{x.t_begin, +1, c});
        ev.push_back(Event{x.t_end, -1, c});
      }
      // Equal times give a zero gap, so the order among ties is irrelevant.
      std::sort(ev.begin(), ev.end(),
                [](const Event& a, const Event& b) { return a.t < b.t; });
      std::vector<int64_t> cnt(K, 0);
      for (size_t k = 0; k + 1 < ev.size(); ++k) {
        cnt[ev[k].cls] += ev[k].delta;
        const uint64_t gap = ev[k + 1].t - ev[k].t;
        // A zero gap adds nothing; skipping it also skips the transient
        // counts seen in the middle of a group of equal times.
        if (gap == 0) continue;
        for (uint64_t a = 0; a < K; ++a) {
          for (uint64_t b = a; b < K; ++b) {
            const uint64_t ca = static_cast<uint64_t>(cnt[a]);
            const uint64_t cb = static_cast<uint64_t>(cnt[b]);
            if (ca > 0 && cb > 0) U[a * K + b] += gap;
            if (a != b)
              Q[a * K + b] += gap * ca * cb;
            else if (ca > 1)
              Q[a * K + b] += gap * (ca * (ca - 1) / 2);
          }
        }
      }
      for (uint64_t a = 0; a < K; ++a)
        for (uint64_t b = 0; b < a; ++b) {
          U[a * K + b] = U[b * K + a];
          Q[a * K + b] = Q[b * K + a];
        }
      if (overlap_group) {
        uint64_t* out = overlap_group + g * 2 * KK;
        std::memcpy(out, U.data(), sizeof(uint64_t) * KK);
        std::memcpy(out + KK, Q.data(), sizeof(uint64_t) * KK);
      }
      if (overlap_global)
        for (uint64_t j = 0; j < KK; ++j) {
          overlap_global[j] += U[j];
          overlap_global[KK + j] += Q[j];
        }
    }
  }

  // ---- Instance outputs, in canonical (begin-rank) order.
  if (instances_v || instance_excl) {
    if (inst.size() > inst_cap) return -2;
    if (instances_v)
      std::memcpy(instances_v, inst.data(), sizeof(Instance) * inst.size());
    if (instance_excl)
      std::memcpy(instance_excl, excl.data(), sizeof(uint64_t) * excl.size());
  }
  return 0;
}
