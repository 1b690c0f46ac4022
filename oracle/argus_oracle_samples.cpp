// argus_oracle_samples.cpp -- CPU oracle for attributing PC samples to
// region instances and lifting PC-keyed metrics into regions.
//
// TEST INFRASTRUCTURE ONLY, like argus_oracle.cpp: single-threaded, plain
// C++17, sharing nothing with the GPU library.
//
// Section 3.2 of the paper: a separate mapping run replays each warp's
// region transitions as a stack of open regions, and every execution of
// the instruction at PC p is counted for the region that is innermost at
// that moment; so n(r, p) is the number of executions of p under region r.
// Section 3.5: alpha(r, p) = n(r, p) / sum over regions r' of n(r', p);
// m_hat(r) = sum over p of alpha(r, p) m(p) for an additive PC-keyed metric
// m; H(p) = - sum over r of alpha(r, p) log alpha(r, p), the association
// entropy, reported as metadata about shared ownership.
//
// Readings (the paper states the rule for well-formed traces only):
//   * An instance x is active at time t when t_begin <= t < t_end (half-open
//     as for durations; an unclosed instance stays active from t_begin on).
//     The active instances of one context form a chain; the innermost is
//     the one at the deepest level.
//   * A sample is given to the innermost active instance whose BEGIN and END
//     regions agree (MATCHED): a mismatched or unclosed instance has no
//     single region.  When the innermost active instance is not matched but
//     an enclosing matched one is, the weight still goes to the matched one
//     and is counted as "inner unmatched" (ambiguity exposed).  With no
//     matched active instance the weight is unattributed.
//   * Floating point: IEEE double, each alpha by one division
//     n(r, p) / T(p); each product alpha(r, p) * m(p) rounded before it is
//     added, over the p with n(r, p) > 0.  The paper fixes no order for the
//     sum over p; m_hat(r) takes it in 512 strands: strand j adds, from +0
//     and in increasing p, the products with p mod 512 = j; then the strands
//     are combined by halving, strand j += strand j + h for j < h, with
//     h = 256, 128, ..., 1, and m_hat(r) is strand 0.  H(p) adds
//     alpha log alpha in increasing r.

#include "argus_oracle.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <set>
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

struct Sample {
  uint64_t ts;
  uint32_t ctx;
  uint32_t pc;
};
static_assert(sizeof(Sample) == 16, "sample is 16 bytes");

const uint16_t kNoEnd = 0xFFFF;

bool is_matched(const Instance& x) { return x.end_region != kNoEnd && x.end_region == x.region; }

}  // namespace

extern "C" int argus_oracle_samples(const void* instances_v, uint64_t n_inst,
                                    const void* samples_v, uint64_t n_samples,
                                    const uint32_t* weights, uint32_t num_regions,
                                    uint32_t num_pcs, uint32_t num_metrics,
                                    const double* metrics, uint64_t* counters,
                                    uint64_t* n_rp, double* alpha, uint64_t* pc_total,
                                    uint32_t* pc_owners, double* entropy,
                                    uint64_t* region_total, double* mhat) {
  if (!counters || !n_rp || !pc_total || !pc_owners || !entropy || !region_total) return -1;
  if (num_regions < 1 || num_regions > 65535 || num_pcs < 1) return -1;
  if (num_metrics > 0 && (!metrics || !mhat)) return -1;
  if (n_inst > 0 && !instances_v) return -1;
  if (n_samples > 0 && !samples_v) return -1;
  const Instance* inst = static_cast<const Instance*>(instances_v);
  const Sample* smp = static_cast<const Sample*>(samples_v);
  const uint64_t R = num_regions, P = num_pcs, M = num_metrics;

  std::memset(counters, 0, sizeof(uint64_t) * ORC_S_NUM_COUNTERS);
  std::memset(n_rp, 0, sizeof(uint64_t) * P * R);

  // Samples of each context, in time order (ties: input order).
  std::map<uint32_t, std::vector<uint64_t>> by_ctx;
  for (uint64_t i = 0; i < n_samples; ++i) {
    counters[ORC_S_N_SAMPLES] += 1;
    if (smp[i].pc >= num_pcs) {
      counters[ORC_S_N_BAD_PC] += 1;
      continue;
    }
    by_ctx[smp[i].ctx].push_back(i);
  }
  // Instances of each context (canonical order is by context, then begin).
  std::map<uint32_t, std::vector<uint32_t>> inst_of;
  for (uint64_t x = 0; x < n_inst; ++x) inst_of[inst[x].ctx].push_back(static_cast<uint32_t>(x));

  for (auto& kv : by_ctx) {
    std::vector<uint64_t>& ids = kv.second;
    std::stable_sort(ids.begin(), ids.end(),
                     [&](uint64_t a, uint64_t b) { return smp[a].ts < smp[b].ts; });
    // The context's instances by begin time and, for the closed ones, by end
    // time; `active` holds (level, id) of the instances begun and not ended.
    std::vector<std::pair<uint64_t, uint32_t>> begins, ends;
    auto it = inst_of.find(kv.first);
    if (it != inst_of.end())
      for (uint32_t x : it->second) {
        begins.push_back({inst[x].t_begin, x});
        if (inst[x].end_region != kNoEnd) ends.push_back({inst[x].t_end, x});
      }
    std::sort(begins.begin(), begins.end());
    std::sort(ends.begin(), ends.end());
    std::set<std::pair<uint32_t, uint32_t>> active;
    size_t bi = 0, ei = 0;
    for (uint64_t i : ids) {
      const uint64_t t = smp[i].ts;
      // Every instance with t_begin <= t enters, then every one with
      // t_end <= t leaves: what remains has t_begin <= t < t_end.
      for (; bi < begins.size() && begins[bi].first <= t; ++bi)
        active.insert({inst[begins[bi].second].level, begins[bi].second});
      for (; ei < ends.size() && ends[ei].first <= t; ++ei)
        active.erase({inst[ends[ei].second].level, ends[ei].second});
      const uint64_t w = weights ? weights[i] : 1;
      counters[ORC_S_W_TOTAL] += w;
      // Innermost matched instance: walk the chain from the deepest level.
      bool inner_unmatched = false;
      int64_t owner = -1;
      for (auto a = active.rbegin(); a != active.rend(); ++a) {
        if (is_matched(inst[a->second])) {
          owner = a->second;
          break;
        }
        inner_unmatched = true;
      }
      if (owner < 0) {
        counters[ORC_S_W_UNATTRIBUTED] += w;
        continue;
      }
      counters[ORC_S_W_ATTRIBUTED] += w;
      if (inner_unmatched) counters[ORC_S_W_INNER_UNMATCHED] += w;
      n_rp[uint64_t(smp[i].pc) * R + inst[owner].region] += w;
    }
  }

  // Per PC: total count, owners, alpha and entropy (Section 3.5).
  for (uint64_t p = 0; p < P; ++p) {
    const uint64_t* row = n_rp + p * R;
    uint64_t T = 0;
    uint32_t owners = 0;
    for (uint64_t r = 0; r < R; ++r) {
      T += row[r];
      if (row[r] > 0) owners += 1;
    }
    pc_total[p] = T;
    pc_owners[p] = owners;
    counters[ORC_S_N_PAIRS] += owners;
    double h = 0.0;
    for (uint64_t r = 0; r < R; ++r) {
      const double a = row[r] > 0 ? double(row[r]) / double(T) : 0.0;
      if (alpha) alpha[p * R + r] = a;
      if (row[r] > 0) h -= a * std::log(a);
    }
    entropy[p] = h;
  }
  // Per region: total count and the lifted metrics, summed in the strand
  // order stated at the top of this file.
  const uint64_t kStrands = 512;
  std::vector<double> strand(kStrands);
  for (uint64_t r = 0; r < R; ++r) {
    uint64_t tot = 0;
    for (uint64_t p = 0; p < P; ++p) tot += n_rp[p * R + r];
    region_total[r] = tot;
    for (uint64_t k = 0; k < M; ++k) {
      std::fill(strand.begin(), strand.end(), 0.0);
      for (uint64_t p = 0; p < P; ++p) {
        const uint64_t n = n_rp[p * R + r];
        if (n == 0) continue;
        const double a = double(n) / double(pc_total[p]);
        const double term = a * metrics[k * P + p];
        strand[p % kStrands] = strand[p % kStrands] + term;
      }
      for (uint64_t h = kStrands / 2; h >= 1; h /= 2)
        for (uint64_t j = 0; j < h; ++j) strand[j] = strand[j] + strand[j + h];
      mhat[k * R + r] = strand[0];
    }
  }
  return 0;
}
