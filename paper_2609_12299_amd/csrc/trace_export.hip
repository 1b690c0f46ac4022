// trace_export.hip -- Chrome Trace Viewer export of region instances and
// probe summaries (host code).
//
// Appendix B of the paper shows the synthesised asynchronous timeline in
// Chrome Trace Viewer with lanes per warp: the reference trace of the warp
// (its region instances), then, for each kind of asynchronous operation, a
// lane with the mean exposed latency drawn from the operation's issue in
// the reference trace and a lane with its percentile bands (0th, 20th,
// 40th, 60th and 80th percentile, each a slice from the issue, the longer
// ones enclosing the shorter).  Here one process is one group of contexts
// (ctx_key >> group_shift, an SM or a block) and its threads are the lanes
// of its contexts: one lane per nesting level of the reference instances
// (deeper levels share the last one), then a mean lane and a percentile
// lane for every operation region that has probe groups in that context.
#include <stdio.h>
#include <string.h>

#include <map>
#include <string>
#include <utility>
#include <vector>

#include "internal.h"

namespace {

constexpr uint32_t kRefLanes = 8;        // reference lanes per context (levels >= 7 share the last)
constexpr uint32_t kLanesPerCtx = 1024;  // lane ids of one context: [ctx_local * 1024, + 1024)

std::string json_escape(const char* s) {
  std::string o;
  for (; *s; ++s) {
    const unsigned char c = (unsigned char)*s;
    if (c == '"' || c == '\\') {
      o += '\\';
      o += (char)c;
    } else if (c < 0x20) {
      char b[8];
      snprintf(b, sizeof b, "\\u%04x", c);
      o += b;
    } else {
      o += (char)c;
    }
  }
  return o;
}

struct Writer {
  FILE* f;
  bool first = true;
  bool ok = true;
  void event(const char* body) {
    if (fprintf(f, "%s\n%s", first ? "" : ",", body) < 0) ok = false;
    first = false;
  }
};

}  // namespace

extern "C" int argus_attr_chrome_trace(const argus_instance* h_instances, uint64_t n_instances,
                                       const uint64_t* h_groups, const double* h_mean,
                                       uint64_t n_groups, const argus_trace_options* opt,
                                       const char* path) {
  if (!opt || !path || (n_instances > 0 && !h_instances)) return ARGUS_E_INVAL;
  if (n_groups > 0 && (!h_groups || !h_mean)) return ARGUS_E_INVAL;
  if (!(opt->cycles_per_us > 0.0) || opt->group_shift > 32 || opt->num_regions < 1 ||
      opt->num_regions > 65535)
    return ARGUS_E_INVAL;
  for (uint64_t g = 0; g < n_groups; ++g)
    if (h_groups[g * ARGUS_PG_WIDTH + ARGUS_PG_INSTANCE] >= n_instances) return ARGUS_E_INVAL;
  FILE* f = fopen(path, "w");
  if (!f) return ARGUS_E_IO;

  const double k = 1.0 / opt->cycles_per_us;
  const uint32_t shift = opt->group_shift;
  auto pid_of = [&](uint32_t ctx) -> uint64_t { return shift >= 32 ? 0 : (ctx >> shift); };
  auto local_of = [&](uint32_t ctx) -> uint64_t {
    return shift >= 32 ? ctx : (ctx & (shift ? ((1u << shift) - 1u) : 0u));
  };
  auto name_of = [&](uint32_t r) -> std::string {
    if (opt->region_names && r < opt->num_regions && opt->region_names[r])
      return json_escape(opt->region_names[r]);
    return "r" + std::to_string(r);
  };
  const bool unmatched = (opt->flags & ARGUS_TRACE_UNMATCHED) != 0;

  Writer w{f};
  if (fprintf(f, "{\"displayTimeUnit\": \"ns\", \"traceEvents\": [") < 0) w.ok = false;
  std::string buf;
  char num[160];
  // lanes that carry events: (pid, tid) -> name
  std::map<std::pair<uint64_t, uint64_t>, std::string> lanes;

  for (uint64_t x = 0; x < n_instances && w.ok; ++x) {
    const argus_instance& a = h_instances[x];
    const bool closed = a.end_region_id != ARGUS_UNCLOSED;
    const bool matched = closed && a.end_region_id == a.region_id;
    if (!closed || (!matched && !unmatched)) continue;
    const uint32_t lane = a.level < kRefLanes ? a.level : kRefLanes - 1;
    const uint64_t pid = pid_of(a.ctx_key), tid = local_of(a.ctx_key) * kLanesPerCtx + lane;
    lanes.emplace(std::make_pair(pid, tid), "ctx " + std::to_string(a.ctx_key) + " reference L" +
                                                std::to_string(lane));
    buf = "{\"ph\": \"X\", \"cat\": \"reference\", \"name\": \"";
    buf += name_of(a.region_id);
    if (!matched) buf += " / " + name_of(a.end_region_id) + " (mismatched)";
    snprintf(num, sizeof num, "\", \"pid\": %llu, \"tid\": %llu, \"ts\": %.4f, \"dur\": %.4f",
             (unsigned long long)pid, (unsigned long long)tid, (double)a.t_begin * k,
             (double)(a.t_end - a.t_begin) * k);
    buf += num;
    snprintf(num, sizeof num, ", \"args\": {\"instance\": %llu, \"level\": %u, \"cycles\": %llu}}",
             (unsigned long long)x, a.level, (unsigned long long)(a.t_end - a.t_begin));
    buf += num;
    w.event(buf.c_str());
  }

  // Probe summaries: per context, one lane pair per operation region.
  std::map<std::pair<uint32_t, uint32_t>, uint32_t> op_lane;  // (ctx, region) -> index
  std::map<uint32_t, uint32_t> ops_in_ctx;
  static const char* kBand[5] = {"p0", "p20", "p40", "p60", "p80"};
  static const char* kColor[5] = {"rail_response", "thread_state_runnable", "yellow",
                                  "rail_load", "terrible"};
  for (uint64_t g = 0; g < n_groups && w.ok; ++g) {
    const uint64_t* row = h_groups + g * ARGUS_PG_WIDTH;
    const argus_instance& a = h_instances[row[ARGUS_PG_INSTANCE]];
    auto key = std::make_pair(a.ctx_key, (uint32_t)a.region_id);
    auto it = op_lane.find(key);
    if (it == op_lane.end()) it = op_lane.emplace(key, ops_in_ctx[a.ctx_key]++).first;
    const uint64_t pid = pid_of(a.ctx_key);
    const uint64_t base = local_of(a.ctx_key) * kLanesPerCtx + kRefLanes + 2ull * it->second;
    const std::string op = name_of(a.region_id);
    lanes.emplace(std::make_pair(pid, base), "ctx " + std::to_string(a.ctx_key) + " " + op +
                                                 " mean exposed latency");
    lanes.emplace(std::make_pair(pid, base + 1), "ctx " + std::to_string(a.ctx_key) + " " + op +
                                                     " percentiles");
    const double issue = (double)row[ARGUS_PG_ISSUE] * k;
    buf = "{\"ph\": \"X\", \"cat\": \"mean\", \"name\": \"" + op + " mean";
    snprintf(num, sizeof num, "\", \"pid\": %llu, \"tid\": %llu, \"ts\": %.4f, \"dur\": %.4f",
             (unsigned long long)pid, (unsigned long long)base, issue, h_mean[g] * k);
    buf += num;
    snprintf(num, sizeof num,
             ", \"args\": {\"instance\": %llu, \"probes\": %llu, \"mean_cycles\": %.3f}}",
             (unsigned long long)row[ARGUS_PG_INSTANCE], (unsigned long long)row[ARGUS_PG_COUNT],
             h_mean[g]);
    buf += num;
    w.event(buf.c_str());
    // the longest band first, so that each later one nests inside it
    for (int b = 4; b >= 0 && w.ok; --b) {
      const uint64_t v = row[ARGUS_PG_P0 + b];
      buf = std::string("{\"ph\": \"X\", \"cat\": \"percentile\", \"name\": \"") + op + " " +
            kBand[b] + "\", \"cname\": \"" + kColor[b];
      snprintf(num, sizeof num, "\", \"pid\": %llu, \"tid\": %llu, \"ts\": %.4f, \"dur\": %.4f",
               (unsigned long long)pid, (unsigned long long)(base + 1), issue, (double)v * k);
      buf += num;
      snprintf(num, sizeof num, ", \"args\": {\"instance\": %llu, \"cycles\": %llu}}",
               (unsigned long long)row[ARGUS_PG_INSTANCE], (unsigned long long)v);
      buf += num;
      w.event(buf.c_str());
    }
  }

  // Lane names and their order (metadata events).
  for (const auto& kv : lanes) {
    if (!w.ok) break;
    buf = "{\"ph\": \"M\", \"name\": \"thread_name\"";
    snprintf(num, sizeof num, ", \"pid\": %llu, \"tid\": %llu", (unsigned long long)kv.first.first,
             (unsigned long long)kv.first.second);
    buf += num;
    buf += ", \"args\": {\"name\": \"" + kv.second + "\"}}";
    w.event(buf.c_str());
    buf = "{\"ph\": \"M\", \"name\": \"thread_sort_index\"";
    snprintf(num, sizeof num, ", \"pid\": %llu, \"tid\": %llu, \"args\": {\"sort_index\": %llu}}",
             (unsigned long long)kv.first.first, (unsigned long long)kv.first.second,
             (unsigned long long)kv.first.second);
    buf += num;
    w.event(buf.c_str());
  }
  if (fprintf(f, "\n]}\n") < 0) w.ok = false;
  if (fclose(f) != 0) w.ok = false;
  return w.ok ? ARGUS_OK : ARGUS_E_IO;
}
