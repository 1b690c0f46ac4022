// attr_host.hip -- the C ABI: handle, argument checks, workspace layout and
// the launch sequence of one run.  Every argument check happens before the
// first HIP call, so error paths can be exercised without a GPU.
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

using namespace argus;

struct argus_attr {
  argus_attr_config cfg;
  std::string err;
  int device_checked = -1;  // device ordinal verified to be gfx950
  bool timing = false;
  std::string filter;  // time only the launches of this step ("": all)
  // Timing: for every timed run, a start event and one event per launch, or
  // (filter set) an event before and one after each matching launch.
  struct TimedRun {
    std::vector<hipEvent_t> ev;
    std::vector<const char*> names;
    bool pairs = false;
  };
  std::vector<TimedRun> runs;
  std::vector<hipEvent_t> pool;  // recycled events
};

namespace argus {

uint64_t persistent_blocks(const void* kernel, int threads) {
  int dev = 0, cus = 256, per_cu = 1;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  return (uint64_t)cus * (uint64_t)per_cu;
}

}  // namespace argus

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) & ~(kAlign - 1); }

// Workspace layout for n records.  Offsets only; the base is added in run.
struct Layout {
  size_t plan, rec_hist, rec_off, ev_hist, ev_off, tile_ctr;
  size_t key[2], pay[2], ctxw[2], lb[2], tsum, carry, bsum, slb, mslb, tiles, tree;
  size_t chunk_runs, run_base, run_cnt, run_pos, run_hist, scan_bsum;
  size_t pop_ts, pop_reg, pushes, op_parent, op_sum;
  size_t inst, excl, hist_key, agg_part, ov_mask, ov_q;
  size_t push_pos, pop_pos, ctx_list, seg_run, seg_tile0, seg_samp0, part;
  size_t total;
  uint64_t lb_words, tree_leaves, match_tiles, pool_cap, ctx_cap, tiles_cap, chunks, run_cap;
};

Layout make_layout(const argus_attr_config& c, uint64_t n, bool own_instances) {
  Layout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + (bytes ? bytes : 1));
    return at;
  };
  const uint64_t nn = n ? n : 1;
  L.plan = take(sizeof(DevPlan));
  L.rec_hist = take(sizeof(uint32_t) * kDigitPositions * kRadixBins);
  L.rec_off = take(sizeof(uint32_t) * kDigitPositions * kRadixBins);
  L.ev_hist = take(sizeof(uint32_t) * kDigitPositions * kRadixBins);
  L.ev_off = take(sizeof(uint32_t) * kDigitPositions * kRadixBins);
  L.tile_ctr = take(sizeof(uint32_t) * kCtrCount);
  for (int b = 0; b < 2; ++b) {
    // key[1] first holds the chunks' run lists: 256 places per chunk
    L.key[b] = take(sizeof(uint64_t) * ceil_div(nn, kChunk) * kChunk);
    L.pay[b] = take(sizeof(uint32_t) * nn);
    L.ctxw[b] = take(sizeof(uint32_t) * nn);
  }
  // The first event pass reads 2 * n_begin <= 2 * n slots.
  L.lb_words = ceil_div(2 * nn, kSortTile) * kRadixBins;
  for (int b = 0; b < 2; ++b) L.lb[b] = take(sizeof(uint64_t) * L.lb_words);
  L.match_tiles = ceil_div(nn, kMatchTile);
  L.tsum = take(sizeof(uint64_t) * L.match_tiles);
  L.carry = take(sizeof(TileCarry) * L.match_tiles);
  L.bsum = take(sizeof(BlockSum) * kMaxScanBlocks);
  // context sort over runs: taken when the runs are at most an eighth of the records
  L.chunks = ceil_div(nn, kChunk);
  L.run_cap = nn / 8 + kChunk;
  L.chunk_runs = take(sizeof(uint32_t) * L.chunks);
  L.run_base = take(sizeof(uint32_t) * L.chunks);
  L.run_cnt = take(sizeof(uint32_t) * L.run_cap);
  L.run_pos = take(sizeof(uint32_t) * L.run_cap);
  L.run_hist = take(sizeof(uint32_t) * 4 * kRadixBins);
  L.scan_bsum = take(sizeof(uint64_t) * kMaxScanBlocks);
  L.slb = take(sizeof(uint64_t) * 8 * ceil_div(nn, kSweepTile));
  L.tiles = take(sizeof(TileDesc) * L.match_tiles);
  uint64_t leaves = 1;
  while (leaves < L.match_tiles) leaves <<= 1;
  L.tree_leaves = leaves;
  L.tree = take(sizeof(int64_t) * 2 * leaves);
  L.pool_cap = L.match_tiles * (uint64_t)kMatchTile;
  L.pop_ts = take(sizeof(uint64_t) * L.pool_cap);
  L.pop_reg = take(sizeof(uint32_t) * L.pool_cap);
  L.pushes = take(sizeof(uint32_t) * L.pool_cap);
  L.op_parent = take(sizeof(uint32_t) * L.pool_cap);
  L.op_sum = take(sizeof(uint64_t) * L.pool_cap);
  L.inst = own_instances ? take(sizeof(argus_instance) * nn) : 0;
  L.excl = take(sizeof(uint64_t) * nn);
  L.hist_key = take(sizeof(uint32_t) * nn);
  L.agg_part = take(sizeof(uint64_t) * agg_part_words(n, c.num_regions));
  const uint64_t G = c.num_classes ? c.num_groups : 0;
  L.ov_mask = take(sizeof(uint64_t) * kMasks * (G ? G : 1));
  L.ov_q = take(sizeof(uint64_t) * kQPairs * (G ? G : 1));
  // merge path of the overlap events
  const bool ev = c.num_classes > 0;
  L.ctx_cap = ev ? (nn < kCtxCap ? nn : kCtxCap) : 0;
  // a segment of L events takes at most ceil(L / 4096) tiles in a two-way
  // pass and (L / 127 + 4) / 28 + 1 in a four-way one
  L.tiles_cap = ev ? ceil_div(nn, kSampStride * kSampPerTile) + L.ctx_cap + ceil_div(L.ctx_cap, 2) : 0;
  L.push_pos = take(ev ? sizeof(uint32_t) * L.pool_cap : 0);
  L.pop_pos = take(ev ? sizeof(uint32_t) * L.pool_cap : 0);
  L.ctx_list = take(sizeof(uint2) * L.ctx_cap);
  // segment arrays of every merge pass, ctx_cap + 1 entries per pass
  const uint64_t segs = ev ? kMaxMergePasses * (L.ctx_cap + 1) : 0;
  L.seg_run = take(sizeof(uint4) * segs);
  L.seg_tile0 = take(sizeof(uint32_t) * segs);
  L.seg_samp0 = take(sizeof(uint32_t) * segs);
  L.part = take(48 * L.tiles_cap);
  // tile records of the last merge round (2 + 2K + K(K + 1) words each)
  const uint64_t kc = c.num_classes;
  L.mslb = take(sizeof(uint64_t) * (2 + 2 * kc + kc * (kc + 1)) * L.tiles_cap);
  L.total = o;
  return L;
}

int fail(argus_attr* h, int code, const char* fmt, const char* detail = "") {
  if (h) {
    char buf[512];
    snprintf(buf, sizeof buf, fmt, detail);
    h->err = buf;
  }
  return code;
}

int check_config(const argus_attr_config* c, std::string* why) {
  if (!c) { *why = "config is NULL"; return ARGUS_E_INVAL; }
  if (c->abi_version != ARGUS_ATTR_ABI_VERSION) { *why = "abi_version mismatch"; return ARGUS_E_ABI; }
  if (c->num_regions < 1 || c->num_regions > 65535) { *why = "num_regions must be 1..65535"; return ARGUS_E_INVAL; }
  if (c->num_classes > 8) { *why = "num_classes must be 0..8"; return ARGUS_E_INVAL; }
  if (c->group_shift > 32) { *why = "group_shift must be 0..32"; return ARGUS_E_INVAL; }
  if (c->num_classes > 0) {
    if (c->num_groups < 1 || c->num_groups > (1u << 20)) { *why = "num_groups must be 1..2^20 when num_classes > 0"; return ARGUS_E_INVAL; }
    if (!c->d_region_class) { *why = "d_region_class is NULL while num_classes > 0"; return ARGUS_E_INVAL; }
  }
  if (c->flags & ~31u) { *why = "unknown flag bits"; return ARGUS_E_INVAL; }
  if (c->max_records >= (1ull << 31)) { *why = "max_records must be < 2^31"; return ARGUS_E_CAPACITY; }
  return ARGUS_OK;
}

}  // namespace

extern "C" {

int argus_attr_create(const argus_attr_config* cfg, argus_attr** out) {
  if (!out) return ARGUS_E_INVAL;
  *out = nullptr;
  std::string why;
  int rc = check_config(cfg, &why);
  if (rc != ARGUS_OK) return rc;
  argus_attr* h = new (std::nothrow) argus_attr();
  if (!h) return ARGUS_E_INVAL;
  h->cfg = *cfg;
  *out = h;
  return ARGUS_OK;
}

size_t argus_attr_workspace_bytes(const argus_attr* h, uint64_t n_records) {
  if (!h || n_records > h->cfg.max_records) return 0;
  return make_layout(h->cfg, n_records, true).total;
}

void argus_attr_destroy(argus_attr* h) {
  if (!h) return;
  for (auto& r : h->runs)
    for (hipEvent_t e : r.ev) (void)hipEventDestroy(e);
  for (hipEvent_t e : h->pool) (void)hipEventDestroy(e);
  delete h;
}

const char* argus_attr_last_error(const argus_attr* h) { return h ? h->err.c_str() : "handle is NULL"; }

int argus_attr_set_timing(argus_attr* h, int enable) {
  if (!h) return ARGUS_E_INVAL;
  h->timing = enable != 0;
  return ARGUS_OK;
}

int argus_attr_set_timing_filter(argus_attr* h, const char* name) {
  if (!h) return ARGUS_E_INVAL;
  h->filter = name ? name : "";
  return ARGUS_OK;
}

int argus_attr_kernel_times(argus_attr* h, const char** names, float* ms, int cap) {
  if (!h) return ARGUS_E_INVAL;
  int total = 0, k = 0;
  for (auto& r : h->runs) {
    if (r.ev.size() < 2) continue;
    if (hipEventSynchronize(r.ev.back()) != hipSuccess)
      return fail(h, ARGUS_E_HIP, "%s", "hipEventSynchronize failed");
    // launch j spans events (j, j + 1), or (2j, 2j + 1) when recorded in pairs
    const size_t nl = r.pairs ? r.ev.size() / 2 : r.ev.size() - 1;
    for (size_t j = 0; j < nl; ++j, ++total) {
      if (k >= cap) continue;
      const size_t e0 = r.pairs ? 2 * j : j;
      float t = 0;
      if (hipEventElapsedTime(&t, r.ev[e0], r.ev[e0 + 1]) != hipSuccess)
        return fail(h, ARGUS_E_HIP, "%s", "hipEventElapsedTime failed");
      if (names) names[k] = r.names[j];
      if (ms) ms[k] = t;
      ++k;
    }
  }
  for (auto& r : h->runs)
    for (hipEvent_t e : r.ev) h->pool.push_back(e);
  h->runs.clear();
  return total;
}

}  // extern "C"

namespace {

// Argument checks shared by both run entry points (no GPU call).
int check_run_args(argus_attr* h, const argus_record* d_records, uint64_t n,
                   const argus_attr_outputs* out) {
  const argus_attr_config& c = h->cfg;
  if (!out) return fail(h, ARGUS_E_INVAL, "%s", "outputs is NULL");
  if (n > c.max_records) return fail(h, ARGUS_E_CAPACITY, "%s", "n_records exceeds max_records");
  if (n > 0 && !d_records) return fail(h, ARGUS_E_INVAL, "%s", "d_records is NULL");
  if (!out->d_counters || !out->d_region_stats)
    return fail(h, ARGUS_E_INVAL, "%s", "d_counters and d_region_stats are required");
  if (c.num_classes > 0 && (!out->d_overlap_group || !out->d_overlap_global))
    return fail(h, ARGUS_E_INVAL, "%s", "overlap outputs are required when num_classes > 0");
  if ((c.flags & ARGUS_OUT_INSTANCES) && !out->d_instances)
    return fail(h, ARGUS_E_INVAL, "%s", "ARGUS_OUT_INSTANCES set but d_instances is NULL");
  if ((c.flags & ARGUS_OUT_INSTANCE_EXCL) && !out->d_instance_excl)
    return fail(h, ARGUS_E_INVAL, "%s", "ARGUS_OUT_INSTANCE_EXCL set but d_instance_excl is NULL");
  if (((uintptr_t)d_records & 15) != 0) return fail(h, ARGUS_E_ALIGN, "%s", "records must be 16-byte aligned");
  return ARGUS_OK;
}

// The current device, checked (once per device and handle) to be gfx950.
int current_device(argus_attr* h, int* dev_out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(h, ARGUS_E_HIP, "%s", "hipGetDevice failed");
  if (h->device_checked != dev) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess)
      return fail(h, ARGUS_E_HIP, "%s", "hipGetDeviceProperties failed");
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
      return fail(h, ARGUS_E_DEVICE, "device is %s, this library is built for gfx950", prop.gcnArchName);
    h->device_checked = dev;
  }
  *dev_out = dev;
  return ARGUS_OK;
}

// Enqueue every step of one run on `stream_v`, with the workspace at `base`
// (256-byte aligned, at least make_layout(...).total bytes).
int enqueue_run(argus_attr* h, const argus_record* d_records, uint64_t n, char* base,
                const argus_attr_outputs* out, void* stream_v) {
  const argus_attr_config& c = h->cfg;
  const bool own_inst = !(c.flags & ARGUS_OUT_INSTANCES);
  const Layout L = make_layout(c, n, own_inst);
  hipStream_t s = (hipStream_t)stream_v;
  RunArgs a{};
  a.rec = d_records;
  a.n = n;
  a.R = c.num_regions;
  a.K = c.num_classes;
  a.G = c.num_classes ? c.num_groups : 0;
  a.shift = c.group_shift;
  a.flags = c.flags;
  a.region_class = c.d_region_class;
  a.out = *out;
  Work& w = a.w;
  w.plan = (DevPlan*)(base + L.plan);
  w.rec_hist = (uint32_t*)(base + L.rec_hist);
  w.rec_off = (uint32_t*)(base + L.rec_off);
  w.ev_hist = (uint32_t*)(base + L.ev_hist);
  w.ev_off = (uint32_t*)(base + L.ev_off);
  w.tile_ctr = (uint32_t*)(base + L.tile_ctr);
  for (int b = 0; b < 2; ++b) {
    w.key[b] = (uint64_t*)(base + L.key[b]);
    w.pay[b] = (uint32_t*)(base + L.pay[b]);
    w.ctxw[b] = (uint32_t*)(base + L.ctxw[b]);
    w.lb[b] = (uint64_t*)(base + L.lb[b]);
  }
  w.tsum = (uint64_t*)(base + L.tsum);
  w.carry = (TileCarry*)(base + L.carry);
  w.bsum = (BlockSum*)(base + L.bsum);
  w.chunk_runs = (uint32_t*)(base + L.chunk_runs);
  w.run_base = (uint32_t*)(base + L.run_base);
  w.run_cnt = (uint32_t*)(base + L.run_cnt);
  w.run_pos = (uint32_t*)(base + L.run_pos);
  w.run_hist = (uint32_t*)(base + L.run_hist);
  w.scan_bsum = (uint64_t*)(base + L.scan_bsum);
  w.chunks = L.chunks;
  w.run_cap = L.run_cap;
  w.slb = (uint64_t*)(base + L.slb);
  w.mslb = (uint64_t*)(base + L.mslb);
  w.tiles = (TileDesc*)(base + L.tiles);
  w.tree = (int64_t*)(base + L.tree);
  w.pop_ts = (uint64_t*)(base + L.pop_ts);
  w.pop_reg = (uint32_t*)(base + L.pop_reg);
  w.pushes = (uint32_t*)(base + L.pushes);
  w.op_parent = (uint32_t*)(base + L.op_parent);
  w.op_sum = (uint64_t*)(base + L.op_sum);
  w.inst = own_inst ? (argus_instance*)(base + L.inst) : out->d_instances;
  // exclusive times are accumulated in place, in the caller's output when
  // it asks for them
  w.excl = (h->cfg.flags & ARGUS_OUT_INSTANCE_EXCL) ? out->d_instance_excl
                                                   : (uint64_t*)(base + L.excl);
  w.hist_key = (uint32_t*)(base + L.hist_key);
  w.agg_part = agg_part_words(n, h->cfg.num_regions) ? (uint64_t*)(base + L.agg_part) : nullptr;
  w.ov_mask = (uint64_t*)(base + L.ov_mask);
  w.ov_q = (uint64_t*)(base + L.ov_q);
  w.push_pos = (uint32_t*)(base + L.push_pos);
  w.pop_pos = (uint32_t*)(base + L.pop_pos);
  w.ctx_list = (uint2*)(base + L.ctx_list);
  w.seg_run = (uint4*)(base + L.seg_run);
  w.seg_tile0 = (uint32_t*)(base + L.seg_tile0);
  w.seg_samp0 = (uint32_t*)(base + L.seg_samp0);
  w.part = (uint32_t*)(base + L.part);
  w.ctx_cap = L.ctx_cap;
  w.tiles_cap = L.tiles_cap;
  w.lb_words = L.lb_words;
  w.tree_leaves = L.tree_leaves;
  w.match_tiles = L.match_tiles;
  w.pool_cap = L.pool_cap;

  // Timing events (one per launch, recorded on the run's stream).
  argus_attr::TimedRun* tr = nullptr;
  auto new_event = [&](hipEvent_t* e) -> bool {
    if (!h->pool.empty()) {
      *e = h->pool.back();
      h->pool.pop_back();
      return true;
    }
    return hipEventCreate(e) == hipSuccess;
  };
  if (h->timing) {
    h->runs.emplace_back();
    tr = &h->runs.back();
    tr->pairs = !h->filter.empty();
    if (!tr->pairs) {
      hipEvent_t e;
      if (!new_event(&e) || hipEventRecord(e, s) != hipSuccess)
        return fail(h, ARGUS_E_HIP, "%s", "timing event failed");
      tr->ev.push_back(e);
    }
  }
  auto record = [&]() -> bool {
    hipEvent_t ev;
    if (!new_event(&ev) || hipEventRecord(ev, s) != hipSuccess) return false;
    tr->ev.push_back(ev);
    return true;
  };
  auto step = [&](const char* name, auto&& launch) -> bool {
    const bool timed = tr && (!tr->pairs || h->filter == name);
    if (timed && tr->pairs && !record()) return false;  // before the launch
    hipError_t e = launch();
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) {
      fail(h, ARGUS_E_HIP, "launch failed: %s", name);
      h->err += std::string(" (") + hipGetErrorString(e) + ")";
      return false;
    }
    if (timed) {
      if (!record()) return false;
      tr->names.push_back(name);
    }
    return true;
  };

  if (!step("init", [&] { return launch_init(a, s); })) return ARGUS_E_HIP;
  if (n == 0) return ARGUS_OK;
  if (!step("ingest", [&] { return launch_ingest(a, s); })) return ARGUS_E_HIP;
  if (!step("plan", [&] { return launch_plan(a, s); })) return ARGUS_E_HIP;
  static const char* rnames[kSlots] = {
      "radix_ctx0", "radix_ctx1", "radix_ctx2", "radix_ctx3", "radix_ts0", "radix_ts1",
      "radix_ts2", "radix_ts3", "radix_ts4", "radix_ts5", "radix_ts6", "radix_ts7",
      "radix_ctx0b", "radix_ctx1b", "radix_ctx2b", "radix_ctx3b"};
  // context sort over runs (each launch returns at once on the radix path)
  if (!step("runs_base", [&] { return launch_runs_base(a, s); })) return ARGUS_E_HIP;
  if (!step("runs_compact", [&] { return launch_runs_compact(a, s); })) return ARGUS_E_HIP;
  if (!step("runs_plan", [&] { return launch_runs_plan(a, s); })) return ARGUS_E_HIP;
  for (int sl = 0; sl < kPhase2Slot; ++sl)
    if (!step(rnames[sl], [&] { return launch_radix_pass(a, 0, sl, n, s); })) return ARGUS_E_HIP;
  if (!step("runs_pos", [&] { return launch_runs_pos(a, s); })) return ARGUS_E_HIP;
  if (!step("runs_scatter", [&] { return launch_runs_scatter(a, s); })) return ARGUS_E_HIP;
  if (!step("tile_sums", [&] { return launch_tsum(a, 0, s); })) return ARGUS_E_HIP;
  if (!step("runs_check", [&] { return launch_runs_check(a, s); })) return ARGUS_E_HIP;
  if (!step("tile_sums_runs", [&] { return launch_tsum_codes(a, s); })) return ARGUS_E_HIP;
  if (!step("ts_hist", [&] { return launch_ts_hist(a, s); })) return ARGUS_E_HIP;
  if (!step("lb_clear", [&] { return launch_lb_clear(a, s); })) return ARGUS_E_HIP;
  if (!step("plan2", [&] { return launch_plan2(a, s); })) return ARGUS_E_HIP;
  for (int sl = kPhase2Slot; sl < kSlots; ++sl)
    if (!step(rnames[sl], [&] { return launch_radix_pass(a, 0, sl, n, s); })) return ARGUS_E_HIP;
  if (!step("tile_sums_full", [&] { return launch_tsum(a, 1, s); })) return ARGUS_E_HIP;
  if (!step("tile_scan", [&] { return launch_mscan(a, s); })) return ARGUS_E_HIP;
  if (!step("match", [&] { return launch_match(a, s); })) return ARGUS_E_HIP;
  if (!step("tree", [&] { return launch_tree(a, s); })) return ARGUS_E_HIP;
  if (!step("resolve", [&] { return launch_resolve(a, s); })) return ARGUS_E_HIP;
  if (a.K > 0 && !step("merge_plan", [&] { return launch_mplan(a, s); })) return ARGUS_E_HIP;
  if (!step("agg", [&] { return launch_agg(a, s); })) return ARGUS_E_HIP;
  if (!step("hist", [&] { return launch_hist(a, s); })) return ARGUS_E_HIP;
  if (a.K > 0) {
    static const char* enames[kSlots] = {
        "ev_radix_ts0", "ev_radix_ts1", "ev_radix_ts2", "ev_radix_ts3", "ev_radix_ts4",
        "ev_radix_ts5", "ev_radix_ts6", "ev_radix_ts7", "ev_radix_g0", "ev_radix_g1",
        "ev_radix_g2", "ev_radix_g3", "ev_unused12", "ev_unused13", "ev_unused14", "ev_unused15"};
    if (!step("ev_plan", [&] { return launch_ev_plan(a, s); })) return ARGUS_E_HIP;
    if (!step("ev_clear", [&] { return launch_ev_clear(a, s); })) return ARGUS_E_HIP;
    for (int sl = 0; sl < 12; ++sl)
      if (!step(enames[sl], [&] { return launch_radix_pass(a, 1, sl, 2 * n, s); })) return ARGUS_E_HIP;
    // Merge passes (device-planned; a pass beyond the plan returns at once).
    // Bits are merged two per pass; the last pass is merged and swept by one
    // kernel; there is always at least one pass (a group of one context is a
    // run by itself).
    static const char* mnames[kMaxMergePasses][2] = {
        {"mpart0", "merge0"}, {"mpart1", "merge1"}, {"mpart2", "merge2"}, {"mpart3", "merge3"}};
    const int bits = a.shift < (uint32_t)kMaxMergeBits ? (int)a.shift : kMaxMergeBits;
    int rounds = (bits + 1) / 2;
    if (rounds < 1) rounds = 1;
    if (!step("mseg", [&] { return launch_mseg(a, rounds, s); })) return ARGUS_E_HIP;
    for (int r = 0; r < rounds; ++r) {
      if (!step(mnames[r][0], [&] { return launch_mpart(a, r, s); })) return ARGUS_E_HIP;
      if (r + 1 < rounds && !step(mnames[r][1], [&] { return launch_merge(a, r, s); })) return ARGUS_E_HIP;
    }
    if (!step("merge_sweep", [&] { return launch_merge_sweep(a, s); })) return ARGUS_E_HIP;
    if (!step("sweep", [&] { return launch_sweep(a, s); })) return ARGUS_E_HIP;
    if (!step("ov_final", [&] { return launch_ov_final(a, s); })) return ARGUS_E_HIP;
  }
  return ARGUS_OK;
}

// Built-in workspace of the allocation-free entry point: one copy per device,
// held until the process ends.  Host code never uses the array's name as a
// device address (on the host it names a stand-in); it uses the address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[ARGUS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (the current device), looked
// up on the first call for that device.
int scratch_on_device(argus_attr* h, int dev, char** out) {
  if (dev < 0 || dev >= kMaxDevices)
    return fail(h, ARGUS_E_DEVICE, "%s", "device ordinal beyond the built-in workspace table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      fail(h, ARGUS_E_HIP, "%s", "hipGetSymbolAddress of the built-in workspace failed");
      if (e != hipSuccess) h->err += std::string(" (") + hipGetErrorString(e) + ")";
      return ARGUS_E_HIP;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = (char*)g_scratch_ptr[dev];
  return ARGUS_OK;
}

}  // namespace

extern "C" {

int argus_attr_run(argus_attr* h, const argus_record* d_records, uint64_t n,
                   void* d_workspace, size_t workspace_bytes,
                   const argus_attr_outputs* out, void* stream_v) {
  if (!h) return ARGUS_E_INVAL;
  h->err.clear();
  int rc = check_run_args(h, d_records, n, out);
  if (rc != ARGUS_OK) return rc;
  if (!d_workspace) return fail(h, ARGUS_E_INVAL, "%s", "d_workspace is NULL");
  if (((uintptr_t)d_workspace & (kAlign - 1)) != 0)
    return fail(h, ARGUS_E_ALIGN, "%s", "workspace must be 256-byte aligned");
  const bool own_inst = !(h->cfg.flags & ARGUS_OUT_INSTANCES);
  if (workspace_bytes < make_layout(h->cfg, n, own_inst).total)
    return fail(h, ARGUS_E_CAPACITY, "%s", "workspace too small");
  int dev = 0;
  rc = current_device(h, &dev);
  if (rc != ARGUS_OK) return rc;
  return enqueue_run(h, d_records, n, (char*)d_workspace, out, stream_v);
}

int argus_attr_run_noalloc(argus_attr* h, const argus_record* d_records, uint64_t n,
                           const argus_attr_outputs* out, void* stream_v) {
  if (!h) return ARGUS_E_INVAL;
  h->err.clear();
  int rc = check_run_args(h, d_records, n, out);
  if (rc != ARGUS_OK) return rc;
  const bool own_inst = !(h->cfg.flags & ARGUS_OUT_INSTANCES);
  const size_t need = make_layout(h->cfg, n, own_inst).total;
  if (need > (size_t)ARGUS_NOALLOC_SCRATCH_BYTES) {
    char buf[256];
    snprintf(buf, sizeof buf,
             "n_records needs %zu bytes of workspace; the built-in workspace holds %zu "
             "(use argus_attr_run with a caller workspace)",
             need, (size_t)ARGUS_NOALLOC_SCRATCH_BYTES);
    h->err = buf;
    return ARGUS_E_CAPACITY;
  }
  int dev = 0;
  rc = current_device(h, &dev);
  if (rc != ARGUS_OK) return rc;
  char* base = nullptr;
  rc = scratch_on_device(h, dev, &base);
  if (rc != ARGUS_OK) return rc;
  return enqueue_run(h, d_records, n, base, out, stream_v);
}

}  // extern "C"
