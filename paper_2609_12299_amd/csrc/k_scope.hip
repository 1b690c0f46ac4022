// k_scope.hip -- iteration ordinals and scoped per-region statistics.
//
// The paper's Section 3.2 separates a region (the code a developer changes)
// from its scope (which dynamic executions are reported: a warp role, an
// iteration window, an SM subset), and Section 3.3 specialises probes to one
// iteration of a loop region.  The iteration of an instance is its ordinal
// among the instances of its context with the same BEGIN region, in
// canonical (context, begin time) order.
//
// Ordinals: the instance array is already ordered by context, so a stable
// sort by region alone yields (region, context, canonical) order, in which
// the instances of one (context, region) form a run; an instance's ordinal
// is its distance from the start of its run.  The sort is an LSD radix sort
// over the region's 8-bit digits (one pass for up to 256 regions, else two):
// per 4096-element tile a digit histogram, one exclusive scan over the
// digit-major histograms, then a stable scatter that ranks each tile's
// elements with eight ballots per wave.  Run starts come from a wave
// max-scan of the run heads, with one binary search per wave for a run that
// began before it.  The ordinals are scattered back to canonical order and
// the scoped statistics are taken in canonical order with global atomics.
#include <string.h>

#include <mutex>

#include "internal.h"

namespace argus {

constexpr int kScThreads = 256;
constexpr int kScRounds = 16;
constexpr uint32_t kScTile = kScThreads * kScRounds;  // 4096 elements
constexpr uint32_t kScScanBlock = 4096;                // entries per scan block

struct ScopeArgs {
  const argus_instance* inst;
  const uint64_t* excl;
  const uint64_t* n_inst;
  uint64_t max_inst;
  uint32_t R;
  argus_scope sc;
  const uint8_t* region_mask;
  uint32_t* ordinal;
  uint64_t* stats;
  uint64_t* counters;
  // workspace
  uint32_t* key[2];
  uint64_t* val[2];  // ctx << 32 | canonical index
  uint32_t* hist;    // [256][tiles_max], digit-major
  uint32_t* bsum;    // scan block sums
  uint64_t tiles_max;
};

__device__ __forceinline__ uint64_t sc_count(const ScopeArgs& a) {
  const uint64_t v = *a.n_inst;
  return v < a.max_inst ? v : a.max_inst;
}

// Element e of pass `pass` (source: the instances for pass 0, else the
// buffer the previous pass wrote).
__device__ __forceinline__ void sc_load(const ScopeArgs& a, int pass, uint64_t e, uint32_t* key,
                                        uint64_t* val) {
  if (pass == 0) {
    const uint4 h1 = reinterpret_cast<const uint4*>(a.inst)[2 * e + 1];
    *key = h1.w & 0xFFFFu;
    *val = ((uint64_t)h1.x << 32) | e;
  } else {
    *key = a.key[(pass - 1) & 1][e];
    *val = a.val[(pass - 1) & 1][e];
  }
}

// Fill kernel for the outputs that are accumulated.
__global__ __launch_bounds__(kScThreads) void k_sc_init(ScopeArgs a) {
  const uint64_t total = (uint64_t)a.R * ARGUS_RS_WIDTH;
  for (uint64_t i = (uint64_t)blockIdx.x * kScThreads + threadIdx.x; i < total;
       i += (uint64_t)gridDim.x * kScThreads) {
    const uint32_t col = (uint32_t)(i % ARGUS_RS_WIDTH);
    a.stats[i] = (col == ARGUS_RS_INCL_MIN || col == ARGUS_RS_EXCL_MIN) ? kU64Max : 0ull;
  }
  if (blockIdx.x == 0 && threadIdx.x < ARGUS_SC_NUM_COUNTERS) a.counters[threadIdx.x] = 0;
}

// Per tile: counts of each digit, written digit-major (zeros for tiles past
// the element count, so that the scan sees a complete table).
__global__ __launch_bounds__(kScThreads) void k_sc_hist(ScopeArgs a, int pass) {
  __shared__ uint32_t s_cnt[256];
  const uint64_t n = sc_count(a);
  const uint64_t tile = blockIdx.x;
  s_cnt[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t base = tile * kScTile;
  for (uint32_t j = 0; j < kScRounds; ++j) {
    const uint64_t e = base + (uint64_t)j * kScThreads + threadIdx.x;
    if (e < n) {
      uint32_t key;
      uint64_t val;
      sc_load(a, pass, e, &key, &val);
      atomicAdd(&s_cnt[(key >> (8 * pass)) & 0xFFu], 1u);
    }
  }
  __syncthreads();
  a.hist[(uint64_t)threadIdx.x * a.tiles_max + tile] = s_cnt[threadIdx.x];
}

// Exclusive scan of the digit-major table, in three launches: block sums,
// their scan (one block), then each block's scan plus its base.
__global__ __launch_bounds__(kScThreads) void k_sc_scan_sums(ScopeArgs a) {
  __shared__ uint32_t s_part[kScThreads / 64];
  const uint64_t total = 256ull * a.tiles_max;
  const uint64_t base = (uint64_t)blockIdx.x * kScScanBlock;
  uint32_t s = 0;
  for (uint32_t j = threadIdx.x; j < kScScanBlock; j += kScThreads)
    if (base + j < total) s += a.hist[base + j];
  s = rows_sum32(row_sum32(s));
  if ((threadIdx.x & 63) == 0) s_part[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) a.bsum[blockIdx.x] = s_part[0] + s_part[1] + s_part[2] + s_part[3];
}

__global__ __launch_bounds__(1024) void k_sc_scan_top(ScopeArgs a, uint32_t blocks) {
  __shared__ uint32_t s_carry;
  __shared__ uint32_t s_w[16];
  if (threadIdx.x == 0) s_carry = 0;
  __syncthreads();
  for (uint32_t b0 = 0; b0 < blocks; b0 += 1024) {
    const uint32_t b = b0 + threadIdx.x;
    const uint32_t v = b < blocks ? a.bsum[b] : 0u;
    // inclusive scan over the block of 1024 values
    uint32_t x = v;
    const uint32_t lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(x, d);
      if (lane >= (uint32_t)d) x += y;
    }
    if (lane == 63) s_w[w] = x;
    __syncthreads();
    uint32_t wpre = 0;
    for (uint32_t k = 0; k < w; ++k) wpre += s_w[k];
    const uint32_t carry = s_carry;
    if (b < blocks) a.bsum[b] = carry + wpre + x - v;  // exclusive
    __syncthreads();
    if (threadIdx.x == 1023) s_carry = carry + wpre + x;
    __syncthreads();
  }
}

__global__ __launch_bounds__(kScThreads) void k_sc_scan_apply(ScopeArgs a) {
  __shared__ uint32_t s_w[kScThreads / 64];
  __shared__ uint32_t s_carry;
  const uint64_t total = 256ull * a.tiles_max;
  const uint64_t base = (uint64_t)blockIdx.x * kScScanBlock;
  if (threadIdx.x == 0) s_carry = a.bsum[blockIdx.x];
  __syncthreads();
  const uint32_t lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (uint32_t j0 = 0; j0 < kScScanBlock; j0 += kScThreads) {
    const uint64_t i = base + j0 + threadIdx.x;
    const uint32_t v = i < total ? a.hist[i] : 0u;
    uint32_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(x, d);
      if (lane >= (uint32_t)d) x += y;
    }
    if (lane == 63) s_w[w] = x;
    __syncthreads();
    uint32_t wpre = 0;
    for (uint32_t k = 0; k < w; ++k) wpre += s_w[k];
    const uint32_t carry = s_carry;
    if (i < total) a.hist[i] = carry + wpre + x - v;
    __syncthreads();
    if (threadIdx.x == kScThreads - 1) s_carry = carry + wpre + x;
    __syncthreads();
  }
}

// Stable scatter of one tile: in each round of 256 elements, each wave finds
// the lanes that share its digit with eight ballots; per-wave digit counts
// in LDS give the wave's offset within the round, and a running count per
// digit carries the tile's earlier rounds.
__global__ __launch_bounds__(kScThreads) void k_sc_scatter(ScopeArgs a, int pass) {
  __shared__ uint32_t s_wcnt[4][256];
  __shared__ uint32_t s_run[256];
  __shared__ uint32_t s_base[256];
  const uint64_t n = sc_count(a);
  const uint64_t tile = blockIdx.x;
  const uint32_t tid = threadIdx.x, w = tid >> 6;
  s_run[tid] = 0;
  s_base[tid] = a.hist[(uint64_t)tid * a.tiles_max + tile];
  const uint64_t lt = lanemask_lt();
  uint32_t* dk = a.key[pass & 1];
  uint64_t* dv = a.val[pass & 1];
  for (uint32_t j = 0; j < kScRounds; ++j) {
    const uint64_t e = tile * kScTile + (uint64_t)j * kScThreads + tid;
    const bool valid = e < n;
    uint32_t key = 0;
    uint64_t val = 0;
    if (valid) sc_load(a, pass, e, &key, &val);
    const uint32_t d = (key >> (8 * pass)) & 0xFFu;
#pragma unroll
    for (int q = 0; q < 4; ++q) s_wcnt[q][tid] = 0;
    __syncthreads();
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t bal = __ballot((d >> b) & 1u);
      peers &= ((d >> b) & 1u) ? bal : ~bal;
    }
    const uint32_t rank = (uint32_t)__popcll(peers & lt);
    if (valid && rank == 0) s_wcnt[w][d] = (uint32_t)__popcll(peers);
    __syncthreads();
    {
      // thread tid owns digit tid: wave offsets within the round, in place
      uint32_t run = s_run[tid];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t c = s_wcnt[q][tid];
        s_wcnt[q][tid] = run;
        run += c;
      }
      s_run[tid] = run;
    }
    __syncthreads();
    if (valid) {
      const uint64_t dst = (uint64_t)s_base[d] + s_wcnt[w][d] + rank;
      dk[dst] = key;
      dv[dst] = val;
    }
    __syncthreads();
  }
}

// First position in the sorted (key, context) sequence [0, hi] that equals
// (key, ctx): the start of that run.
__device__ __forceinline__ uint64_t sc_run_start(const uint32_t* k, const uint64_t* v,
                                                 uint64_t hi, uint32_t key, uint32_t ctx) {
  uint64_t lo = 0;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) >> 1;
    const uint32_t km = k[mid], cm = (uint32_t)(v[mid] >> 32);
    const bool less = km < key || (km == key && cm < ctx);
    if (less) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Ordinal of each sorted element: its distance from the start of its
// (region, context) run, scattered to canonical order.
__global__ __launch_bounds__(kScThreads) void k_sc_ordinal(ScopeArgs a, int buf) {
  const uint64_t n = sc_count(a);
  const uint32_t* k = a.key[buf];
  const uint64_t* v = a.val[buf];
  const uint32_t lane = threadIdx.x & 63;
  uint32_t best = 0;
  const uint64_t nwaves = (uint64_t)gridDim.x * (kScThreads / 64);
  for (uint64_t wv = ((uint64_t)blockIdx.x * kScThreads + threadIdx.x) >> 6;
       wv * 64 < n; wv += nwaves) {
    const uint64_t e0 = wv * 64, e = e0 + lane;
    const bool valid = e < n;
    uint32_t key = 0, ctx = 0, idx = 0;
    bool head = false;
    if (valid) {
      key = k[e];
      const uint64_t vv = v[e];
      ctx = (uint32_t)(vv >> 32);
      idx = (uint32_t)vv;
      head = e == 0 || k[e - 1] != key || (uint32_t)(v[e - 1] >> 32) != ctx;
    }
    // start of the run: the last head at or before this lane, else the run
    // that was open when the wave began (one binary search for the wave)
    int64_t h = head ? (int64_t)e : -1;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int64_t o = __shfl_up(h, d);
      if (lane >= (uint32_t)d && o > h) h = o;
    }
    if (__ballot(valid && h < 0)) {
      const uint32_t k0 = __shfl(key, 0), c0 = __shfl(ctx, 0);
      uint64_t s0 = 0;
      if (lane == 0) s0 = sc_run_start(k, v, e0, k0, c0);
      s0 = __shfl(s0, 0);
      if (h < 0) h = (int64_t)s0;
    }
    if (valid) {
      const uint32_t ord = (uint32_t)(e - (uint64_t)h);
      a.ordinal[idx] = ord;
      best = best > ord + 1 ? best : ord + 1;
    }
  }
  // wave maximum, one atomic per wave
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    const uint32_t o = __shfl_xor(best, d);
    best = best > o ? best : o;
  }
  if (lane == 0 && best)
    atomicMax((unsigned long long*)&a.counters[ARGUS_SC_N_ITERATIONS], (unsigned long long)best);
}

__device__ __forceinline__ bool in_range32(uint64_t v, uint32_t lo, uint32_t hi) {
  return lo <= v && v <= hi;
}

// Scoped statistics in canonical order.
__global__ __launch_bounds__(kScThreads) void k_sc_stats(ScopeArgs a) {
  const uint64_t n = sc_count(a);
  const uint4* inst = reinterpret_cast<const uint4*>(a.inst);
  uint32_t c_in = 0, c_m = 0, c_mm = 0, c_u = 0, c_s = 0;
  for (uint64_t x = (uint64_t)blockIdx.x * kScThreads + threadIdx.x; x < n;
       x += (uint64_t)gridDim.x * kScThreads) {
    const uint4 h0 = inst[2 * x], h1 = inst[2 * x + 1];
    const uint32_t ctx = h1.x, reg = h1.w & 0xFFFFu, ereg = h1.w >> 16;
    const uint64_t group = a.sc.group_shift >= 32 ? 0ull : (uint64_t)(ctx >> a.sc.group_shift);
    const bool in = in_range32(ctx & a.sc.role_mask, a.sc.role_lo, a.sc.role_hi) &&
                    in_range32(group, a.sc.group_lo, a.sc.group_hi) &&
                    in_range32(a.ordinal[x], a.sc.iter_lo, a.sc.iter_hi) && reg < a.R &&
                    (!a.region_mask || a.region_mask[reg] != 0);
    if (!in) continue;
    c_in += 1;
    unsigned long long* row = (unsigned long long*)(a.stats + (uint64_t)reg * ARGUS_RS_WIDTH);
    if (ereg == kNoEnd) {
      c_u += 1;
      atomicAdd(&row[ARGUS_RS_UNCLOSED], 1ull);
      continue;
    }
    if (ereg != reg) {
      c_mm += 1;
      atomicAdd(&row[ARGUS_RS_MISM_AS_BEGIN], 1ull);
      if (ereg < a.R)
        atomicAdd((unsigned long long*)(a.stats + (uint64_t)ereg * ARGUS_RS_WIDTH +
                                        ARGUS_RS_MISM_AS_END), 1ull);
      continue;
    }
    c_m += 1;
    const uint64_t tb = (uint64_t)h0.x | ((uint64_t)h0.y << 32);
    const uint64_t te = (uint64_t)h0.z | ((uint64_t)h0.w << 32);
    const uint64_t d = te - tb, ex = a.excl[x];
    atomicAdd(&row[ARGUS_RS_COUNT], 1ull);
    atomicAdd(&row[ARGUS_RS_INCL_SUM], (unsigned long long)d);
    atomicAdd(&row[ARGUS_RS_EXCL_SUM], (unsigned long long)ex);
    atomicMin(&row[ARGUS_RS_INCL_MIN], (unsigned long long)d);
    atomicMax(&row[ARGUS_RS_INCL_MAX], (unsigned long long)d);
    atomicMin(&row[ARGUS_RS_EXCL_MIN], (unsigned long long)ex);
    atomicMax(&row[ARGUS_RS_EXCL_MAX], (unsigned long long)ex);
    atomicAdd(&row[ARGUS_RS_HIST_INCL + bit_width64(d)], 1ull);
    atomicAdd(&row[ARGUS_RS_HIST_EXCL + bit_width64(ex)], 1ull);
    const uint32_t par = h1.y;
    if (par != kNoParent && par < n && (inst[2 * (uint64_t)par + 1].w & 0xFFFFu) == reg) {
      c_s += 1;
      atomicAdd(&row[ARGUS_RS_SELF_NESTED], 1ull);
    }
  }
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t v[5] = {c_in, c_m, c_mm, c_u, c_s};
  const int slot[5] = {ARGUS_SC_N_IN_SCOPE, ARGUS_SC_N_MATCHED, ARGUS_SC_N_MISMATCHED,
                       ARGUS_SC_N_UNCLOSED, ARGUS_SC_N_SELF_NESTED};
#pragma unroll
  for (int q = 0; q < 5; ++q) {
    const uint32_t t = rows_sum32(row_sum32(v[q]));
    if (lane == 0 && t) atomicAdd((unsigned long long*)&a.counters[slot[q]], (unsigned long long)t);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) a.counters[ARGUS_SC_N_INSTANCES] = n;
}

}  // namespace argus

using namespace argus;

namespace {

constexpr size_t kScAlign = 256;
size_t sc_align(size_t v) { return (v + kScAlign - 1) & ~(kScAlign - 1); }

struct ScLayout {
  size_t key[2], val[2], hist, bsum, total;
  uint64_t tiles, scan_blocks;
};

ScLayout sc_layout(uint64_t max_inst) {
  ScLayout L{};
  const uint64_t m = max_inst ? max_inst : 1;
  L.tiles = (m + kScTile - 1) / kScTile;
  L.scan_blocks = (256ull * L.tiles + kScScanBlock - 1) / kScScanBlock;
  size_t o = 0;
  auto take = [&](size_t b) {
    const size_t at = o;
    o = sc_align(o + (b ? b : 1));
    return at;
  };
  for (int b = 0; b < 2; ++b) {
    L.key[b] = take(sizeof(uint32_t) * m);
    L.val[b] = take(sizeof(uint64_t) * m);
  }
  L.hist = take(sizeof(uint32_t) * 256 * L.tiles);
  L.bsum = take(sizeof(uint32_t) * L.scan_blocks);
  L.total = o;
  return L;
}

std::mutex g_sc_mu;
int g_sc_dev_ok[64] = {};

int sc_check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ARGUS_E_HIP;
  if (dev < 0 || dev >= 64) return ARGUS_E_DEVICE;
  std::lock_guard<std::mutex> lock(g_sc_mu);
  if (!g_sc_dev_ok[dev]) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return ARGUS_E_HIP;
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return ARGUS_E_DEVICE;
    g_sc_dev_ok[dev] = 1;
  }
  return ARGUS_OK;
}

uint32_t sc_grid(uint64_t items, uint64_t per_block, uint32_t cap) {
  uint64_t g = (items + per_block - 1) / per_block;
  if (g > cap) g = cap;
  return g < 1 ? 1u : (uint32_t)g;
}

}  // namespace

extern "C" size_t argus_attr_scope_workspace_bytes(uint64_t max_instances) {
  if (max_instances >= (1ull << 31)) return 0;
  return sc_layout(max_instances).total;
}

extern "C" int argus_attr_scope(const argus_scope_config* cfg, const argus_scope_io* io,
                                void* d_workspace, size_t workspace_bytes, void* stream_v) {
  if (!cfg || !io) return ARGUS_E_INVAL;
  if (cfg->abi_version != ARGUS_ATTR_ABI_VERSION) return ARGUS_E_ABI;
  if (cfg->num_regions < 1 || cfg->num_regions > 65535) return ARGUS_E_INVAL;
  if (io->max_instances >= (1ull << 31)) return ARGUS_E_CAPACITY;
  if (!io->d_n_instances || !io->d_ordinal || !io->d_stats || !io->d_counters)
    return ARGUS_E_INVAL;
  if (io->max_instances > 0 && (!io->d_instances || !io->d_instance_excl)) return ARGUS_E_INVAL;
  if (!d_workspace) return ARGUS_E_INVAL;
  if (((uintptr_t)io->d_instances & 15) || ((uintptr_t)io->d_instance_excl & 7) ||
      ((uintptr_t)io->d_n_instances & 7) || ((uintptr_t)io->d_ordinal & 3) ||
      ((uintptr_t)io->d_stats & 7) || ((uintptr_t)io->d_counters & 7) ||
      ((uintptr_t)d_workspace & (kScAlign - 1)))
    return ARGUS_E_ALIGN;
  const ScLayout L = sc_layout(io->max_instances);
  if (workspace_bytes < L.total) return ARGUS_E_CAPACITY;
  const int dc = sc_check_device();
  if (dc != ARGUS_OK) return dc;

  char* base = (char*)d_workspace;
  ScopeArgs a{};
  a.inst = io->d_instances;
  a.excl = io->d_instance_excl;
  a.n_inst = io->d_n_instances;
  a.max_inst = io->max_instances;
  a.R = cfg->num_regions;
  a.sc = cfg->scope;
  a.region_mask = io->d_region_mask;
  a.ordinal = io->d_ordinal;
  a.stats = io->d_stats;
  a.counters = io->d_counters;
  for (int b = 0; b < 2; ++b) {
    a.key[b] = (uint32_t*)(base + L.key[b]);
    a.val[b] = (uint64_t*)(base + L.val[b]);
  }
  a.hist = (uint32_t*)(base + L.hist);
  a.bsum = (uint32_t*)(base + L.bsum);
  a.tiles_max = L.tiles;
  hipStream_t s = (hipStream_t)stream_v;
  const uint32_t tiles = (uint32_t)L.tiles;
  const int passes = cfg->num_regions > 256 ? 2 : 1;
  hipLaunchKernelGGL(k_sc_init, dim3(sc_grid((uint64_t)a.R * ARGUS_RS_WIDTH, kScThreads, 1024)),
                     dim3(kScThreads), 0, s, a);
  for (int p = 0; p < passes; ++p) {
    hipLaunchKernelGGL(k_sc_hist, dim3(tiles), dim3(kScThreads), 0, s, a, p);
    hipLaunchKernelGGL(k_sc_scan_sums, dim3((uint32_t)L.scan_blocks), dim3(kScThreads), 0, s, a);
    hipLaunchKernelGGL(k_sc_scan_top, dim3(1), dim3(1024), 0, s, a, (uint32_t)L.scan_blocks);
    hipLaunchKernelGGL(k_sc_scan_apply, dim3((uint32_t)L.scan_blocks), dim3(kScThreads), 0, s, a);
    hipLaunchKernelGGL(k_sc_scatter, dim3(tiles), dim3(kScThreads), 0, s, a, p);
  }
  hipLaunchKernelGGL(k_sc_ordinal, dim3(sc_grid(io->max_instances, kScThreads, 4096)),
                     dim3(kScThreads), 0, s, a, (passes - 1) & 1);
  hipLaunchKernelGGL(k_sc_stats, dim3(sc_grid(io->max_instances, kScThreads, 4096)),
                     dim3(kScThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? ARGUS_OK : ARGUS_E_HIP;
}
