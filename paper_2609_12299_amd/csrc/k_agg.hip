// k_agg.hip -- per-region observed statistics and ambiguity counts, and the
// planning of the overlap events.
//
// Section 3.5 of the paper: a region's report holds measured durations and
// makes ambiguous attributions visible.  Statistics are taken
// over matched instances; unclosed, mismatched and self-nested instances are
// counted per region.  Per-block partial results live in LDS and are flushed
// once per block with global atomics (all integer: the result does not
// depend on the order).
#include "internal.h"

namespace argus {

constexpr uint32_t kAggLdsBytes = 96 * 1024;  // per-block statistics budget
constexpr uint32_t kStatBytes = 6 * 8 + 5 * 4;  // per region
constexpr uint32_t kHistBytes = 130 * 4;         // per region
constexpr uint32_t kHistLdsBytes = 152 * 1024;  // per-block budget of the histogram pass (160 KiB of LDS)
// Region statistics of one block, in this order in the per-block buffer:
// count, inclusive sum/min/max, exclusive sum/min/max, unclosed, mismatched as
// begin and as end, self-nested.
constexpr uint32_t kAggFields = 11;
constexpr uint64_t kAggPartBytes = 64ull << 20;  // per-block buffer budget

__device__ __forceinline__ uint32_t agg_parent(const argus_instance& x, const TileDesc* tiles,
                                               const uint32_t* op_parent) {
  uint32_t pf = x.parent;
  if (pf == kNoParent || !(pf & kParentPending)) return pf;
  const uint64_t t = pf & ~kParentPending;
  const TileDesc d = tiles[t];
  const uint32_t L = x.level - 1;
  if (x.level == 0 || L < d.op_lo || L - d.op_lo >= d.n_op) return kNoParent;  // not reached
  return op_parent[t * kMatchTile + (L - d.op_lo)];
}

struct AggArgs {
  const DevPlan* plan;
  argus_instance* inst;
  const uint64_t* excl;  // exclusive times (closed instances), accumulated in place
  const TileDesc* tiles;
  const uint32_t* op_parent;
  uint64_t* excl_out;  // NULL unless requested; then the same buffer as excl
  uint32_t* hist_key;  // NULL when histograms are done here
  uint64_t* part;      // [block][kAggFields][R], or NULL: flush with atomics
  uint64_t* counters;
  uint64_t* rstats;
  uint32_t R;
  uint32_t lds_regions;  // R if statistics fit in LDS, else 0
  uint32_t hist_lds;     // histograms in LDS too
  // overlap events (K > 0): digit histograms of the events' sort keys
  const uint8_t* region_class;
  uint32_t K, G, shift;
  uint32_t* ev_hist;  // [12][256]
  DevPlan* wplan;
};

template <typename T>
__device__ __forceinline__ T wsum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Adds this wave's digits (lanes in `valid`) to an LDS histogram: one atomic
// when every valid lane holds the same digit (high digits of nearby
// timestamps, groups of one context), else one per lane (low digits, which
// rarely collide).
__device__ __forceinline__ void whist(uint32_t* hist, uint32_t d, bool valid) {
  const uint64_t vm = __ballot(valid);
  if (vm == 0) return;
  const int first = __ffsll((long long)vm) - 1;
  const uint32_t d0 = __shfl(d, first);
  const uint64_t same = __ballot(valid && d == d0);
  if (same == vm) {
    if ((int)lane_id() == first) atomicAdd(&hist[d0], (uint32_t)__popcll(vm));
    return;
  }
  if (valid) atomicAdd(&hist[d], 1u);
}

// Four waves per SIMD (two blocks per compute unit): the registers and the
// dynamic LDS of a block are sized for that.
__global__ __launch_bounds__(512, 4) void k_agg(AggArgs a) {
  extern __shared__ __align__(16) uint8_t smem[];
  const uint32_t RL = a.lds_regions;
  uint64_t* s_isum = (uint64_t*)smem;
  uint64_t* s_esum = s_isum + RL;
  uint64_t* s_imin = s_esum + RL;
  uint64_t* s_imax = s_imin + RL;
  uint64_t* s_emin = s_imax + RL;
  uint64_t* s_emax = s_emin + RL;
  uint32_t* s_cnt = (uint32_t*)(s_emax + RL);
  uint32_t* s_unc = s_cnt + RL;
  uint32_t* s_mab = s_unc + RL;
  uint32_t* s_mae = s_mab + RL;
  uint32_t* s_sn = s_mae + RL;
  uint32_t* s_hist = s_sn + RL;  // [RL][130] when hist_lds
  uint32_t* s_evh = s_hist + (a.hist_lds ? RL * 130 : 0);  // [12][256] when K > 0
  constexpr uint32_t NT = 512;
  for (uint32_t r = threadIdx.x; r < RL; r += NT) {
    s_isum[r] = 0;
    s_esum[r] = 0;
    s_imin[r] = kU64Max;
    s_imax[r] = 0;
    s_emin[r] = kU64Max;
    s_emax[r] = 0;
    s_cnt[r] = 0;
    s_unc[r] = 0;
    s_mab[r] = 0;
    s_mae[r] = 0;
    s_sn[r] = 0;
  }
  if (a.hist_lds)
    for (uint32_t i = threadIdx.x; i < RL * 130; i += NT) s_hist[i] = 0;
  // Events for the radix sort only: the merge path needs no histograms.
  const bool evk = a.K && !a.plan->ev_merge;
  if (evk)
    for (uint32_t i = threadIdx.x; i < kDigitPositions * kRadixBins; i += NT) s_evh[i] = 0;
  __syncthreads();

  const uint64_t nb = a.plan->n_begin;
  // Overlap-event digits that can vary: group digits below the width of
  // G - 1, timestamp digits above which ts_min and ts_max differ.
  uint32_t vary = 0;
  if (evk) {
    const uint64_t ts_lo = a.plan->rec.ts_min;
    const uint64_t ts_hi = ts_lo + a.plan->rec.ts_mask;
    const bool full_ts = a.plan->rec.ts_bits >= 64 || ts_hi < ts_lo;
    for (int d = 0; d < 4; ++d)
      if (d == 0 || ((uint64_t)(a.G - 1) >> (8 * d)) != 0) vary |= 1u << d;
    for (int d = 0; d < 8; ++d)
      if (full_ts || (ts_lo >> (8 * d)) != (ts_hi >> (8 * d))) vary |= 1u << (4 + d);
  }
  uint64_t n_m = 0, n_mm = 0, n_u = 0, n_sn = 0, n_ev = 0, n_skip = 0;
  unsigned long long* rs = (unsigned long long*)a.rstats;
  // Each wave takes 2 x 64 consecutive instances per step, with their loads
  // (and then the parents' regions) in flight together, and the next step's
  // loads issued before this step's statistics; every lane of a wave
  // iterates the same number of times (the event histograms use ballots).
  constexpr int B = 2;
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t stride = (uint64_t)gridDim.x * NT * B;
  const uint64_t wfirst = ((uint64_t)blockIdx.x * (NT / 64) + (threadIdx.x >> 6)) * (64 * B);
  argus_instance pxs[B];
  uint64_t pcs[B];
  auto issue = [&](uint64_t wbs) {
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const uint64_t id = wbs + (uint64_t)j * 64 + lane;
      const uint64_t ic = id < nb ? id : nb - 1;
      pxs[j] = a.inst[ic];
      pcs[j] = a.excl[ic];
    }
  };
  if (wfirst < nb) issue(wfirst);
  for (uint64_t wb = wfirst; wb < nb; wb += stride) {
    argus_instance xs[B];
    uint64_t cs[B];
    uint32_t par[B];
    uint16_t preg[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      xs[j] = pxs[j];
      cs[j] = pcs[j];
    }
    // Parents in earlier tiles (agg_parent's reading), the instances'
    // loads issued together at each of two steps: tile bounds, then the
    // enclosing-instance entry.  A lane without such a parent reads tile 0
    // and entry 0, which exist whenever the loop runs, and drops the value.
    uint32_t olo[B], nop[B], opv[B];
    bool pend[B], inr[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const uint32_t pf = xs[j].parent;
      pend[j] = pf != kNoParent && (pf & kParentPending) != 0;
      const uint64_t t = pend[j] ? (pf & ~kParentPending) : 0;
      olo[j] = a.tiles[t].op_lo;
      nop[j] = a.tiles[t].n_op;
    }
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const uint32_t pf = xs[j].parent;
      const uint64_t t = pend[j] ? (pf & ~kParentPending) : 0;
      const uint32_t L = xs[j].level - 1;
      inr[j] = pend[j] & (xs[j].level != 0) & (L >= olo[j]) & (L - olo[j] < nop[j]);
      opv[j] = a.op_parent[inr[j] ? t * kMatchTile + (L - olo[j]) : 0];
    }
#pragma unroll
    for (int j = 0; j < B; ++j) {
      par[j] = !pend[j] ? xs[j].parent : (inr[j] ? opv[j] : kNoParent);
      if (par[j] != kNoParent && par[j] >= nb) {
        flag_internal_error(a.counters, 4);
        par[j] = kNoParent;
      }
    }
    // the parents' regions and, with overlap events, the instances' classes
    // (loaded together, before the first is used)
    uint32_t rcl[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const bool matched = xs[j].end_region_id != kNoEnd && xs[j].end_region_id == xs[j].region_id;
      preg[j] = (matched && par[j] != kNoParent) ? a.inst[par[j]].region_id : (uint16_t)kNoEnd;
    }
    if (a.K) {
#pragma unroll
      for (int j = 0; j < B; ++j) {
        const uint32_t rg = xs[j].region_id;
        rcl[j] = a.region_class[rg < a.R ? rg : 0u];
      }
    }
    // the next step's loads, issued after this step's dependent loads
    if (wb + stride < nb) issue(wb + stride);
#pragma unroll
    for (int j = 0; j < B; ++j) {
    const uint64_t id = wb + (uint64_t)j * 64 + lane;
    bool ev = false;
    uint64_t eg = 0, et0 = 0, et1 = 0;
    if (id < nb) {
    const argus_instance& x = xs[j];
    if (par[j] != x.parent) a.inst[id].parent = par[j];
    const uint32_t region = x.region_id, ereg = x.end_region_id;
    const bool closed = ereg != kNoEnd;
    const bool matched = closed && ereg == region;
    const uint64_t incl = closed ? x.t_end - x.t_begin : 0;
    const uint64_t excl = closed ? cs[j] : 0;
    // the output holds the closed instances' exclusive times already
    if (a.excl_out && !closed) a.excl_out[id] = 0;
    uint32_t hk = 0xFFFFFFFFu;
    if (matched) {
      n_m++;
      if (a.K) {
        const uint32_t cls = rcl[j];
        if (cls < a.K) {
          eg = a.shift >= 32 ? 0 : (x.ctx_key >> a.shift);
          if (eg < a.G) {
            ev = true;
            et0 = x.t_begin;
            et1 = x.t_end;
            n_ev += 2;
          } else {
            n_skip++;
          }
        }
      }
      const bool sn = preg[j] == region;
      n_sn += sn;
      const uint32_t bi = bit_width64(incl), be = bit_width64(excl);
      hk = (region << 16) | (bi << 8) | be;
      if (RL) {
        atomicAdd(&s_cnt[region], 1u);
        atomicAdd((unsigned long long*)&s_isum[region], (unsigned long long)incl);
        atomicAdd((unsigned long long*)&s_esum[region], (unsigned long long)excl);
        atomicMin((unsigned long long*)&s_imin[region], (unsigned long long)incl);
        atomicMax((unsigned long long*)&s_imax[region], (unsigned long long)incl);
        atomicMin((unsigned long long*)&s_emin[region], (unsigned long long)excl);
        atomicMax((unsigned long long*)&s_emax[region], (unsigned long long)excl);
        if (sn) atomicAdd(&s_sn[region], 1u);
        if (a.hist_lds) {
          atomicAdd(&s_hist[region * 130 + bi], 1u);
          atomicAdd(&s_hist[region * 130 + 65 + be], 1u);
        }
      } else {
        unsigned long long* row = rs + (uint64_t)region * ARGUS_RS_WIDTH;
        atomicAdd(&row[ARGUS_RS_COUNT], 1ull);
        atomicAdd(&row[ARGUS_RS_INCL_SUM], (unsigned long long)incl);
        atomicAdd(&row[ARGUS_RS_EXCL_SUM], (unsigned long long)excl);
        atomicMin(&row[ARGUS_RS_INCL_MIN], (unsigned long long)incl);
        atomicMax(&row[ARGUS_RS_INCL_MAX], (unsigned long long)incl);
        atomicMin(&row[ARGUS_RS_EXCL_MIN], (unsigned long long)excl);
        atomicMax(&row[ARGUS_RS_EXCL_MAX], (unsigned long long)excl);
        if (sn) atomicAdd(&row[ARGUS_RS_SELF_NESTED], 1ull);
      }
    } else if (closed) {
      n_mm++;
      if (RL) {
        atomicAdd(&s_mab[region], 1u);
        atomicAdd(&s_mae[ereg], 1u);
      } else {
        atomicAdd(&rs[(uint64_t)region * ARGUS_RS_WIDTH + ARGUS_RS_MISM_AS_BEGIN], 1ull);
        atomicAdd(&rs[(uint64_t)ereg * ARGUS_RS_WIDTH + ARGUS_RS_MISM_AS_END], 1ull);
      }
    } else {
      n_u++;
      if (RL) atomicAdd(&s_unc[region], 1u);
      else atomicAdd(&rs[(uint64_t)region * ARGUS_RS_WIDTH + ARGUS_RS_UNCLOSED], 1ull);
    }
    if (a.hist_key) a.hist_key[id] = hk;
    }
    if (evk) {
#pragma unroll
      for (int d = 0; d < 4; ++d)
        if ((vary >> d) & 1u) {
          const uint32_t dg = (uint32_t)(eg >> (8 * d)) & 0xFFu;
          whist(s_evh + d * kRadixBins, dg, ev);
          whist(s_evh + d * kRadixBins, dg, ev);
        }
#pragma unroll
      for (int d = 0; d < 8; ++d)
        if ((vary >> (4 + d)) & 1u) {
          whist(s_evh + (4 + d) * kRadixBins, (uint32_t)(et0 >> (8 * d)) & 0xFFu, ev);
          whist(s_evh + (4 + d) * kRadixBins, (uint32_t)(et1 >> (8 * d)) & 0xFFu, ev);
        }
    }
  }  // j
  }

  n_m = wsum(n_m);
  n_mm = wsum(n_mm);
  n_u = wsum(n_u);
  n_sn = wsum(n_sn);
  n_ev = wsum(n_ev);
  n_skip = wsum(n_skip);
  __syncthreads();  // every wave's LDS adds are done
  if (evk)
    for (uint32_t i = threadIdx.x; i < kDigitPositions * kRadixBins; i += NT)
      if (s_evh[i]) atomicAdd(&a.ev_hist[i], s_evh[i]);
  if (a.part) {
    // plain stores; k_agg_reduce combines the blocks (many blocks adding
    // into the same rows with atomics serialise on them)
    uint64_t* pb = a.part + (uint64_t)blockIdx.x * kAggFields * RL;
    for (uint32_t r = threadIdx.x; r < RL; r += NT) {
      pb[0 * RL + r] = s_cnt[r];
      pb[1 * RL + r] = s_isum[r];
      pb[2 * RL + r] = s_imin[r];
      pb[3 * RL + r] = s_imax[r];
      pb[4 * RL + r] = s_esum[r];
      pb[5 * RL + r] = s_emin[r];
      pb[6 * RL + r] = s_emax[r];
      pb[7 * RL + r] = s_unc[r];
      pb[8 * RL + r] = s_mab[r];
      pb[9 * RL + r] = s_mae[r];
      pb[10 * RL + r] = s_sn[r];
    }
  } else {
    for (uint32_t r = threadIdx.x; r < RL; r += NT) {
      unsigned long long* row = rs + (uint64_t)r * ARGUS_RS_WIDTH;
      if (s_cnt[r]) {
        atomicAdd(&row[ARGUS_RS_COUNT], (unsigned long long)s_cnt[r]);
        atomicAdd(&row[ARGUS_RS_INCL_SUM], (unsigned long long)s_isum[r]);
        atomicAdd(&row[ARGUS_RS_EXCL_SUM], (unsigned long long)s_esum[r]);
        atomicMin(&row[ARGUS_RS_INCL_MIN], (unsigned long long)s_imin[r]);
        atomicMax(&row[ARGUS_RS_INCL_MAX], (unsigned long long)s_imax[r]);
        atomicMin(&row[ARGUS_RS_EXCL_MIN], (unsigned long long)s_emin[r]);
        atomicMax(&row[ARGUS_RS_EXCL_MAX], (unsigned long long)s_emax[r]);
      }
      if (s_unc[r]) atomicAdd(&row[ARGUS_RS_UNCLOSED], (unsigned long long)s_unc[r]);
      if (s_mab[r]) atomicAdd(&row[ARGUS_RS_MISM_AS_BEGIN], (unsigned long long)s_mab[r]);
      if (s_mae[r]) atomicAdd(&row[ARGUS_RS_MISM_AS_END], (unsigned long long)s_mae[r]);
      if (s_sn[r]) atomicAdd(&row[ARGUS_RS_SELF_NESTED], (unsigned long long)s_sn[r]);
    }
  }
  if (a.hist_lds) {
    for (uint32_t i = threadIdx.x; i < RL * 130; i += NT) {
      const uint32_t h = s_hist[i];
      if (h) {
        const uint32_t r = i / 130, b = i % 130;
        atomicAdd(&rs[(uint64_t)r * ARGUS_RS_WIDTH + ARGUS_RS_HIST_INCL + b], (unsigned long long)h);
      }
    }
  }
  // the counters, per block, through the start of the (now read) LDS area
  // (static LDS would keep two blocks from sharing a compute unit)
  __syncthreads();
  uint64_t* s_red = (uint64_t*)smem;  // [8][6]
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    s_red[w * 6 + 0] = n_m;
    s_red[w * 6 + 1] = n_mm;
    s_red[w * 6 + 2] = n_u;
    s_red[w * 6 + 3] = n_sn;
    s_red[w * 6 + 4] = n_skip;
    s_red[w * 6 + 5] = n_ev;
  }
  __syncthreads();
  if (threadIdx.x < 6) {
    uint64_t v = 0;
    for (int q = 0; q < (int)(NT / 64); ++q) v += s_red[q * 6 + threadIdx.x];
    const int idx = threadIdx.x == 0   ? ARGUS_C_N_MATCHED
                    : threadIdx.x == 1 ? ARGUS_C_N_MISMATCHED
                    : threadIdx.x == 2 ? ARGUS_C_N_UNCLOSED
                    : threadIdx.x == 3 ? ARGUS_C_N_SELF_NESTED
                                       : ARGUS_C_N_OVERLAP_SKIPPED;
    if (v && threadIdx.x < 5) atomicAdd((unsigned long long*)&a.counters[idx], (unsigned long long)v);
    if (v && threadIdx.x == 5 && evk) atomicAdd((unsigned long long*)&a.wplan->n_ev, (unsigned long long)v);
  }
}

static void agg_sizes(uint32_t R, uint32_t* rl, uint32_t* hist_lds, size_t* bytes) {
  if ((uint64_t)R * (kStatBytes + kHistBytes) <= kAggLdsBytes) {
    *rl = R;
    *hist_lds = 1;
    *bytes = (size_t)R * (kStatBytes + kHistBytes);
  } else if ((uint64_t)R * kStatBytes <= kAggLdsBytes) {
    *rl = R;
    *hist_lds = 0;
    *bytes = (size_t)R * kStatBytes;
  } else {
    *rl = 0;
    *hist_lds = 0;
    *bytes = 0;
  }
}

static uint64_t agg_grid(uint64_t n) {
  const uint64_t blocks = ceil_div(n ? n : 1, 512 * 16);
  return blocks > 512 ? 512 : blocks;
}

uint64_t agg_part_words(uint64_t n, uint32_t R) {
  uint32_t rl, hl;
  size_t bytes;
  agg_sizes(R, &rl, &hl, &bytes);
  if (!rl) return 0;
  const uint64_t words = agg_grid(n) * kAggFields * rl;
  return words * sizeof(uint64_t) <= kAggPartBytes ? words : 0;
}

// Combines the per-block statistics of k_agg into the region rows: one
// thread per (field, region) and run of kAggRun blocks (reads coalesced over
// regions), then one atomic per thread.
constexpr uint32_t kAggRun = 32;
__global__ __launch_bounds__(256) void k_agg_reduce(const uint64_t* part, uint32_t nblk, uint32_t R,
                                                    uint64_t* rstats) {
  const uint32_t idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= kAggFields * R) return;
  const uint32_t f = idx / R, r = idx - f * R;
  const bool is_min = f == 2 || f == 5, is_max = f == 3 || f == 6;
  const uint32_t b0 = blockIdx.y * kAggRun, b1 = b0 + kAggRun < nblk ? b0 + kAggRun : nblk;
  uint64_t v = is_min ? kU64Max : 0;
#pragma unroll 8
  for (uint32_t b = b0; b < b1; ++b) {
    const uint64_t x = part[((uint64_t)b * kAggFields + f) * R + r];
    v = is_min ? (x < v ? x : v) : is_max ? (x > v ? x : v) : v + x;
  }
  if (v == (is_min ? kU64Max : 0)) return;
  constexpr int col[kAggFields] = {ARGUS_RS_COUNT,      ARGUS_RS_INCL_SUM,      ARGUS_RS_INCL_MIN,
                                   ARGUS_RS_INCL_MAX,   ARGUS_RS_EXCL_SUM,      ARGUS_RS_EXCL_MIN,
                                   ARGUS_RS_EXCL_MAX,   ARGUS_RS_UNCLOSED,      ARGUS_RS_MISM_AS_BEGIN,
                                   ARGUS_RS_MISM_AS_END, ARGUS_RS_SELF_NESTED};
  unsigned long long* dst = (unsigned long long*)(rstats + (uint64_t)r * ARGUS_RS_WIDTH + col[f]);
  if (is_min)
    atomicMin(dst, (unsigned long long)v);
  else if (is_max)
    atomicMax(dst, (unsigned long long)v);
  else
    atomicAdd(dst, (unsigned long long)v);
}

hipError_t launch_agg(const RunArgs& a, hipStream_t s) {
  uint32_t rl, hl;
  size_t bytes;
  agg_sizes(a.R, &rl, &hl, &bytes);
  if (a.K) bytes += sizeof(uint32_t) * kDigitPositions * kRadixBins;
  if (bytes < 8 * 6 * sizeof(uint64_t)) bytes = 8 * 6 * sizeof(uint64_t);  // the counter sums at the end
  AggArgs g{};
  g.plan = a.w.plan;
  g.inst = a.w.inst;
  g.excl = a.w.excl;
  g.tiles = a.w.tiles;
  g.op_parent = a.w.op_parent;
  g.excl_out = (a.flags & ARGUS_OUT_INSTANCE_EXCL) ? a.out.d_instance_excl : nullptr;
  g.hist_key = hl ? nullptr : a.w.hist_key;
  g.counters = a.out.d_counters;
  g.rstats = a.out.d_region_stats;
  g.R = a.R;
  g.lds_regions = rl;
  g.hist_lds = hl;
  g.region_class = a.region_class;
  g.K = a.K;
  g.G = a.G;
  g.shift = a.shift;
  g.ev_hist = a.w.ev_hist;
  g.wplan = a.w.plan;
  g.part = a.w.agg_part;
  const uint64_t blocks = agg_grid(a.n);
  if (bytes > 64 * 1024)
    (void)hipFuncSetAttribute((const void*)k_agg, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  hipLaunchKernelGGL(k_agg, dim3((uint32_t)blocks), dim3(512), bytes, s, g);
  if (g.part) {
    const uint32_t threads = kAggFields * rl;
    hipLaunchKernelGGL(k_agg_reduce, dim3(ceil_div(threads, 256), ceil_div(blocks, kAggRun)), dim3(256), 0, s,
                       (const uint64_t*)g.part, (uint32_t)blocks, rl, a.out.d_region_stats);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------ histograms

struct HistArgs {
  const uint64_t* count;  // keys (device), at most count_max
  uint64_t count_max;
  const uint32_t* hist_key;
  uint64_t* rstats;
  uint32_t R;
  uint32_t slice;   // regions per slice
  uint32_t slices;
  uint32_t ranges;  // key ranges (a multiple of 8)
};

// Log2 histograms when they do not fit next to the statistics: each block
// covers one slice of regions in LDS over one range of the keys.  Blocks are
// numbered so that the slices of one key range are 8 apart: dispatched to
// the same XCD at about the same time, they read the keys once from HBM and
// otherwise from that XCD's L2.
__global__ __launch_bounds__(1024) void k_hist(HistArgs a) {
  extern __shared__ __align__(16) uint8_t smem[];
  constexpr uint32_t NT = 1024;
  uint32_t* s_h = (uint32_t*)smem;
  const uint32_t b = blockIdx.x, grp = b / (8 * a.slices), rem = b % (8 * a.slices);
  const uint32_t range = grp * 8 + rem % 8, sl = rem / 8;
  if (range >= a.ranges || sl * a.slice >= a.R) return;
  const uint32_t r0 = sl * a.slice;
  const uint32_t r1 = r0 + a.slice < a.R ? r0 + a.slice : a.R;
  const uint32_t nr = r1 - r0;
  for (uint32_t i = threadIdx.x; i < nr * 130; i += NT) s_h[i] = 0;
  __syncthreads();
  const uint64_t nb = *a.count < a.count_max ? *a.count : a.count_max;
  auto add = [&](uint32_t k) {
    const uint32_t r = k >> 16;
    if (k == 0xFFFFFFFFu || r < r0 || r >= r1) return;
    atomicAdd(&s_h[(r - r0) * 130 + ((k >> 8) & 0xFFu)], 1u);
    atomicAdd(&s_h[(r - r0) * 130 + 65 + (k & 0xFFu)], 1u);
  };
  // four keys per load (the key array is 256-byte aligned)
  const uint64_t n4 = nb / 4;
  const uint4* k4 = (const uint4*)a.hist_key;
  // eight loads per thread in flight
  const uint64_t stride = (uint64_t)a.ranges * NT;
  uint64_t q = (uint64_t)range * NT + threadIdx.x;
  for (; q + 7 * stride < n4; q += 8 * stride) {
    uint4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = k4[q + u * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      add(v[u].x);
      add(v[u].y);
      add(v[u].z);
      add(v[u].w);
    }
  }
  for (; q < n4; q += stride) {
    const uint4 v = k4[q];
    add(v.x);
    add(v.y);
    add(v.z);
    add(v.w);
  }
  if (range == 0 && threadIdx.x < nb - n4 * 4) add(a.hist_key[n4 * 4 + threadIdx.x]);
  __syncthreads();
  unsigned long long* rs = (unsigned long long*)a.rstats;
  for (uint32_t i = threadIdx.x; i < nr * 130; i += NT) {
    const uint32_t h = s_h[i];
    if (h) {
      const uint32_t r = r0 + i / 130, b = i % 130;
      atomicAdd(&rs[(uint64_t)r * ARGUS_RS_WIDTH + ARGUS_RS_HIST_INCL + b], (unsigned long long)h);
    }
  }
}

hipError_t launch_hist_keys(const uint32_t* keys, const uint64_t* d_count, uint64_t count_max,
                            uint64_t* rstats, uint32_t R, hipStream_t s) {
  // as few slices as fit, of equal size
  const uint32_t slices = (uint32_t)ceil_div((uint64_t)R * kHistBytes, kHistLdsBytes);
  const uint32_t slice = (uint32_t)ceil_div(R, slices);
  uint64_t ranges = ceil_div(count_max ? count_max : 1, 1024 * 64);
  if (ranges > 256) ranges = 256;
  ranges = ceil_div(ranges, 8) * 8;
  HistArgs h{d_count, count_max, keys, rstats, R, slice, slices, (uint32_t)ranges};
  const size_t hb = (size_t)slice * kHistBytes;
  (void)hipFuncSetAttribute((const void*)k_hist, hipFuncAttributeMaxDynamicSharedMemorySize, (int)hb);
  hipLaunchKernelGGL(k_hist, dim3((uint32_t)(ranges * slices)), dim3(1024), hb, s, h);
  return hipGetLastError();
}

hipError_t launch_hist(const RunArgs& a, hipStream_t s) {
  uint32_t rl, hl;
  size_t bytes;
  agg_sizes(a.R, &rl, &hl, &bytes);
  if (hl) return hipSuccess;
  return launch_hist_keys(a.w.hist_key, &a.w.plan->n_begin, a.n, a.out.d_region_stats, a.R, s);
}

// ------------------------------------------------------- overlap events

struct EvPlanArgs {
  DevPlan* plan;
  const uint32_t* hist;
  uint32_t* off;
  uint32_t G;
};

__global__ __launch_bounds__(256) void k_ev_plan(EvPlanArgs a) {
  __shared__ uint32_t s_scr[4];
  __shared__ uint32_t s_active[kDigitPositions];
  DevPlan* p = a.plan;
  const int t = threadIdx.x;
  if (p->ev_merge) return;  // events are merged, not sorted (all slots stay inactive)
  for (int pos = 0; pos < kDigitPositions; ++pos) {
    const uint32_t h = a.hist[pos * kRadixBins + t];
    const int used = __syncthreads_count(h != 0);
    uint32_t x = h;
    const int lane = t & 63, w = t >> 6;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      uint32_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) s_scr[w] = x;
    __syncthreads();
    uint32_t pre = 0;
    for (int k = 0; k < w; ++k) pre += s_scr[k];
    a.off[pos * kRadixBins + t] = pre + x - h;
    if (t == 0) s_active[pos] = used > 1;
    __syncthreads();
  }
  if (t != 0) return;
  KeySpace k = p->rec;
  k.ctx_min = 0;
  k.ctx_bits = bit_width64(a.G > 0 ? a.G - 1 : 0);
  k.wide = (k.ts_bits + k.ctx_bits > 64) ? 1u : 0u;
  p->ev = k;
  p->ev_slots = 2 * p->n_begin;
  // LSD order: timestamp digits, then group digits.
  uint32_t nact = 0;
  for (int pos = 0; pos < kDigitPositions; ++pos) nact += s_active[pos];
  uint32_t j = 0;
  for (int sl = 0; sl < kSlots; ++sl) {
    SlotPlan& sp = p->es[sl];
    sp.active = 0;
    if (sl >= 12) continue;
    const uint32_t pos = sl < 8 ? (uint32_t)(4 + sl) : (uint32_t)(sl - 8);
    sp.pos = pos;
    const bool act = s_active[pos] || (nact == 0 && sl == 0 && p->n_ev > 0);
    if (!act) continue;
    sp.active = 1;
    sp.src = j == 0 ? 2u : ((j - 1) & 1u);
    sp.dst = j & 1u;
    sp.lb = j & 1u;
    sp.n_elems = j == 0 ? p->ev_slots : p->n_ev;
    sp.n_out = (uint32_t)p->n_ev;
    sp.tiles = ceil_div(sp.n_elems, kSortTile);
    p->ev_final = sp.dst;
    ++j;
  }
}

hipError_t launch_ev_plan(const RunArgs& a, hipStream_t s) {
  EvPlanArgs e{a.w.plan, a.w.ev_hist, a.w.ev_off, a.G};
  hipLaunchKernelGGL(k_ev_plan, dim3(1), dim3(256), 0, s, e);
  return hipGetLastError();
}

struct EvClearArgs {
  const DevPlan* plan;
  uint64_t* lb0;
};

// Clears the look-back status the first event pass uses.
__global__ __launch_bounds__(256) void k_ev_clear(EvClearArgs a) {
  if (a.plan->ev_merge) return;
  const uint64_t words = ceil_div(a.plan->ev_slots, kSortTile) * kRadixBins;
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < words; i += stride) a.lb0[i] = 0;
}

hipError_t launch_ev_clear(const RunArgs& a, hipStream_t s) {
  EvClearArgs e{a.w.plan, a.w.lb[0]};
  uint64_t blocks = ceil_div(ceil_div(2 * (a.n ? a.n : 1), kSortTile) * kRadixBins, 256 * 4);
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_ev_clear, dim3((uint32_t)blocks), dim3(256), 0, s, e);
  return hipGetLastError();
}

}  // namespace argus
