// k_radix.hip -- one stable LSD radix pass over 8-bit digits.
//
// Stable sorting is how the records of every execution context are put in
// execution order before the per-context stack is replayed (the paper's
// Section 3.2 keeps a stack of open regions for each warp); the same
// pass orders the overlap events by (group, time).
//
// One pass, per tile of 4096 elements (4 waves x 16 rounds x 64 lanes):
//   * rank: each wave finds, with eight ballots, the lanes holding the same
//     digit and counts them in per-wave LDS digit counters (stable order is
//     wave, round, lane = element order);
//   * the tile's 256 digit counts are published for decoupled look-back
//     (Merrill & Garland 2016) with tile ids taken in launch order from an
//     atomic counter, so every predecessor tile is already running;
//   * elements are staged in LDS in digit order and written out so that a
//     run of equal digits goes to consecutive addresses.
// The first pass of a sort reads its raw source (records or instances),
// drops invalid elements (they are never written) and packs the key.
#include "internal.h"

namespace argus {

struct RadixArgs {
  const DevPlan* plan;
  int which;  // 0: records, 1: overlap events
  int slot;
  const uint4* rec;
  const argus_instance* inst;
  const uint8_t* region_class;
  uint32_t R, K, G, shift;
  uint64_t* key[2];
  uint32_t* pay[2];
  uint32_t* ctxw[2];
  uint64_t* lb[2];
  const uint32_t* off;  // [12][256] exclusive digit offsets
  uint32_t* tile_ctr;
  uint64_t* counters;
};

__device__ __forceinline__ uint32_t digit_of(uint32_t pos, uint64_t raw_ctx, uint64_t raw_ts) {
  return pos < 4 ? (uint32_t)(raw_ctx >> (8 * pos)) & 0xFFu
                 : (uint32_t)(raw_ts >> (8 * (pos - 4))) & 0xFFu;
}

// WHICH (records / events) and SLOT are template parameters so that every
// pass of a sort is a distinct kernel in profiles.
template <int WHICH, int SLOT>
__global__ __launch_bounds__(kSortThreads) void k_radix_pass(RadixArgs a) {
  const SlotPlan sp = WHICH ? a.plan->es[SLOT] : a.plan->rs[SLOT];
  if (!sp.active) return;
  const KeySpace ks = WHICH ? a.plan->ev : a.plan->rec;

  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_wave[4][kRadixBins];  // per-wave counts, then wave prefixes
  __shared__ uint32_t s_start[kRadixBins];    // tile-local start of each digit
  __shared__ uint32_t s_gbase[kRadixBins];    // global start of this tile's digit run
  __shared__ uint32_t s_scr[4];
  __shared__ uint32_t s_total;
  __shared__ uint64_t s_key[kSortTile];
  __shared__ uint32_t s_pay[kSortTile];
  __shared__ uint32_t s_cw[kSortTile];
  __shared__ uint8_t s_dig[kSortTile];

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  // Persistent blocks: tiles are taken in order from an atomic counter, so a
  // tile's predecessors always belong to blocks that are already running.
  for (;;) {
  if (tid == 0) s_tile = atomicAdd(&a.tile_ctr[(WHICH ? kCtrEv : kCtrRec) + SLOT], 1u);
  for (int i = tid; i < 4 * kRadixBins; i += kSortThreads) (&s_wave[0][0])[i] = 0;
  __syncthreads();
  const uint64_t tile = s_tile;
  if (tile >= sp.tiles) break;

  const uint64_t base = tile * kSortTile;
  const uint64_t left = sp.n_elems - base;
  const uint32_t cnt = left < (uint64_t)kSortTile ? (uint32_t)left : (uint32_t)kSortTile;
  const bool wide = ks.wide != 0;
  const uint32_t pos = sp.pos;

  uint64_t key[kSortItems];
  uint32_t pay[kSortItems], cw[kSortItems], dig[kSortItems], rank[kSortItems];

  // Loads first, all of them unconditional (an index past the tile's end is
  // clamped to its last element, whose digit is then discarded), so that
  // every load of the tile is in flight before the first one is used.
  auto elem = [&](int r) -> uint32_t {
    return (uint32_t)w * (kSortItems * 64) + (uint32_t)r * 64 + lane;
  };
  auto clamp = [&](uint32_t el) -> uint64_t { return base + (el < cnt ? el : cnt - 1); };
  if (sp.src < 2) {
    const uint64_t* ksrc = sp.src ? a.key[1] : a.key[0];
    const uint32_t* psrc = sp.src ? a.pay[1] : a.pay[0];
    const uint32_t* csrc = sp.src ? a.ctxw[1] : a.ctxw[0];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      const uint64_t e = clamp(elem(r));
      key[r] = ksrc[e];
      pay[r] = psrc[e];
      cw[r] = wide ? csrc[e] : 0u;
    }
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      uint64_t ctx_rel, ts_off;
      if (wide) {
        ctx_rel = cw[r];
        ts_off = key[r];
      } else {
        ctx_rel = ks.ts_bits >= 64 ? 0 : (key[r] >> ks.ts_bits);
        ts_off = key[r] & ks.ts_mask;
      }
      dig[r] = elem(r) < cnt ? digit_of(pos, ks.ctx_min + ctx_rel, ks.ts_min + ts_off) : 256u;
    }
  } else if (WHICH == 0) {
    uint4 rr[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) rr[r] = a.rec[clamp(elem(r))];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      // branch-free, so that the whole 16-byte record is loaded up front
      const uint64_t ts = (uint64_t)rr[r].x | ((uint64_t)rr[r].y << 32);
      const uint32_t ctx = rr[r].z;
      const uint32_t region = rr[r].w & 0xFFFFu;
      const uint32_t kind = (rr[r].w >> 16) & 0xFFu;
      const bool ok = elem(r) < cnt && (kind == 1 || kind == 2) && region < a.R;
      const uint64_t ts_off = ts - ks.ts_min;
      const uint64_t ctx_rel = (uint64_t)ctx - ks.ctx_min;
      const uint64_t k = wide ? ts_off : ((ks.ts_bits >= 64 ? 0 : (ctx_rel << ks.ts_bits)) | ts_off);
      key[r] = ok ? k : 0;
      cw[r] = ok ? (uint32_t)ctx_rel : 0u;
      const uint32_t cls = ok && swept_ctx(ctx, a.K, a.G, a.shift) ? a.region_class[region] : 0xFFu;
      pay[r] = ok ? pack_payload(region, kind, cls) : 0u;
      dig[r] = ok ? digit_of(pos, ctx, ts) : 256u;  // 256: invalid (never written)
    }
  } else {
    // Overlap events: element e is the begin (even) or end (odd) of instance
    // e / 2; only matched, classified instances of a group < G.
    uint64_t tv[kSortItems];
    uint32_t cv[kSortItems], rv[kSortItems], cl[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      const uint64_t e = clamp(elem(r));
      const argus_instance* ip = a.inst + (e >> 1);
      tv[r] = (e & 1) ? ip->t_end : ip->t_begin;
      cv[r] = ip->ctx_key;
      rv[r] = *(const uint32_t*)&ip->region_id;  // region | end_region << 16
    }
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) cl[r] = a.region_class[rv[r] & 0xFFFFu];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      uint32_t d = 256;
      const uint32_t el = elem(r);
      const uint32_t is_end = (uint32_t)((base + el) & 1);
      const uint32_t region = rv[r] & 0xFFFFu, eregion = rv[r] >> 16;
      const uint64_t g = a.shift >= 32 ? 0 : (cv[r] >> a.shift);
      key[r] = 0;
      pay[r] = 0;
      cw[r] = 0;
      if (el < cnt && region == eregion && cl[r] < a.K && g < a.G) {
        const uint64_t ts_off = tv[r] - ks.ts_min;
        key[r] = wide ? ts_off : ((ks.ts_bits >= 64 ? 0 : (g << ks.ts_bits)) | ts_off);
        cw[r] = (uint32_t)g;
        pay[r] = cl[r] | (is_end << 8);
        d = digit_of(pos, g, tv[r]);
      }
      dig[r] = d;
    }
  }
  // Rank among this wave's elements with the same digit (stable order is
  // wave, round, lane).  All loads above are already in flight.
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const uint32_t d = dig[r];
    const bool part = d < 256;
    const uint64_t vm = __ballot(part);
    uint64_t peers = vm;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint32_t bit = (d >> b) & 1u;
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    uint32_t rk = 0;
    if (part) {
      const uint32_t before = (uint32_t)__popcll(peers & lanemask_lt());
      const uint32_t old = s_wave[w][d];
      rk = old + before;
      __builtin_amdgcn_wave_barrier();
      if ((peers >> lane) == 1ull) s_wave[w][d] = old + (uint32_t)__popcll(peers);
    }
    __builtin_amdgcn_wave_barrier();
    rank[r] = rk;
  }
  __syncthreads();

  // Digit totals of the tile, per-wave prefixes and tile-local starts.
  const int dgt = tid;
  uint32_t c0 = s_wave[0][dgt], c1 = s_wave[1][dgt], c2 = s_wave[2][dgt], c3 = s_wave[3][dgt];
  const uint32_t tot = c0 + c1 + c2 + c3;
  uint32_t lane_total;
  {
    uint32_t x = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      uint32_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) s_scr[w] = x;
    __syncthreads();
    uint32_t pre = 0, all = 0;
    for (int k = 0; k < 4; ++k) {
      if (k < w) pre += s_scr[k];
      all += s_scr[k];
    }
    s_start[dgt] = pre + x - tot;
    lane_total = all;
  }
  s_wave[0][dgt] = 0;
  s_wave[1][dgt] = c0;
  s_wave[2][dgt] = c0 + c1;
  s_wave[3][dgt] = c0 + c1 + c2;
  if (tid == 0) s_total = lane_total;

  // Decoupled look-back on the count of this digit in earlier tiles.
  uint64_t* lb = a.lb[sp.lb];
  uint64_t excl = 0;
  if (tile == 0) {
    st_agent(&lb[dgt], kFlagIncl | tot);
  } else {
    st_agent(&lb[tile * kRadixBins + dgt], kFlagAgg | tot);
    // Four predecessors per round trip; consume them nearest first.
    int64_t tt = (int64_t)tile - 1;
    uint32_t spins = 0;
    bool done = false;
    while (!done && tt >= 0) {
      uint64_t v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        v[q] = tt - q >= 0 ? ld_agent(&lb[(uint64_t)(tt - q) * kRadixBins + dgt]) : kFlagIncl;
      int used = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (done || used != q) break;
        const uint64_t f = v[q] & ~kValMask;
        if (f == 0) break;  // not published yet: reload from here
        excl += v[q] & kValMask;
        ++used;
        if (f == kFlagIncl) done = true;
      }
      tt -= used;
      if (used == 0) {
        if (++spins > kMaxSpins) {
          flag_internal_error(a.counters, 1);
          break;
        }
        backoff();
      }
    }
    st_agent(&lb[tile * kRadixBins + dgt], kFlagIncl | (excl + tot));
  }
  s_gbase[dgt] = a.off[pos * kRadixBins + dgt] + (uint32_t)excl;
  // The other status array is the one the next pass uses: clear our slots.
  a.lb[sp.lb ^ 1u][tile * kRadixBins + dgt] = 0;
  __syncthreads();

  // Stage in LDS in digit order.
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const uint32_t d = dig[r];
    if (d < 256) {
      const uint32_t lp = s_start[d] + s_wave[w][d] + rank[r];
      s_key[lp] = key[r];
      s_pay[lp] = pay[r];
      s_cw[lp] = cw[r];
      s_dig[lp] = (uint8_t)d;
    }
  }
  __syncthreads();

  // Write out: consecutive staged elements of one digit go to consecutive
  // global positions.
  const uint32_t total = s_total;
  uint64_t* kd = a.key[sp.dst];
  uint32_t* pd = a.pay[sp.dst];
  uint32_t* cd = a.ctxw[sp.dst];
  const uint32_t n_out = sp.n_out;
  for (uint32_t i = tid; i < total; i += kSortThreads) {
    const uint32_t d = s_dig[i];
    const uint32_t gp = s_gbase[d] + (i - s_start[d]);
    if (gp >= n_out) {
      flag_internal_error(a.counters, 2);
      continue;
    }
    kd[gp] = s_key[i];
    pd[gp] = s_pay[i];
    if (wide) cd[gp] = s_cw[i];
  }
  __syncthreads();
  }  // tiles
}

hipError_t launch_radix_pass(const RunArgs& a, int which, int slot, uint64_t max_elems,
                             hipStream_t s) {
  RadixArgs ra{};
  ra.plan = a.w.plan;
  ra.which = which;
  ra.slot = slot;
  ra.rec = (const uint4*)a.rec;
  ra.inst = a.w.inst;
  ra.region_class = a.region_class;
  ra.R = a.R;
  ra.K = a.K;
  ra.G = a.G;
  ra.shift = a.shift;
  for (int b = 0; b < 2; ++b) {
    ra.key[b] = a.w.key[b];
    ra.pay[b] = a.w.pay[b];
    ra.ctxw[b] = a.w.ctxw[b];
    ra.lb[b] = a.w.lb[b];
  }
  ra.off = which ? a.w.ev_off : a.w.rec_off;
  ra.tile_ctr = a.w.tile_ctr;
  ra.counters = a.out.d_counters;
  uint64_t blocks = ceil_div(max_elems ? max_elems : 1, kSortTile);
  const uint64_t resident = persistent_blocks((const void*)k_radix_pass<0, 0>, kSortThreads);
  if (blocks > resident) blocks = resident;
  using K = void (*)(RadixArgs);
#define ARGUS_SLOTS(W) \
  k_radix_pass<W, 0>, k_radix_pass<W, 1>, k_radix_pass<W, 2>, k_radix_pass<W, 3>, \
  k_radix_pass<W, 4>, k_radix_pass<W, 5>, k_radix_pass<W, 6>, k_radix_pass<W, 7>, \
  k_radix_pass<W, 8>, k_radix_pass<W, 9>, k_radix_pass<W, 10>, k_radix_pass<W, 11>, \
  k_radix_pass<W, 12>, k_radix_pass<W, 13>, k_radix_pass<W, 14>, k_radix_pass<W, 15>
  static const K table[2][kSlots] = {{ARGUS_SLOTS(0)}, {ARGUS_SLOTS(1)}};
#undef ARGUS_SLOTS
  hipLaunchKernelGGL(table[which][slot], dim3((uint32_t)blocks), dim3(kSortThreads), 0, s, ra);
  return hipGetLastError();
}

}  // namespace argus
