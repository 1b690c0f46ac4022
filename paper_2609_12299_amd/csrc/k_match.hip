// k_match.hip -- replay of the per-context nested region stack, in parallel.
//
// The paper's Section 3.2 attributes work to regions through a nested
// region-context stack per warp: begin(id) pushes, end(id) closes the
// innermost active region.  Over records sorted by (ctx, ts, input index)
// the stack size after record i of a context is the clamped depth
//   s_i = max(0, s_{i-1} + delta_i),  delta = +1 for BEGIN, -1 for END,
// reset to 0 at the start of each context; an END with s_{i-1} = 0 is an
// orphan.  With x_i = s_{i-1} (the depth before record i, -1 at the start of
// a context):
//   * the BEGIN closed by a (non-orphan) END at position j with s_j = L is the
//     last position q < j with x_q <= L;
//   * the parent of a BEGIN at position k with level L >= 1 is the last
//     position q < k with x_q <= L - 1.
// Both are previous-smaller-value searches, answered here on a min-tree over
// x held in LDS.  The map s -> max(c, s + a) (or a constant after a context
// start) composes associatively, so the depth entering each tile comes from
// a scan over per-tile sums done beforehand (k_tsum, k_mscan), and tiles are
// processed independently.  What a tile cannot resolve locally --
// ENDs that pop a level open at the tile start, BEGINs still open at its end,
// parents opened in an earlier tile -- is summarised per tile and resolved
// by k_resolve.
//
// Exclusive time is its inclusive duration less those of its closed
// children, accumulated in place (mod 2^64): a closed instance adds its
// duration to its own slot and takes it off its parent's.  Instances of the
// tile accumulate in LDS; what goes to instances open when the tile starts
// is kept per enclosing level for k_resolve.
#include "internal.h"

namespace argus {

// Min tree over the tile's 2048 leaves with fan-out 8, in LDS.  A leaf is
// the pair (x + 1, rank | region << 11): the local BEGIN rank and the region
// of the record (meaningful for BEGINs, the only records a search can hit),
// so that one read of a leaf group answers a search.  The upper levels live
// in their own array: level 1 (256 nodes) at 0, level 2 (32) at 256,
// level 3 (4, padded to 8) at 288.  Every group of 8 siblings is 32-byte
// aligned.
constexpr int kU1 = 0, kU2 = 256, kU3 = 288, kUpSize = 296;
// The 8 leaves of each level-1 node are 64 bytes, stored 80 bytes apart so
// that threads writing or reading their own node hit different banks.
constexpr int kLeafStride = 10;  // uint2 slots per node
__device__ __forceinline__ uint32_t leaf_slot(uint32_t p) { return (p >> 3) * kLeafStride + (p & 7u); }
constexpr uint32_t kNoHit = 0xFFFFFFFFu;
static_assert(kMatchTile == 2048, "tree levels assume 2048 leaves");

// Last j < lim of the 8 siblings at g whose value is <= v, or -1.
__device__ __forceinline__ int last_le8(const uint32_t* g, uint32_t lim, uint32_t v) {
  const uint4 a = *(const uint4*)g, b = *(const uint4*)(g + 4);
  const uint32_t x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  int r = -1;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if ((uint32_t)j < lim && x[j] <= v) r = j;
  return r;
}

// The last of 8 leaves whose x + 1 is <= v (one exists): its second word.
__device__ __forceinline__ uint32_t leaf_hit8(const uint2* g, uint32_t v) {
  const uint4 a = *(const uint4*)g, b = *(const uint4*)(g + 2);
  const uint4 c = *(const uint4*)(g + 4), d = *(const uint4*)(g + 6);
  const uint32_t x[8] = {a.x, a.z, b.x, b.z, c.x, c.z, d.x, d.z};
  const uint32_t y[8] = {a.y, a.w, b.y, b.w, c.y, c.w, d.y, d.w};
  uint32_t r = kNoHit;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if (x[j] <= v) r = y[j];
  return r;
}

// Second word of the last leaf q < 8 * chunk with x + 1 <= v, or kNoHit.
__device__ __forceinline__ uint32_t psv_hit(const uint2* leaf, const uint32_t* up, uint32_t chunk,
                                            uint32_t v) {
  int j = last_le8(up + kU1 + (chunk & ~7u), chunk & 7u, v);
  int n1;
  if (j >= 0) {
    n1 = (int)(chunk & ~7u) + j;
  } else {
    const uint32_t i2 = chunk >> 3, i3 = chunk >> 6;
    int n2;
    j = last_le8(up + kU2 + (i2 & ~7u), i2 & 7u, v);
    if (j >= 0) {
      n2 = (int)(i2 & ~7u) + j;
    } else {
      j = last_le8(up + kU3, i3, v);
      if (j < 0) return kNoHit;
      n2 = j * 8 + last_le8(up + kU2 + j * 8, 8u, v);
    }
    n1 = n2 * 8 + last_le8(up + kU1 + n2 * 8, 8u, v);
  }
  return leaf_hit8(leaf + n1 * kLeafStride, v);
}

struct MatchArgs {
  const DevPlan* plan;
  DevPlan* wplan;
  const uint64_t* key[2];
  const uint32_t* pay[2];
  const uint32_t* ctxw[2];
  argus_instance* inst;
  uint64_t* excl;
  TileDesc* tiles;
  const TileCarry* carry;
  uint64_t* pop_ts;
  uint32_t* pop_reg;
  uint32_t* pushes;
  uint64_t* op_sum;
  uint64_t* counters;
  uint64_t* rstats;
  uint32_t* tile_ctr;
  // overlap events in sorted-record order (merge path)
  uint64_t* ev[2];
  uint32_t K, G, shift, R;
  uint32_t* push_pos;
  uint32_t* pop_pos;
  uint2* ctx_list;
  uint64_t ctx_cap;
};

constexpr uint32_t kParNone = 0xFFFFFFFFu;
constexpr uint32_t kParOut = 0xFFFFFFFEu;
// What the tile takes off enclosing instances (open when it starts) is kept
// in LDS for the nearest kOcCap levels; deeper ones go to global memory.
constexpr uint32_t kOcCap = 512;
constexpr uint32_t kQueueCap = kMatchTile / 4;  // queued searches per wave

// WIDE: keys hold only the timestamp and contexts come from their own array
// (one instantiation runs, the other returns at once).
template <bool WIDE>
__global__ __launch_bounds__(kMatchThreads, 3) void k_match(MatchArgs a) {
  const DevPlan* P = a.plan;
  if ((P->rec.wide != 0) != WIDE) return;
  const uint32_t tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  constexpr int IT = kMatchItems;

  __shared__ __align__(16) uint2 s_leaf[kMatchTile / 8 * kLeafStride];  // tree leaves
  __shared__ uint32_t s_up[kUpSize];  // upper tree levels
  // exclusive times of the local BEGINs share the leaves' LDS: the tree is
  // dead once the searches are answered
  uint64_t* const s_cs = reinterpret_cast<uint64_t*>(s_leaf);
  // search queues (one per wave) during the searches; then the end time of
  // each local BEGIN closed in the tile
  __shared__ uint64_t s_tend[kMatchTile];
  __shared__ uint16_t s_ereg[kMatchTile];  // end region of each local BEGIN (0xFFFF: open)
  __shared__ uint64_t s_oc[kOcCap];        // taken off enclosing instances (zero between tiles)
  __shared__ Fn s_wfn[4];
  __shared__ uint32_t s_wnb[4];
  __shared__ uint32_t s_first, s_lastp1, s_heads, s_lo, s_sout, s_maxlvl, s_orph;
  __shared__ uint32_t s_sin, s_nbpre_lo, s_nbpre_hi, s_hpre, s_need;

  const KeySpace ks = P->rec;
  constexpr bool wide = WIDE;
  const uint64_t nv = P->n_valid;
  const uint32_t buf = P->rec_final;
  const uint64_t* gk = a.key[buf];
  const uint32_t* gp = a.pay[buf];
  const uint32_t* gc = a.ctxw[buf];
  auto ctx_of_key = [&](uint64_t k) -> uint32_t {
    return ks.ts_bits >= 64 ? 0u : (uint32_t)(k >> ks.ts_bits);
  };
  // Overlap events in sorted-record order: one word per record,
  // group << (ts_bits + 5) | ts_off << 5 | code, code = 0 for a record that
  // is no event, else 1 + 2 * class + is_end.
  const uint32_t g_bits = a.G > 1 ? bit_width64(a.G - 1) : 0u;
  const bool ev_on = a.K > 0 && ks.ts_bits + g_bits + kEvCodeBits <= 64;
  const uint32_t es = ks.ts_bits + kEvCodeBits;
  uint64_t* evo = a.ev[buf ^ 1u];
  auto group_of = [&](uint32_t raw_ctx) -> uint32_t {
    return a.shift >= 32 ? 0u : (raw_ctx >> a.shift);
  };

  // Tiles are independent: tile = block + k * grid, with the next tile's
  // records loaded while this one is processed.
  const uint64_t n_tiles = P->match_tiles;
  const uint32_t p0 = tid * IT;
  uint64_t tile = blockIdx.x;
  if (tile >= n_tiles) return;
  uint64_t nk[IT];
  uint32_t np[IT], nc[WIDE ? IT : 1];
  uint64_t nprev = 0;  // (lane 0) key or context word of the record before the thread's first
  TileCarry ncarry;  // values entering the tile (a uniform load)
  auto issue = [&](uint64_t t) {
    const uint64_t b = t * kMatchTile;
    ncarry = a.carry[t];
    if (lane == 0 && b + p0 > 0 && b + p0 <= nv) nprev = wide ? gc[b + p0 - 1] : gk[b + p0 - 1];
    const uint32_t c = nv - b < (uint64_t)kMatchTile ? (uint32_t)(nv - b) : (uint32_t)kMatchTile;
    if (p0 + IT <= c) {
      const uint4* k4 = (const uint4*)(gk + b + p0);
#pragma unroll
      for (int q = 0; q < IT / 2; ++q) {
        const uint4 v = k4[q];
        nk[2 * q] = (uint64_t)v.x | ((uint64_t)v.y << 32);
        nk[2 * q + 1] = (uint64_t)v.z | ((uint64_t)v.w << 32);
      }
      const uint4* p4 = (const uint4*)(gp + b + p0);
#pragma unroll
      for (int q = 0; q < IT / 4; ++q) {
        const uint4 v = p4[q];
        np[4 * q] = v.x;
        np[4 * q + 1] = v.y;
        np[4 * q + 2] = v.z;
        np[4 * q + 3] = v.w;
      }
      if constexpr (WIDE) {
        const uint4* c4 = (const uint4*)(gc + b + p0);
#pragma unroll
        for (int q = 0; q < IT / 4; ++q) {
          const uint4 v = c4[q];
          nc[4 * q] = v.x;
          nc[4 * q + 1] = v.y;
          nc[4 * q + 2] = v.z;
          nc[4 * q + 3] = v.w;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < IT; ++i) {
        const uint32_t q = p0 + i;
        nk[i] = q < c ? gk[b + q] : 0;
        np[i] = q < c ? gp[b + q] : 0;
        if constexpr (WIDE) nc[i] = q < c ? gc[b + q] : 0;
      }
    }
  };
  for (uint32_t k = tid; k < kOcCap; k += kMatchThreads) s_oc[k] = 0;
  if (tid == 0) {
    s_first = kMatchTile;
    s_lastp1 = 0;
    s_heads = 0;
    s_lo = 0xFFFFFFFFu;
    s_maxlvl = 0;
    s_orph = 0;
    s_need = 0;
  }
  __syncthreads();

  for (;;) {
  issue(tile);
  // thread indices opaque per tile: lane-condition masks derived from them
  // are then computed where used, not held in scalar registers (spilled)
  // across the tile loop
  uint32_t tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const uint32_t lane = tid & 63, w = tid >> 6;
  const uint64_t base = tile * kMatchTile;
  const uint32_t cnt = nv - base < (uint64_t)kMatchTile ? (uint32_t)(nv - base) : (uint32_t)kMatchTile;
  const uint64_t next = tile + gridDim.x;

  // ---- this thread's 8 consecutive records (loaded one tile ahead)
  // the sort key of each record: its timestamp and context are recomputed
  // from it where needed (fewer live registers)
  uint64_t kk[IT];
  uint32_t ctxw[WIDE ? IT : 1], reg[IT];
  auto TS = [&](int i) -> uint64_t { return ks.ts_min + (wide ? kk[i] : (kk[i] & ks.ts_mask)); };
  auto CTX = [&](int i) -> uint32_t { return wide ? ctxw[WIDE ? i : 0] : ctx_of_key(kk[i]); };
  uint32_t fb = 0, fv = 0;  // bit i: BEGIN / valid
  uint64_t prev_raw;
  // overlap class of each record (8 bits each, 0xFF: none), from the payload
  uint32_t clsp[2] = {0xFFFFFFFFu, 0xFFFFFFFFu};
  {
    uint64_t key[IT];
    uint32_t pay[IT];
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      key[i] = nk[i];
      pay[i] = np[i];
      if constexpr (WIDE) ctxw[WIDE ? i : 0] = nc[WIDE ? i : 0];
    }
    prev_raw = nprev;
    if (tid == 0) {
      // read by every thread after the scan below; the previous tile's reads
      // of these are behind the barrier that ended it
      s_sin = ncarry.s_in;
      s_hpre = ncarry.hpre;
      s_nbpre_lo = (uint32_t)ncarry.nbpre;
      s_nbpre_hi = (uint32_t)(ncarry.nbpre >> 32);
    }
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      kk[i] = key[i];
      reg[i] = pay[i] & 0xFFFFu;
      if (p0 + i < cnt) {
        fv |= 1u << i;
        if (((pay[i] >> 16) & 1u) == 0) fb |= 1u << i;
        const uint32_t c = pay[i] >> kPayClsShift;
        clsp[i >> 2] = (clsp[i >> 2] & ~(0xFFu << (8 * (i & 3)))) | (c << (8 * (i & 3)));
      }
    }
  }
  // the record flags opaque: later tests of them are not tied back to the
  // compares that made them (whose masks would stay live across the tile)
  asm volatile("" : "+v"(fv), "+v"(fb));
  // context of the record before this thread's first one: the previous
  // lane's last record, or (lane 0) a load of the record before
  uint32_t prev0 = lane_prev(CTX(IT - 1), 0u);
  bool has_prev0 = true;
  if (lane == 0) {
    const uint64_t pp = base + p0;
    has_prev0 = pp > 0;
    prev0 = pp > 0 ? (wide ? (uint32_t)prev_raw : ctx_of_key(prev_raw)) : 0u;
  }

  uint32_t fh = 0;  // bit i: context start
  Fn f = fn_id();
  uint32_t nb = 0;
  uint32_t first_head = kMatchTile, last_p1 = 0, nheads = 0;
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    const uint32_t p = p0 + i;
    if ((fv >> i) & 1u) {
      const bool isb = (fb >> i) & 1u;
      const bool head = i > 0 ? CTX(i - 1) != CTX(i) : (!has_prev0 || prev0 != CTX(i));
      if (head) {
        fh |= 1u << i;
        first_head = p < first_head ? p : first_head;
        last_p1 = p + 1;
        nheads++;
      }
      const Fn e = head ? Fn{1u, 0, isb ? 1 : 0} : Fn{0u, isb ? 1 : -1, 0};
      f = compose(f, e);
      nb += isb;
    }
  }
  asm volatile("" : "+v"(fh));
  if (nheads) {
    atomicMin(&s_first, first_head);
    atomicMax(&s_lastp1, last_p1);
    atomicAdd(&s_heads, nheads);
  }

  // ---- block exclusive scan of the per-thread maps, BEGIN counts and
  // context-start counts (packed as nb | starts << 16)
  const Fn x = wave_scan_fn(f);
  const uint32_t nbh = nb | (nheads << 16);
  const uint32_t nbx = (uint32_t)wave_incl_scan32((int32_t)nbh);
  if (lane == 63) {
    s_wfn[w] = x;
    s_wnb[w] = nbx;
  }
  // the previous lane's inclusive map (the identity in lane 0)
  const Fn id = fn_id();
  const Fn ex = Fn{lane_prev(x.reset, id.reset), (int32_t)lane_prev((uint32_t)x.a, (uint32_t)id.a),
                   (int32_t)lane_prev((uint32_t)x.c, (uint32_t)id.c)};
  uint32_t nbex = nbx - nbh;
  __syncthreads();
  Fn pre = fn_id();
  uint32_t pnb = 0;
  for (uint32_t k = 0; k < w; ++k) {
    pre = compose(pre, s_wfn[k]);
    pnb += s_wnb[k];
  }
  const Fn tfn = compose(pre, ex);  // map from tile input to this thread's input
  const uint32_t tnbh = pnb + nbex;
  const uint32_t tnb = tnbh & 0xFFFFu;  // BEGINs of the tile before this thread
  const uint32_t thd = tnbh >> 16;      // context starts of the tile before this thread

  // ---- entering values of the tile (depth, BEGINs and context starts
  // before it), from the scan over the tile sums (all written before the
  // barrier above)
  const uint32_t tile_nb = (s_wnb[0] + s_wnb[1] + s_wnb[2] + s_wnb[3]) & 0xFFFFu;

  const uint32_t s_in = s_sin;
  const uint64_t nbpre = (uint64_t)s_nbpre_lo | ((uint64_t)s_nbpre_hi << 32);
  const uint32_t first = s_first, lastp1 = s_lastp1;
  const bool first_is_head = first == 0;

  // ---- context list (key and first sorted position of every context, in
  // order) and the bits in which neighbouring contexts of one group first
  // differ: the merge rounds that ordering the overlap events needs
  if (ev_on && fh) {
    uint32_t ord = s_hpre + thd, need = 0;
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      if (!((fh >> i) & 1u)) continue;
      const uint32_t c1 = CTX(i) + (uint32_t)ks.ctx_min;
      if (ord < a.ctx_cap) a.ctx_list[ord] = make_uint2(c1, (uint32_t)(base + p0 + i));
      ++ord;
      if (i > 0 || has_prev0) {
        const uint32_t c0 = (i > 0 ? CTX(i - 1) : prev0) + (uint32_t)ks.ctx_min;
        const uint32_t hb = 31u - (uint32_t)__clz(c0 ^ c1);
        if (hb < a.shift && group_of(c1) < a.G) need |= 1u << hb;
      }
    }
    if (need) atomicOr(&s_need, need);
  }

  // ---- depths before each record (sb); leaves x + 1 and the lower tree
  // levels.  The depth after a record is sb + 1 (BEGIN), sb - 1 (END with
  // sb > 0) or 0 (orphan END).
  uint32_t sb[IT];
  uint32_t lo = 0xFFFFFFFFu, maxlvl = 0, norph = 0;
  {
    uint32_t cur = (uint32_t)apply(tfn, (int64_t)s_in);
    if (tid == 0 && !first_is_head) lo = s_in;
    uint32_t xp[IT];
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const uint32_t p = p0 + i;
      sb[i] = 0;
      xp[i] = 0xFFFFFFFFu;
      if ((fv >> i) & 1u) {
        const bool head = (fh >> i) & 1u;
        const bool isb = (fb >> i) & 1u;
        const uint32_t before = head ? 0u : cur;
        uint32_t after;
        if (isb) {
          after = before + 1;
          maxlvl = before > maxlvl ? before : maxlvl;
        } else if (before == 0) {
          after = 0;  // orphan END
          norph++;
          atomicAdd((unsigned long long*)&a.rstats[(uint64_t)reg[i] * ARGUS_RS_WIDTH + ARGUS_RS_ORPHAN_END], 1ull);
        } else {
          after = before - 1;
        }
        sb[i] = before;
        xp[i] = head ? 0u : before + 1;  // x + 1, so that a context start is 0
        if (p < first) lo = after < lo ? after : lo;
        cur = after;
        if (p + 1 == cnt) s_sout = after;
      }
    }
    uint4* leaf4 = (uint4*)&s_leaf[leaf_slot(p0)];
    uint32_t r = tnb;
#pragma unroll
    for (int q = 0; q < IT / 2; ++q) {
      const uint32_t r0 = r;
      r += (fb >> (2 * q)) & 1u;
      const uint32_t r1 = r;
      r += (fb >> (2 * q + 1)) & 1u;
      leaf4[q] = make_uint4(xp[2 * q], r0 | (reg[2 * q] << 11), xp[2 * q + 1], r1 | (reg[2 * q + 1] << 11));
    }
    uint32_t m = xp[0];
#pragma unroll
    for (int i = 1; i < IT; ++i) m = min(m, xp[i]);
    s_up[kU1 + tid] = m;
    // minima over 8 lanes (quads, then the mirrored half row), over the row
    // of 16, then over the wave from the four rows
    m = min(m, dpp32<kDppQuad1032>(m));
    m = min(m, dpp32<kDppQuad2301>(m));
    m = min(m, dpp32<kDppHalfMirror>(m));
    if ((lane & 7) == 0) s_up[kU2 + (tid >> 3)] = m;
    m = min(m, dpp32<kDppMirror>(m));
    m = min(min((uint32_t)__builtin_amdgcn_readlane((int)m, 0), (uint32_t)__builtin_amdgcn_readlane((int)m, 16)),
            min((uint32_t)__builtin_amdgcn_readlane((int)m, 32), (uint32_t)__builtin_amdgcn_readlane((int)m, 48)));
    if (lane == 0) {
      s_up[kU3 + w] = m;
      s_up[kU3 + 4 + w] = 0xFFFFFFFFu;
    }
  }
  if (lo != 0xFFFFFFFFu) atomicMin(&s_lo, lo);
  if (maxlvl) atomicMax(&s_maxlvl, maxlvl);
  if (norph) atomicAdd(&s_orph, norph);
  for (uint32_t k = tid; k < (uint32_t)kMatchTile; k += kMatchThreads) s_ereg[k] = 0xFFFF;
  __syncthreads();
  const uint32_t lo_head = first_is_head ? 0u : s_lo;
  const uint32_t sin_eff = first_is_head ? 0u : s_in;
  const uint32_t op_lo = lo_head >= 1 ? lo_head - 1 : 0;
  const bool has_head = lastp1 > 0;
  const uint32_t lo_tail = has_head ? 0u : lo_head;
  const uint64_t pool = tile * kMatchTile;

  // ---- searches.  An END with depth sb before it closes level sb - 1: its
  // BEGIN is the last q < p with x + 1 <= sb; a BEGIN at level sb >= 1 has
  // as parent the last q < p with x + 1 <= sb.  This thread's own records
  // are scanned in registers; the others are queued per wave and answered
  // on the tree by all lanes of the wave together.
  uint32_t hit[IT];   // rank | region << 11 of the answer, or kNoHit
  uint32_t qmask = 0; // bit i: record i asks a question
  uint32_t pend = 0;  // bit i: answered by the tree
  // Inside the thread both answers are the BEGIN on top of the thread's own
  // stack of open BEGINs (a bit mask over its records; a context start
  // empties it): the last earlier record at depth sb - 1 is the BEGIN that
  // opened that level, and no later record went below it.
  uint32_t open = 0;
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    hit[i] = kNoHit;
    if (!((fv >> i) & 1u)) continue;
    if ((fh >> i) & 1u) open = 0;
    const bool isb = (fb >> i) & 1u;
    if (sb[i] != 0) {  // not a top-level BEGIN or an orphan END
      qmask |= 1u << i;
      if (open) {
        const uint32_t qi = 31u - (uint32_t)__clz(open);
        hit[i] = s_leaf[leaf_slot(p0) + qi].y;
        if (!isb) open &= ~(1u << qi);
      } else {
        pend |= 1u << i;
      }
    }
    if (isb) open |= 1u << i;
  }
  {
    uint32_t* q = (uint32_t*)(s_tend + w * (kQueueCap / 2));  // kQueueCap u32 entries
    const uint32_t np = (uint32_t)__popc(pend);
    const uint32_t off = (uint32_t)wave_incl_scan32((int32_t)np) - np;
    const uint32_t total = __shfl(off + np, 63);
    // entries: the query value and the asking thread (v < 2^23 assumed by
    // the packing; larger depths take the register path below)
    uint32_t k = off;
    bool big = false;
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      if (!((pend >> i) & 1u)) continue;
      big |= sb[i] >= (1u << 23);
      q[k++] = (sb[i] << 9) | (tid << 1);
    }
    const bool any_big = __ballot(big) != 0ull;
    if (!any_big) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // four queries per lane in flight, so that their dependent LDS
      // reads overlap
      for (uint32_t j0 = lane; j0 < total; j0 += 256) {
        uint32_t e[4], h[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) e[u] = j0 + 64u * u < total ? q[j0 + 64u * u] : 0u;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          h[u] = j0 + 64u * u < total ? psv_hit(s_leaf, s_up, (e[u] >> 1) & 0xFFu, e[u] >> 9) : kNoHit;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (j0 + 64u * u < total) q[j0 + 64u * u] = h[u];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      k = off;
#pragma unroll
      for (int i = 0; i < IT; ++i) {
        if (!((pend >> i) & 1u)) continue;
        hit[i] = q[k++];
      }
    } else {
#pragma unroll
      for (int i = 0; i < IT; ++i)
        if ((pend >> i) & 1u) hit[i] = psv_hit(s_leaf, s_up, tid, sb[i]);
    }
  }
  __syncthreads();  // the queues are no longer needed: s_tend takes end times
  for (uint32_t k = tid; k < tile_nb; k += kMatchThreads) s_cs[k] = 0;

  // ---- what the answers mean
  uint32_t par[IT];
  uint32_t mend = 0;  // bit i: END matched to a BEGIN of the same region
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    par[i] = kParNone;
    if (!((qmask >> i) & 1u)) continue;
    const bool isb = (fb >> i) & 1u;
    const bool found = hit[i] != kNoHit;
    const uint32_t qrank = hit[i] & 0x7FFu, qreg = hit[i] >> 11;
    if (!isb) {
      if (found) {
        s_tend[qrank] = TS(i);
        s_ereg[qrank] = (uint16_t)reg[i];
        if (qreg == reg[i]) mend |= 1u << i;
      } else {
        // pops a level that was open when the tile started
        const uint32_t L = sb[i] - 1;
        const uint32_t idx = L - lo_head;
        if (L >= lo_head && idx < (uint32_t)kMatchTile) {
          a.pop_ts[pool + idx] = TS(i);
          a.pop_reg[pool + idx] = reg[i];
          if (ev_on) a.pop_pos[pool + idx] = (uint32_t)(base + p0 + i);
        } else {
          flag_internal_error(a.counters, 16);
        }
      }
    } else {
      par[i] = found ? qrank : kParOut;
    }
  }
  // sums for enclosing instances beyond the LDS ones start at zero
  const uint32_t n_op = (sin_eff > op_lo) ? ((sin_eff - op_lo) < (uint32_t)kMatchTile ? sin_eff - op_lo : (uint32_t)kMatchTile) : 0u;
  for (uint32_t k = kOcCap + tid; k < n_op; k += kMatchThreads) a.op_sum[pool + k] = 0;
  if (n_op > kOcCap) __threadfence_block();
  __syncthreads();  // end times and end regions of the local BEGINs are complete

  // ---- exclusive times, open BEGINs and the instances
  uint32_t mbeg = 0;  // bit i: BEGIN matched to an END of the same region
  {
    uint32_t r = tnb;
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const uint32_t p = p0 + i;
      if (!((fv >> i) & 1u) || !((fb >> i) & 1u)) continue;
      const uint32_t k = r++;
      const uint64_t id = nbpre + k;
      const uint32_t L = sb[i];
      const uint32_t ereg = s_ereg[k];
      if (ereg != kNoEnd) {
        const uint64_t t_end = s_tend[k];
        if (ereg == reg[i]) mbeg |= 1u << i;
        const uint64_t incl = t_end - TS(i);
        // its own duration in, its duration out of its parent's
        atomicAdd((unsigned long long*)&s_cs[k], (unsigned long long)incl);
        const unsigned long long out = (unsigned long long)(0ull - incl);
        if (par[i] == kParOut) {
          const uint32_t oi = (L - 1) - op_lo;
          if (L >= 1 + op_lo && oi < (uint32_t)kMatchTile) {
            if (oi < kOcCap)
              atomicAdd((unsigned long long*)&s_oc[oi], out);
            else
              atomicAdd((unsigned long long*)&a.op_sum[pool + oi], out);
          } else {
            flag_internal_error(a.counters, 16);
          }
        } else if (par[i] != kParNone) {
          atomicAdd((unsigned long long*)&s_cs[par[i]], out);
        }
      } else if (lastp1 <= p + 1) {
        // still open when the tile ends, in a context that may continue
        if (L >= lo_tail && L - lo_tail < (uint32_t)kMatchTile) {
          a.pushes[pool + (L - lo_tail)] = (uint32_t)id;
          if (ev_on) a.push_pos[pool + (L - lo_tail)] = (uint32_t)p + (uint32_t)base;
        } else
          flag_internal_error(a.counters, 16);
      }
      const uint64_t t_end = ereg != kNoEnd ? s_tend[k] : kU64Max;
      uint32_t pf;
      if (par[i] == kParNone) pf = kNoParent;
      else if (par[i] == kParOut) pf = kParentPending | (uint32_t)tile;
      else pf = (uint32_t)(nbpre + par[i]);
      const uint64_t tb = TS(i);
      const uint4 w0 = make_uint4((uint32_t)tb, (uint32_t)(tb >> 32), (uint32_t)t_end,
                                  (uint32_t)(t_end >> 32));
      const uint4 w1 = make_uint4(CTX(i) + (uint32_t)ks.ctx_min, pf, L, reg[i] | (ereg << 16));
      uint4* dst = (uint4*)(a.inst + id);
      dst[0] = w0;
      dst[1] = w1;
    }
  }
  __syncthreads();  // exclusive times of the tile complete
  for (uint32_t k = tid; k < tile_nb; k += kMatchThreads) {
    a.excl[nbpre + k] = s_cs[k];
  }
  const uint32_t n_oc = n_op < kOcCap ? n_op : kOcCap;
  for (uint32_t k = tid; k < n_oc; k += kMatchThreads) {
    a.op_sum[pool + k] = s_oc[k];
    s_oc[k] = 0;
  }

  // ---- overlap event words
  if (ev_on) {
    uint64_t e[IT];
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const uint64_t g = group_of(CTX(i) + (uint32_t)ks.ctx_min);
      const uint32_t c = (clsp[i >> 2] >> (8 * (i & 3))) & 0xFFu;
      const uint32_t ev = (((mend | mbeg) >> i) & 1u) && c < a.K ? 1u + 2u * c + (((fb >> i) & 1u) ^ 1u) : 0u;
      e[i] = (es < 64 ? (g << es) : 0ull) | ((TS(i) - ks.ts_min) << kEvCodeBits) | ev;
    }
    if (p0 + IT <= cnt) {
      uint4* e4 = (uint4*)(evo + base + p0);
#pragma unroll
      for (int q = 0; q < IT / 2; ++q)
        e4[q] = make_uint4((uint32_t)e[2 * q], (uint32_t)(e[2 * q] >> 32), (uint32_t)e[2 * q + 1],
                           (uint32_t)(e[2 * q + 1] >> 32));
    } else {
#pragma unroll
      for (int i = 0; i < IT; ++i)
        if ((fv >> i) & 1u) evo[base + p0 + i] = e[i];
    }
  }

  // ---- per-tile outputs
  if (tid == 0) {
    const uint32_t s_out = cnt ? s_sout : 0u;
    TileDesc d;
    d.key = has_head ? -1 : (int64_t)lo_head;
    d.s_in = sin_eff;
    d.lo_head = lo_head;
    d.s_out = s_out;
    d.lo_tail = lo_tail;
    d.op_lo = op_lo;
    d.pop_base = 0;
    d.push_base = 0;
    d.op_base = 0;
    d.n_pop = sin_eff - lo_head;
    d.n_push = s_out - lo_tail;
    if (d.n_pop > (uint32_t)kMatchTile || d.n_push > (uint32_t)kMatchTile) {
      flag_internal_error(a.counters, 32);
      d.n_pop = d.n_pop > (uint32_t)kMatchTile ? 0u : d.n_pop;
      d.n_push = d.n_push > (uint32_t)kMatchTile ? 0u : d.n_push;
    }
    d.n_op = n_op;
    d.pad = 0;
    a.tiles[tile] = d;
    // every thread has read this tile's scalars: reset them for the next
    // (the counts and the merge bits add up over the block's tiles)
    s_first = kMatchTile;
    s_lastp1 = 0;
    s_lo = 0xFFFFFFFFu;
  }
  __syncthreads();
  if (next >= n_tiles) break;
  tile = next;
  }  // tiles
  if (tid == 0) {
    unsigned long long* c = (unsigned long long*)a.counters;
    if (s_need) atomicOr(&a.wplan->m_need, s_need);
    if (s_heads) atomicAdd(&c[ARGUS_C_N_CTX], (unsigned long long)s_heads);
    if (s_maxlvl) atomicMax(&c[ARGUS_C_MAX_LEVEL], (unsigned long long)s_maxlvl);
    if (s_orph) atomicAdd(&c[ARGUS_C_N_ORPHAN_END], (unsigned long long)s_orph);
  }
}

hipError_t launch_match(const RunArgs& a, hipStream_t s) {
  MatchArgs m{};
  m.plan = a.w.plan;
  m.wplan = a.w.plan;
  for (int b = 0; b < 2; ++b) m.ev[b] = a.w.key[b];
  m.K = a.K;
  m.G = a.G;
  m.shift = a.shift;
  m.R = a.R;
  m.push_pos = a.w.push_pos;
  m.pop_pos = a.w.pop_pos;
  m.ctx_list = a.w.ctx_list;
  m.ctx_cap = a.w.ctx_cap;
  for (int b = 0; b < 2; ++b) {
    m.key[b] = a.w.key[b];
    m.pay[b] = a.w.pay[b];
    m.ctxw[b] = a.w.ctxw[b];
  }
  m.inst = a.w.inst;
  m.excl = a.w.excl;
  m.tiles = a.w.tiles;
  m.carry = a.w.carry;
  m.pop_ts = a.w.pop_ts;
  m.pop_reg = a.w.pop_reg;
  m.pushes = a.w.pushes;
  m.op_sum = a.w.op_sum;
  m.counters = a.out.d_counters;
  m.rstats = a.out.d_region_stats;
  m.tile_ctr = a.w.tile_ctr;
  uint64_t blocks = a.w.match_tiles;
  const uint64_t resident = persistent_blocks((const void*)k_match<false>, kMatchThreads);
  if (blocks > resident) blocks = resident;
  hipLaunchKernelGGL(k_match<false>, dim3((uint32_t)blocks), dim3(kMatchThreads), 0, s, m);
  hipLaunchKernelGGL(k_match<true>, dim3((uint32_t)blocks), dim3(kMatchThreads), 0, s, m);
  return hipGetLastError();
}

}  // namespace argus
