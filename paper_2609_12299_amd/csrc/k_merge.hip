// k_merge.hip -- overlap events put in (group, time) order by merging the
// per-context runs of the sorted records.
//
// The overlap of region classes (the paper's Section 4.3; groups of contexts
// are the Section 3.2 scope) is an endpoint sweep over the begin and end
// events of the matched, classified instances of each group, in time order.
// Within one context those events already appear in time order: they are a
// subsequence of the records sorted by (context, timestamp).  So instead of
// sorting all events, the matching kernel writes one event word per sorted
// record (a record that is no event gets code 0, which changes no count and
// only splits a gap), and the runs of the contexts of each group are merged.
//
// Contexts of one group (ctx >> shift) are adjacent in the sorted records.
// Merging over bit b takes, for every prefix ctx >> (b + 1), the run of its
// contexts whose bit b is 0 and the run of those whose bit b is 1; bits go in
// increasing order, and only bits in which two neighbouring contexts of one
// group first differ are merged (no other bit has a pair to merge).  A pass
// merges two such bits at once: four runs per prefix ctx >> (upper bit + 1),
// in the order of the two bits read as a number, which is the order two
// passes of one bit each would give.  After the last pass every group is one
// run in time order.
//
// A pass is two launches after the segment boundaries of all passes (one
// block per pass): the splits of every output tile, then the merge of each
// tile's input slices in LDS (two stages for four runs: the pairs, then
// their results).  A two-way pass splits at every 4096th output (Green,
// McColl and Bader's merge path: a binary search on the cross diagonal); a
// four-way pass ranks every 127th event of each run among the others and
// cuts at every 28th of them in merged order.  The last pass does not store
// what it merges: k_merge_sweep sweeps each merged tile at once (its
// segments are exactly the groups).
#include "sweep_common.h"

namespace argus {

constexpr uint32_t kNoSplit = 0xFFFFFFFFu;

// ------------------------------------------------------------------ plan

struct MPlanArgs {
  DevPlan* plan;
  const uint2* ctx_list;
  const uint64_t* counters;
  uint32_t K, G, shift;
  uint32_t force_radix;
  uint32_t max_bits;
  uint64_t ctx_cap;
};

// Chooses between merging and the event radix sort, and plans the passes.
// Merging applies when the event word (group, timestamp offset, code) fits
// 64 bits, the context list is complete, and the bits to merge are few
// enough.
__global__ __launch_bounds__(64) void k_mplan(MPlanArgs a) {
  if (threadIdx.x != 0) return;
  DevPlan* p = a.plan;
  p->ev_merge = 0;
  if (a.K == 0 || a.force_radix) return;
  const KeySpace ks = p->rec;
  const uint32_t g_bits = a.G > 1 ? bit_width64(a.G - 1) : 0u;
  if (ks.ts_bits + g_bits + kEvCodeBits > 64) return;
  const uint64_t n_ctx = a.counters[ARGUS_C_N_CTX];
  if (n_ctx > a.ctx_cap) return;
  const uint32_t need = p->m_need;
  const uint32_t bits = (uint32_t)__popc(need);
  // Merging one bit moves 8 + 8 bytes per event, a radix pass 12 + 12 plus
  // its look-back traffic: merging wins up to about twice as many bits (and
  // more, two bits sharing a pass).
  const uint32_t radix_passes = (g_bits + ks.ts_bits + 7) / 8;
  if (bits > a.max_bits || bits > 2 * radix_passes) return;
  // contexts of groups < G form a prefix of the (sorted) context list
  uint64_t lo = 0, hi = n_ctx;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) / 2;
    const uint32_t c = a.ctx_list[mid].x;
    const uint64_t g = a.shift >= 32 ? 0 : (c >> a.shift);
    if (g < a.G) lo = mid + 1;
    else hi = mid;
  }
  p->m_nctx = (uint32_t)lo;
  p->m_end = lo < n_ctx ? a.ctx_list[lo].y : p->n_valid;
  // No bit to merge: every group is one context, already in time order; one
  // pass that merges nothing takes each group as a run of its own.
  p->m_rounds = bits ? (bits + 1) / 2 : 1u;
  uint32_t buf = p->rec_final ^ 1u, r = 0, pending = kNoBit;
  auto emit = [&](uint32_t b, uint32_t b2) {
    MergeRound& m = p->mr[r++];
    m.bit = b;
    m.bit2 = b2;
    m.src = buf;
    m.dst = buf ^ 1u;
    m.n_segs = 0;
    m.n_tiles = 0;
    buf ^= 1u;
  };
  for (uint32_t b = 0; b < 32; ++b) {
    if (!((need >> b) & 1u)) continue;
    if (pending == kNoBit) {
      pending = b;
    } else {
      emit(pending, b);
      pending = kNoBit;
    }
  }
  if (pending != kNoBit) emit(pending, kNoBit);
  if (bits == 0) emit(kSegByGroup, kNoBit);
  p->ev_final = buf;
  p->n_ev = p->m_end;
  KeySpace ek = ks;
  ek.ctx_min = 0;
  ek.ctx_bits = g_bits;
  ek.wide = 0;
  p->ev = ek;
  p->ev_merge = 1;
}

hipError_t launch_mplan(const RunArgs& a, hipStream_t s) {
  MPlanArgs m{a.w.plan, a.w.ctx_list, a.out.d_counters, a.K, a.G, a.shift,
              (a.flags & ARGUS_FORCE_EVENT_SORT) ? 1u : 0u,
              a.shift < (uint32_t)kMaxMergeBits ? a.shift : (uint32_t)kMaxMergeBits,
              a.w.ctx_cap};
  hipLaunchKernelGGL(k_mplan, dim3(1), dim3(64), 0, s, m);
  return hipGetLastError();
}

// -------------------------------------------------------------- segments

// Inclusive sum over the 1024 threads of the block; *total gets the sum.
__device__ __forceinline__ uint32_t block_incl_scan1024(uint32_t v, uint32_t* s_w,
                                                        uint32_t* total) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_w[w] = x;
  __syncthreads();
  uint32_t pre = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const uint32_t c = s_w[k];
    pre += k < w ? c : 0u;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return pre + x;
}

struct MSegArgs {
  DevPlan* plan;
  const uint2* ctx_list;
  uint4* seg_run;
  uint32_t* seg_tile0;
  uint32_t* seg_samp0;
  uint64_t* counters;
  uint64_t stride;  // per-pass stride of the segment arrays
  uint32_t shift;
};

// Samples of a run of len events: every kSampStride-th, from its first.
__device__ __forceinline__ uint32_t run_samples(uint32_t len) {
  return (len + kSampStride - 1) / kSampStride;
}

// Segments of every pass (block r: pass r): maximal runs of contexts with
// equal ctx >> (top + 1), top being the pass's upper bit.  The class of a
// context is the pass's bits read as a number (upper bit high).  Contexts of
// one segment come in class order: two of them first differ in one of the
// pass's bits, or in a bit an earlier pass merged (then they share a class
// and a run already).  So a segment is four runs in a row (two in a two-way
// pass), run q starting at the first context of class >= q (at the segment's
// end when there is none).  The segments depend on the context list only,
// so all passes are planned at once.
__global__ __launch_bounds__(1024) void k_mseg(MSegArgs a) {
  DevPlan* p = a.plan;
  const int round = blockIdx.x;
  if (!p->ev_merge || (uint32_t)round >= p->m_rounds) return;
  const uint64_t off = (uint64_t)round * a.stride;
  uint4* seg_run = a.seg_run + off;
  uint32_t* seg_tile0 = a.seg_tile0 + off;
  uint32_t* seg_samp0 = a.seg_samp0 + off;
  __shared__ uint32_t s_w[16];
  const MergeRound mr = p->mr[round];
  const bool by_group = mr.bit == kSegByGroup;
  const bool four = !by_group && mr.bit2 != kNoBit;
  const uint32_t top = four ? mr.bit2 : mr.bit;
  const uint32_t nc = p->m_nctx;
  const uint32_t end = (uint32_t)p->m_end;
  const uint32_t t = threadIdx.x;
  // segment key: ctx >> (top + 1), or the group for a pass that merges nothing
  auto hi_of = [&](uint32_t c) -> uint32_t {
    if (by_group) return a.shift >= 32 ? 0u : (c >> a.shift);
    return top >= 31 ? 0u : (c >> (top + 1));
  };
  auto cls_of = [&](uint32_t c) -> uint32_t {
    if (by_group) return 0u;
    const uint32_t lo = (c >> mr.bit) & 1u;
    return four ? ((((c >> mr.bit2) & 1u) << 1) | lo) : lo;
  };

  // ---- segments and run starts: four consecutive contexts per thread, 4096
  // per block step.  A context starts the runs of the classes after the one
  // before it in its segment, up to its own; the last context of a segment
  // starts the runs after its class at the segment's end.
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nc; base += 4096) {
    const uint32_t j0 = base + 4 * t;
    uint32_t prev = j0 > 0 && j0 - 1 < nc ? a.ctx_list[j0 - 1].x : 0u;
    bool head[4];
    uint2 e[4];
    uint32_t nh = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t j = j0 + q;
      head[q] = false;
      e[q] = make_uint2(0, 0);
      if (j < nc) {
        e[q] = a.ctx_list[j];
        head[q] = j == 0 || hi_of(prev) != hi_of(e[q].x);
        prev = e[q].x;
      }
      nh += head[q] ? 1u : 0u;
    }
    // the context after the thread's last one: does it start a segment, where
    uint32_t nx_start = end;
    bool nx_head = true;
    if (j0 + 4 < nc) {
      const uint2 f = a.ctx_list[j0 + 4];
      nx_start = f.y;
      nx_head = hi_of(f.x) != hi_of(e[3].x);
    }
    uint32_t total;
    uint32_t seg = carry + block_incl_scan1024(nh, s_w, &total) - nh;  // heads before j0
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t j = j0 + q;
      if (j >= nc) continue;
      if (head[q]) ++seg;
      uint32_t* r = reinterpret_cast<uint32_t*>(&seg_run[seg - 1]);
      const uint32_t c = cls_of(e[q].x);
      const uint32_t pc = head[q] ? 0u : cls_of(q > 0 ? e[q - 1].x : a.ctx_list[j - 1].x);
      if (head[q]) r[0] = e[q].y;
      if (pc > c) flag_internal_error(a.counters, 256);
      for (uint32_t x = pc + 1; x <= c && x < 4; ++x) r[x] = e[q].y;
      // last context of its segment
      const bool tail = q < 3 ? (j + 1 >= nc || head[q + 1]) : nx_head;
      if (tail) {
        const uint32_t s1 = q < 3 ? (j + 1 < nc ? e[q + 1].y : end) : nx_start;
        for (uint32_t x = c + 1; x < 4; ++x) r[x] = s1;
      }
    }
    carry += total;
  }
  const uint32_t n_segs = carry;
  __threadfence_block();
  __syncthreads();
  // ---- tiles and samples per segment, and their prefixes (four segments per
  // thread)
  carry = 0;
  uint32_t carry_s = 0;
  for (uint32_t base = 0; base < n_segs; base += 4096) {
    const uint32_t g0 = base + 4 * t;
    uint32_t tiles[4], samp[4], nt = 0, nsm = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t sg = g0 + q;
      tiles[q] = 0;
      samp[q] = 0;
      if (sg < n_segs) {
        const uint4 r = seg_run[sg];
        const uint32_t s1 = sg + 1 < n_segs ? seg_run[sg + 1].x : end;
        if (four) {
          samp[q] = run_samples(r.y - r.x) + run_samples(r.z - r.y) + run_samples(r.w - r.z) +
                    run_samples(s1 - r.w);
          tiles[q] = (samp[q] + kSampPerTile - 1) / kSampPerTile;
        } else {
          tiles[q] = (uint32_t)ceil_div(s1 - r.x, kMergeTile);
        }
      }
      nt += tiles[q];
      nsm += samp[q];
    }
    uint32_t total, total_s;
    uint32_t pre = carry + block_incl_scan1024(nt, s_w, &total) - nt;
    uint32_t pre_s = carry_s + block_incl_scan1024(nsm, s_w, &total_s) - nsm;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t sg = g0 + q;
      if (sg < n_segs) {
        seg_tile0[sg] = pre;
        seg_samp0[sg] = pre_s;
      }
      pre += tiles[q];
      pre_s += samp[q];
    }
    carry += total;
    carry_s += total_s;
  }
  if (t == 0) {
    seg_tile0[n_segs] = carry;
    seg_samp0[n_segs] = carry_s;
    p->mr[round].n_segs = n_segs;
    p->mr[round].n_tiles = carry;
  }
}

hipError_t launch_mseg(const RunArgs& a, int rounds, hipStream_t s) {
  MSegArgs m{a.w.plan, a.w.ctx_list, a.w.seg_run, a.w.seg_tile0, a.w.seg_samp0,
             a.out.d_counters, a.w.ctx_cap + 1, a.shift};
  hipLaunchKernelGGL(k_mseg, dim3((uint32_t)(rounds > 0 ? rounds : 1)), dim3(1024), 0, s, m);
  return hipGetLastError();
}

// ------------------------------------------------------------ partition

// Runs are in order of (group, time) only -- records of equal time keep
// their input order, whatever their codes -- so merging compares the words
// without the code bits.
__device__ __forceinline__ uint64_t mkey(uint64_t e) { return e >> kEvCodeBits; }

// Events taken from run A among the first d outputs of merging A and B
// (ties: A first): the merge-path split on diagonal d.
__device__ __forceinline__ uint32_t corank(const uint64_t* A, uint32_t la, const uint64_t* B,
                                           uint32_t lb, uint32_t d) {
  uint32_t lo = d > lb ? d - lb : 0u, hi = d < la ? d : la;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (mkey(A[mid]) <= mkey(B[d - 1 - mid])) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Merge tiles are staged in LDS with one pad word after every 16, so that
// threads touching 8 consecutive words each (64 bytes apart) spread over
// the banks.  lpad maps a tile position to its LDS slot.
__device__ __forceinline__ uint32_t lpad(uint32_t i) { return i + (i >> 4); }
constexpr uint32_t kMergeLds = kMergeTile + kMergeTile / 16 + 2;  // + reads just past a run

// corank over the runs P = tile slots [op, op + lp) and Q = [oq, oq + lq)
// staged in LDS.
__device__ __forceinline__ uint32_t corank_lds(const uint64_t* se, uint32_t op, uint32_t lp,
                                               uint32_t oq, uint32_t lq, uint32_t d) {
  uint32_t lo = d > lq ? d - lq : 0u, hi = d < lp ? d : lp;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (mkey(se[lpad(op + mid)]) <= mkey(se[lpad(oq + d - 1 - mid)])) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// One merge tile: where its slice of each of the four runs of its segment
// starts (absolute sorted positions; a two-way pass leaves the last two
// empty), where its output starts, whether it is the first tile of its
// segment, and where the four runs end.  A slice ends where the next tile's
// starts when that tile is in the same segment, else at its run's end.
struct MergeTask {
  uint32_t pos[4];
  uint32_t out_pos, first, pad0, pad1;
  uint32_t end[4];
};
static_assert(sizeof(MergeTask) == 48, "MergeTask layout");

__device__ __forceinline__ void store_task(MergeTask* dst, const uint32_t (&pos)[4], uint32_t out_pos,
                                           bool first, const uint32_t (&end)[4]) {
  uint4* d = reinterpret_cast<uint4*>(dst);
  d[0] = make_uint4(pos[0], pos[1], pos[2], pos[3]);
  d[1] = make_uint4(out_pos, first ? 1u : 0u, 0u, 0u);
  d[2] = make_uint4(end[0], end[1], end[2], end[3]);
}

struct MPartArgs {
  const DevPlan* plan;
  const uint64_t* ev[2];
  const uint4* seg_run;
  const uint32_t* seg_tile0;
  const uint32_t* seg_samp0;
  MergeTask* task;
  uint64_t* counters;
  int round;
  uint64_t stride;
};

// Whether event e comes before an event of key `key` in merged order: e's
// key is <= key when e is from an earlier run (le), else < key.
__device__ __forceinline__ bool before(uint64_t e, uint64_t key, bool le) {
  return le ? mkey(e) <= key : mkey(e) < key;
}

// For each run x, the first index in [lo[x], hi[x]) whose event, at st[x] +
// index * SCALE, does not come before `key`, left in lo[x].  search4_seq
// runs the four searches one after the other, each only as long as its own
// range (the sample ranks: many lanes, often short ranges); search4 runs
// them in lockstep, their loads in flight together, a finished search
// loading `safe` (a valid address) instead (the exact ranks of the few
// samples that start a tile).
template <uint32_t SCALE>
__device__ __forceinline__ void search4_seq(const uint64_t* src, const uint32_t (&st)[5], uint32_t q,
                                            uint64_t key, uint32_t (&lo)[4], const uint32_t (&hi)[4]) {
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    uint32_t l = lo[x], h = hi[x];
    while (l < h) {
      const uint32_t mid = (l + h) >> 1;
      if (before(src[st[x] + mid * SCALE], key, (uint32_t)x < q)) l = mid + 1;
      else h = mid;
    }
    lo[x] = l;
  }
}

template <uint32_t SCALE>
__device__ __forceinline__ void search4(const uint64_t* src, const uint32_t (&st)[5], uint32_t q,
                                        uint64_t key, uint32_t safe, uint32_t (&lo)[4],
                                        uint32_t (&hi)[4]) {
  while (lo[0] < hi[0] || lo[1] < hi[1] || lo[2] < hi[2] || lo[3] < hi[3]) {
    uint32_t mid[4];
    uint64_t v[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      mid[x] = (lo[x] + hi[x]) >> 1;
      v[x] = src[lo[x] < hi[x] ? st[x] + mid[x] * SCALE : safe];
    }
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      if (lo[x] < hi[x]) {
        if (before(v[x], key, (uint32_t)x < q)) lo[x] = mid[x] + 1;
        else hi[x] = mid[x];
      }
    }
  }
}

// Two-way pass: one thread per tile; the tile's start is the merge-path
// split at its first output.  Four-way pass: one thread per sample; its rank
// in merged order is its index in its run plus the samples of the other runs
// before it, and a sample of rank 12 j starts tile j of its segment, whose
// slices start where the events of each run before it end.
__global__ __launch_bounds__(256) void k_mpart(MPartArgs a) {
  const DevPlan* p = a.plan;
  if (!p->ev_merge || (uint32_t)a.round >= p->m_rounds) return;
  const MergeRound mr = p->mr[a.round];
  const uint32_t n_segs = (uint32_t)mr.n_segs;
  const uint64_t n_tiles = mr.n_tiles;
  const uint32_t end = (uint32_t)p->m_end;
  const uint64_t* src = a.ev[mr.src];
  const uint64_t off = (uint64_t)a.round * a.stride;
  const uint4* seg_run = a.seg_run + off;
  const uint32_t* seg_tile0 = a.seg_tile0 + off;
  const uint64_t step = (uint64_t)gridDim.x * 256;
  const uint64_t gid = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  const bool four = mr.bit != kSegByGroup && mr.bit2 != kNoBit;
  if (!four) {
    for (uint64_t k = gid; k < n_tiles; k += step) {
      // segment of tile k: the last one whose first tile is <= k
      uint32_t lo = 0, hi = n_segs;
      while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (seg_tile0[mid] <= k) lo = mid;
        else hi = mid;
      }
      const uint4 R = seg_run[lo];
      const uint32_t s0 = R.x, sp = R.y;
      const uint32_t s1 = lo + 1 < n_segs ? seg_run[lo + 1].x : end;
      const uint32_t L = s1 - s0, la = sp - s0, lb = s1 - sp;
      const uint64_t d0w = (k - seg_tile0[lo]) * (uint64_t)kMergeTile;
      if (!(s0 <= sp && sp <= s1 && s1 <= end && R.z == s1 && R.w == s1 && d0w < L)) {
        flag_internal_error(a.counters, 256);
        const uint32_t z[4] = {end, end, end, end};
        store_task(a.task + k, z, end, true, z);
        continue;
      }
      const uint32_t d0 = (uint32_t)d0w;
      const uint32_t a0 = corank(src + s0, la, src + sp, lb, d0);
      const uint32_t pos[4] = {s0 + a0, sp + (d0 - a0), s1, s1};
      const uint32_t ends[4] = {sp, s1, s1, s1};
      store_task(a.task + k, pos, s0 + d0, k == seg_tile0[lo], ends);
    }
    return;
  }
  const uint32_t* samp0 = a.seg_samp0 + off;
  const uint32_t total = n_segs ? samp0[n_segs] : 0u;
  for (uint64_t u = gid; u < total; u += step) {
    uint32_t lo = 0, hi = n_segs;
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (samp0[mid] <= u) lo = mid;
      else hi = mid;
    }
    const uint4 R = seg_run[lo];
    const uint32_t st[5] = {R.x, R.y, R.z, R.w, lo + 1 < n_segs ? seg_run[lo + 1].x : end};
    bool ok = st[4] <= end;
    uint32_t len[4], ns[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      ok = ok && st[q] <= st[q + 1];
      len[q] = st[q + 1] - st[q];
      ns[q] = run_samples(len[q]);
    }
    // this sample: run q, index k in it
    uint32_t rem = (uint32_t)(u - samp0[lo]), q = 0;
#pragma unroll
    for (int x = 0; x < 3; ++x) {
      if (q == (uint32_t)x && rem >= ns[x]) {
        rem -= ns[x];
        q = x + 1;
      }
    }
    uint32_t sq = st[0], nq = ns[0];
#pragma unroll
    for (int x = 1; x < 4; ++x) {
      sq = q == (uint32_t)x ? st[x] : sq;
      nq = q == (uint32_t)x ? ns[x] : nq;
    }
    const uint32_t tile0 = seg_tile0[lo], tiles = seg_tile0[lo + 1] - tile0;
    ok = ok && rem < nq;
    if (!ok) {
      flag_internal_error(a.counters, 256);
      continue;
    }
    const uint32_t k = rem * kSampStride;
    const uint64_t key = mkey(src[sq + k]);
    // samples of each other run before it
    uint32_t sl[4], sh[4], rho = rem;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      sl[x] = 0;
      sh[x] = (uint32_t)x == q ? 0u : ns[x];
    }
    search4_seq<kSampStride>(src, st, q, key, sl, sh);
#pragma unroll
    for (int x = 0; x < 4; ++x) rho += sl[x];
    if (rho % kSampPerTile) continue;
    const uint32_t j = rho / kSampPerTile;
    if (j >= tiles || tile0 + (uint64_t)j >= n_tiles) {
      flag_internal_error(a.counters, 256);
      continue;
    }
    // events of each other run before it: with c samples before it, between
    // (c - 1) * stride + 1 and c * stride (or the run's end)
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const uint32_t c = sl[x];
      if ((uint32_t)x == q) {
        sl[x] = sh[x] = k;
      } else if (c == 0) {
        sh[x] = 0;
      } else {
        sl[x] = (c - 1) * kSampStride + 1;
        sh[x] = c * kSampStride < len[x] ? c * kSampStride : len[x];
      }
    }
    search4<1>(src, st, q, key, sq + k, sl, sh);
    uint32_t pos[4], out = st[0];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      pos[x] = st[x] + sl[x];
      out += sl[x];
    }
    const uint32_t ends[4] = {st[1], st[2], st[3], st[4]};
    store_task(a.task + tile0 + j, pos, out, j == 0, ends);
  }
}

hipError_t launch_mpart(const RunArgs& a, int round, hipStream_t s) {
  MPartArgs m{};
  m.plan = a.w.plan;
  for (int b = 0; b < 2; ++b) m.ev[b] = a.w.key[b];
  m.seg_run = a.w.seg_run;
  m.seg_tile0 = a.w.seg_tile0;
  m.seg_samp0 = a.w.seg_samp0;
  m.task = (MergeTask*)a.w.part;
  m.counters = a.out.d_counters;
  m.round = round;
  m.stride = a.w.ctx_cap + 1;
  // one thread per sample of a four-way pass at most
  const uint64_t work = a.w.tiles_cap * kSampPerTile;
  uint64_t blocks = ceil_div(work ? work : 1, 256);
  if (blocks > 2048) blocks = 2048;
  hipLaunchKernelGGL(k_mpart, dim3((uint32_t)blocks), dim3(256), 0, s, m);
  return hipGetLastError();
}

// ----------------------------------------------------------------- merge

// A tile as the merge kernels take it: the slices of the four runs (start,
// length), where the runs end, the output start, the event count and
// whether it starts its segment.
struct Tile {
  uint32_t pos[4], n[4], end[4];
  uint32_t out_pos, cnt, first;
};

// Reads tile k (and the start of tile k + 1).  False if its slices or output
// do not lie inside the merged range, or it holds no event or more than its
// LDS staging takes.
__device__ __forceinline__ bool tile_of(const MergeTask* task, uint64_t k, uint64_t n_tiles,
                                        uint32_t m_end, Tile& tl) {
  const uint4* tp = reinterpret_cast<const uint4*>(task + k);
  const uint4 p = tp[0], h = tp[1], e = tp[2];
  uint4 np = e;
  if (k + 1 < n_tiles) {
    const uint4* tq = reinterpret_cast<const uint4*>(task + k + 1);
    const uint4 qp = tq[0], qh = tq[1];
    if (!qh.y) np = qp;
  }
  const uint32_t ps[4] = {p.x, p.y, p.z, p.w}, es[4] = {e.x, e.y, e.z, e.w};
  const uint32_t ns[4] = {np.x, np.y, np.z, np.w};
  bool ok = true;
  uint32_t cnt = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    ok = ok && ps[q] <= ns[q] && ns[q] <= es[q] && es[q] <= m_end;
    tl.pos[q] = ps[q];
    tl.end[q] = es[q];
    tl.n[q] = ns[q] - ps[q];
    cnt += tl.n[q];
  }
  tl.out_pos = h.x;
  tl.first = h.y;
  tl.cnt = cnt;
  // staged with the second pair from the next multiple of 8 on (stage_tile)
  const uint32_t span = ((tl.n[0] + tl.n[1] + 7u) & ~7u) + tl.n[2] + tl.n[3];
  return ok && cnt > 0 && span <= (uint32_t)kMergeTile && h.x <= m_end && cnt <= m_end - h.x;
}

// Loads this thread's share of a tile's inputs, the four slices one after
// the other (element t + 512 j; past the end: the last element again, never
// stored).
__device__ __forceinline__ void load_tile(const uint64_t* src, const Tile& tl, uint32_t t,
                                          uint64_t* v) {
  const uint32_t c1 = tl.n[0], c2 = c1 + tl.n[1], c3 = c2 + tl.n[2], cnt = tl.cnt;
#pragma unroll
  for (int j = 0; j < kMergeItems; ++j) {
    const uint32_t i0 = t + (uint32_t)j * kMergeThreads;
    const uint32_t i = i0 < cnt ? i0 : cnt - 1;
    const uint32_t at = i < c1 ? tl.pos[0] + i
                        : i < c2 ? tl.pos[1] + (i - c1)
                        : i < c3 ? tl.pos[2] + (i - c2)
                                 : tl.pos[3] + (i - c3);
    v[j] = src[at];
  }
}

// LDS slot of the second pair of runs (C, D) of a tile: the first multiple
// of 8 at or after the end of the first pair (A, B), so that no thread's 8
// outputs of the first stage span both pairs.
__device__ __forceinline__ uint32_t pair2_slot(const Tile& tl) {
  return (tl.n[0] + tl.n[1] + 7u) & ~7u;
}

// Stores a thread's share of the inputs in LDS: A | B, then C | D from
// pair2_slot on.
__device__ __forceinline__ void stage_tile(uint64_t* se, const uint64_t* v, const Tile& tl,
                                           uint32_t t) {
  const uint32_t nx = tl.n[0] + tl.n[1], gap = pair2_slot(tl) - nx;
#pragma unroll
  for (int j = 0; j < kMergeItems; ++j) {
    const uint32_t i = t + (uint32_t)j * kMergeThreads;
    if (i < tl.cnt) se[lpad(i < nx ? i : i + gap)] = v[j];
  }
}

// Merges the runs P = slots [0, na) and Q = [oq, oq + nb) (oq >= na) staged
// in se into 8 consecutive outputs per thread, written back in merged order
// to slots [0, na + nb).  Ends with every thread past the read of its
// inputs; the caller synchronises before reading se.
__device__ __forceinline__ void merge_tile(uint64_t* se, uint32_t na, uint32_t oq, uint32_t nb,
                                           uint32_t t) {
  const uint32_t cnt = na + nb, d = t * kMergeItems;
  uint64_t o[kMergeItems];
#pragma unroll
  for (int j = 0; j < kMergeItems; ++j) o[j] = 0;
  if (d < cnt) {
    uint32_t ia = corank_lds(se, 0, na, oq, nb, d), ib = d - ia;
#pragma unroll
    for (int j = 0; j < kMergeItems; ++j) {
      const uint64_t va = se[lpad(ia)], vb = se[lpad(oq + (ib < nb ? ib : nb))];
      const bool take_a = ia < na && (ib >= nb || mkey(va) <= mkey(vb));
      o[j] = take_a ? va : vb;
      ia += take_a;
      ib += !take_a;
    }
  }
  __syncthreads();  // every thread has read its inputs
#pragma unroll
  for (int j = 0; j < kMergeItems; ++j)
    if (d + (uint32_t)j < cnt) se[lpad(d + j)] = o[j];
}

// First stage of a four-run tile staged by stage_tile: A with B and C with
// D, in place (8 consecutive outputs per thread, each thread in one pair).
// Ends like merge_tile.
__device__ __forceinline__ void merge_pairs(uint64_t* se, const Tile& tl, uint32_t t) {
  const uint32_t y0 = pair2_slot(tl), d = t * kMergeItems;
  const bool second = d >= y0;
  const uint32_t o0 = second ? y0 : 0u, lp = second ? tl.n[2] : tl.n[0];
  const uint32_t lq = second ? tl.n[3] : tl.n[1], dd = d - o0, lim = lp + lq;
  uint64_t o[kMergeItems];
#pragma unroll
  for (int j = 0; j < kMergeItems; ++j) o[j] = 0;
  if (dd < lim) {
    uint32_t ip = corank_lds(se, o0, lp, o0 + lp, lq, dd), iq = dd - ip;
#pragma unroll
    for (int j = 0; j < kMergeItems; ++j) {
      const uint64_t va = se[lpad(o0 + ip)], vb = se[lpad(o0 + lp + (iq < lq ? iq : lq))];
      const bool take_p = ip < lp && (iq >= lq || mkey(va) <= mkey(vb));
      o[j] = take_p ? va : vb;
      ip += take_p;
      iq += !take_p;
    }
  }
  __syncthreads();  // every thread has read its inputs
#pragma unroll
  for (int j = 0; j < kMergeItems; ++j)
    if (dd + (uint32_t)j < lim) se[lpad(d + j)] = o[j];
}

// Both stages on a staged tile (each only where it has two non-empty runs to
// merge; the decision is the same for the whole block), leaving the merged
// tile in slots [0, cnt).  Ends synchronised.
__device__ __forceinline__ void merge_staged(uint64_t* se, const Tile& tl, uint32_t t) {
  const uint32_t nx = tl.n[0] + tl.n[1], ny = tl.n[2] + tl.n[3];
  if ((tl.n[0] && tl.n[1]) || (tl.n[2] && tl.n[3])) {
    merge_pairs(se, tl, t);
    __syncthreads();
  }
  if (nx && ny) {
    merge_tile(se, nx, pair2_slot(tl), ny, t);
    __syncthreads();
  }
}

struct MergeArgs {
  const DevPlan* plan;
  uint64_t* ev[2];
  const MergeTask* task;
  uint64_t* counters;
  int round;
};

// Static tiles (tile = block + k * grid; there is no dependency between
// tiles).  Each tile's input slices go through LDS; each thread finds its
// own split and merges 8 outputs per stage, which are staged in LDS again so
// that the stores are contiguous.  The next tile's task and inputs are
// loaded while the current one is merged.
__global__ __launch_bounds__(kMergeThreads) void k_merge(MergeArgs a) {
  const DevPlan* p = a.plan;
  // the last pass is k_merge_sweep's
  if (!p->ev_merge || (uint32_t)a.round + 1 >= p->m_rounds) return;
  __shared__ uint64_t s_e[kMergeLds];
  const MergeRound mr = p->mr[a.round];
  const uint64_t n_tiles = mr.n_tiles;
  const uint32_t end = (uint32_t)p->m_end;
  const uint64_t* src = a.ev[mr.src];
  uint64_t* dst = a.ev[mr.dst];
  const uint32_t t = threadIdx.x;
  uint64_t k = blockIdx.x;
  if (k >= n_tiles) return;
  Tile tk;
  bool ok = tile_of(a.task, k, n_tiles, end, tk);
  uint64_t v[kMergeItems];
  if (ok) load_tile(src, tk, t, v);
  for (; k < n_tiles; k += gridDim.x) {
    const uint64_t kn = k + gridDim.x;
    Tile tn;
    const bool okn = kn < n_tiles && tile_of(a.task, kn, n_tiles, end, tn);
    if (!ok) {
      if (t == 0) flag_internal_error(a.counters, 256);
    } else {
      const uint32_t cnt = tk.cnt;
      stage_tile(s_e, v, tk, t);
      __syncthreads();
      // the next tile's inputs, in flight during this merge
      if (okn) load_tile(src, tn, t, v);
      merge_staged(s_e, tk, t);
#pragma unroll
      for (int j = 0; j < kMergeItems; ++j) {
        const uint32_t i = t + (uint32_t)j * kMergeThreads;
        if (i < cnt) dst[tk.out_pos + i] = s_e[lpad(i)];
      }
      __syncthreads();
    }
    if (!ok && okn) load_tile(src, tn, t, v);
    tk = tn;
    ok = okn;
  }
}

hipError_t launch_merge(const RunArgs& a, int round, hipStream_t s) {
  MergeArgs m{};
  m.plan = a.w.plan;
  for (int b = 0; b < 2; ++b) m.ev[b] = a.w.key[b];
  m.task = (const MergeTask*)a.w.part;
  m.counters = a.out.d_counters;
  m.round = round;
  uint64_t blocks = a.w.tiles_cap ? a.w.tiles_cap : 1;
  const uint64_t resident = persistent_blocks((const void*)k_merge, kMergeThreads);
  if (blocks > resident) blocks = resident;
  hipLaunchKernelGGL(k_merge, dim3((uint32_t)blocks), dim3(kMergeThreads), 0, s, m);
  return hipGetLastError();
}

// -------------------------------------------------- last pass and the sweep
//
// The last pass's segments are the groups, and it is swept tile by tile as
// it is merged.  A tile cannot know the class counts entering it without
// waiting for the tiles before it, so it records sums from which its share
// of U and Q follows once those counts are known (k_ovt_final).  With the
// tile-local count l (0 before the tile's first event; c = c_in + l) and a
// bias B (l' = l + B >= 0, a = c_in - B, so c = a + l'):
//   Q[x][y] (x != y) = sum gap (a_x + l'_x)(a_y + l'_y)
//                    = S2'[x][y] + a_x S1'[y] + a_y S1'[x] + a_x a_y S0,
//   Q[x][x]          = sum gap C(a_x + l'_x, 2)
//                    = S2'[x][x] + a_x S1'[x] + C(a_x, 2) S0,
// with S0 = sum gap, S1'[x] = sum gap l'_x, S2'[x][y] = sum gap l'_x l'_y,
// S2'[x][x] = sum gap C(l'_x, 2) (all exact integers, then mod 2^64).  Counts
// never go below zero, so with m_x the lowest l_x over the tile, class x is
// active in every gap of the tile when c_in_x + m_x > 0 and exactly where
// l_x > m_x otherwise; T[x] = sum gap [l_x > m_x] and T2[x][y] = sum gap
// [l_x > m_x][l_y > m_y] then give U.  A tile spanning 2^32 cycles or more
// is summed again with 64-bit gaps by a second, rarely busy kernel.

constexpr int32_t kLBias = kMergeTile;  // |l| <= 4096 inside a tile

// Words of one tile record for KC classes: group | first << 32 | wide << 33,
// then per class (delta | min << 32), S0, S1'[KC], S2'[NP], T[NP] (pairs
// x <= y in row order; T[x][x] = T[x], T[x][y] = T2[x][y]).
__host__ __device__ constexpr int tile_rec_words(int kc) { return 2 + 2 * kc + kc * (kc + 1); }

struct MergeSweepArgs {
  const DevPlan* plan;
  const uint64_t* ev[2];
  const MergeTask* task;
  uint64_t* rec;  // [tiles][tile_rec_words(K)]
  uint64_t* counters;
};

// The word that follows a tile in merged order (ties: the earlier run), if
// its segment continues.
__device__ __forceinline__ bool tile_next(const uint64_t* src, const Tile& t, uint64_t* w) {
  bool has = false;
  uint64_t best = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t at = t.pos[q] + t.n[q];
    if (at < t.end[q]) {
      const uint64_t e = src[at];
      if (!has || mkey(e) < mkey(best)) best = e;
      has = true;
    }
  }
  *w = best;
  return has;
}

// Per-thread sums over the merged events at tile positions d .. d + nval - 1
// (staged in se) followed by the word `after` (if has_after).  lp: biased local counts l' before the first
// event; mp: biased tile minima m'.  NARROW (the tile spans less than 2^32
// cycles): gaps, S0, T and T2 fit 32 bits.  l' < 2^14 either way.
// BINS (narrow, at most four classes): instead of summing T and T2 per
// event, each event adds its gap to the thread's bin of the event's set of
// active classes (1 << KC bins in LDS at hb); T and T2 follow from the bins.
template <int KC, bool NARROW, bool BINS>
__device__ __forceinline__ void sweep8(const uint64_t* se, uint32_t d, uint32_t nval, uint64_t after,
                                       bool has_after, const uint32_t (&lp0)[KC],
                                       const uint32_t (&mp)[KC],
                                       typename std::conditional<NARROW, uint32_t, uint64_t>::type (&tt)[1 + KC * (KC + 1) / 2],
                                       uint64_t (&s1)[KC], uint64_t (&s2)[KC * (KC + 1) / 2],
                                       uint32_t* hb) {
  using UT = typename std::conditional<NARROW, uint32_t, uint64_t>::type;
  static_assert(!BINS || (NARROW && KC <= 4), "bins: narrow tiles, at most four classes");
  uint32_t l[KC];
#pragma unroll
  for (int x = 0; x < KC; ++x) l[x] = lp0[x];
  uint64_t cur = se[lpad(d)];
#pragma unroll 1
  for (uint32_t j = 0; j < nval; ++j) {
    const uint32_t code = (uint32_t)(cur & ((1u << kEvCodeBits) - 1u));
    const uint32_t cls = (code - 1u) >> 1;  // >= KC when code == 0
    const uint32_t sg = 1u - 2u * ((code - 1u) & 1u);  // +1 BEGIN, -1 END
#pragma unroll
    for (int x = 0; x < KC; ++x) l[x] += cls == (uint32_t)x ? sg : 0u;
    // gap to the next event of the group (none after the last one)
    const bool inside = j + 1 < nval;
    const bool has_nx = inside || has_after;
    const uint64_t nx = inside ? se[lpad(d + j + 1)] : after;
    UT gap;
    if (NARROW)
      gap = has_nx ? (UT)((uint32_t)(nx >> kEvCodeBits) - (uint32_t)(cur >> kEvCodeBits)) : (UT)0;
    else
      gap = has_nx ? (UT)((nx >> kEvCodeBits) - (cur >> kEvCodeBits)) : (UT)0;
    // tt: S0, then T[x] (x <= y: T2[x][y], x == y: T[x]) in pair order
    tt[0] += gap;
    bool act[KC];
#pragma unroll
    for (int x = 0; x < KC; ++x) {
      act[x] = l[x] > mp[x];
      s1[x] += (uint64_t)gap * l[x];
    }
    int k = 0;
#pragma unroll
    for (int x = 0; x < KC; ++x) {
#pragma unroll
      for (int y = x; y < KC; ++y, ++k) {
        const uint32_t w = x != y ? __umul24(l[x], l[y]) : (__umul24(l[x], l[x] - 1u) >> 1);
        s2[k] += (uint64_t)gap * w;
        if constexpr (!BINS) tt[1 + k] += (act[x] && act[y]) ? gap : (UT)0;
      }
    }
    if constexpr (BINS) {
      uint32_t m = 0;
#pragma unroll
      for (int x = 0; x < KC; ++x) m |= act[x] ? 1u << x : 0u;
      atomicAdd(&hb[m], (uint32_t)gap);  // the thread's own bins: no return value needed
    }
    cur = nx;
  }
}

// Wave sum of a 64-bit value, result in lane 0.
__device__ __forceinline__ uint64_t wave_sum64(uint64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off);
  return v;
}

// The sums of a tile are taken by its first kMsThreads threads, each over
// kMsItems consecutive events: fewer, longer sequential runs mean fewer
// per-thread partial sums to reduce across the block.
constexpr int kMsThreads = 256;
constexpr int kMsItems = kMergeTile / kMsThreads;
static_assert(kMsThreads % 64 == 0 && kMsThreads <= kMergeThreads, "sweep threads");
static_assert(1 + 8 + 8 * 9 < kMsThreads - 1, "one thread per sum, and one for the header");

// LDS of one block of the last pass.
template <int KC>
struct MsShared {
  static constexpr int NW = kMsThreads / 64;
  static constexpr int NV = 1 + KC + KC * (KC + 1);  // S0, S1', S2', T
  int32_t wd[NW][KC];
  int32_t wm[NW][KC];
  uint64_t next;
  uint32_t has_next;
  uint64_t red[NV][NW];
  // activity bins of each sweeping thread (17 words apart: spread over banks)
  static constexpr bool BINS = KC <= 4;
  static constexpr int BW = 17;
  uint32_t bins[BINS ? kMsThreads * BW : 1];
};

// Sums of one merged tile (se, cnt events; ss.next / ss.has_next: the word
// after it) into its record.  Returns false, with only the record's header
// written (wide bit set), when !WIDE and the tile spans 2^32 cycles or more.
template <int KC, bool WIDE>
__device__ __forceinline__ bool tile_sums(const uint64_t* se, uint32_t cnt, bool first,
                                          MsShared<KC>& ss, uint64_t* rec, uint32_t es) {
  constexpr int NP = KC * (KC + 1) / 2;
  constexpr int NW = MsShared<KC>::NW;
  constexpr int NV = MsShared<KC>::NV;
  const uint32_t t = threadIdx.x, lane = t & 63, w = t >> 6;
  const bool sweeper = t < (uint32_t)kMsThreads;
  const uint32_t d = t * kMsItems;
  const uint32_t nval = sweeper && d < cnt ? (cnt - d < (uint32_t)kMsItems ? cnt - d : (uint32_t)kMsItems) : 0u;
  const uint64_t first_w = se[0];
  const bool has_next = ss.has_next != 0;
  const uint64_t last_w = has_next ? ss.next : se[lpad(cnt - 1)];
  const uint64_t g = es >= 64 ? 0ull : (first_w >> es);
  const uint64_t head = (g & 0xFFFFFFFFull) | ((uint64_t)(first ? 1u : 0u) << 32);
  if (!WIDE && ((last_w >> kEvCodeBits) - (first_w >> kEvCodeBits)) >= (1ull << 32)) {
    if (t == 0) rec[0] = head | (1ull << 33);
    return false;
  }
  // ---- class-count deltas of the thread's events and the lowest running
  // count after each of them relative to the thread's start, then the
  // deltas scanned over the block
  int32_t dd[KC], lmin[KC], pre[KC];
#pragma unroll
  for (int x = 0; x < KC; ++x) {
    dd[x] = 0;
    lmin[x] = 0x7FFFFFFF;
  }
#pragma unroll 2
  for (uint32_t j = 0; j < nval; ++j) {
    const uint32_t code = (uint32_t)(se[lpad(d + j)] & ((1u << kEvCodeBits) - 1u));
    const uint32_t cls = (code - 1u) >> 1;
    const int32_t sg = 1 - 2 * (int32_t)((code - 1u) & 1u);
#pragma unroll
    for (int x = 0; x < KC; ++x) {
      dd[x] += cls == (uint32_t)x ? sg : 0;
      lmin[x] = dd[x] < lmin[x] ? dd[x] : lmin[x];
    }
  }
  if (sweeper) {
#pragma unroll
    for (int x = 0; x < KC; ++x) {
      const int32_t inc = wave_incl_scan32(dd[x]);
      pre[x] = inc - dd[x];
      if (lane == 63) ss.wd[w][x] = inc;
    }
  }
  __syncthreads();
  if (sweeper) {
    // ---- tile minima of the local counts (after each event)
#pragma unroll
    for (int x = 0; x < KC; ++x) {
#pragma unroll
      for (int q = 0; q < NW; ++q) pre[x] += q < (int)w ? ss.wd[q][x] : 0;
      const int32_t m0 = nval ? pre[x] + lmin[x] : 0x7FFFFFFF;
      const int32_t m = rows_min32(row_min32(m0));
      if (lane == 0) ss.wm[w][x] = m;
    }
  }
  __syncthreads();
  if (!sweeper) {
    __syncthreads();
    return true;
  }
  uint32_t lp[KC], mp[KC];
#pragma unroll
  for (int x = 0; x < KC; ++x) {
    int32_t m = 0x7FFFFFFF;
#pragma unroll
    for (int q = 0; q < NW; ++q) m = ss.wm[q][x] < m ? ss.wm[q][x] : m;
    lp[x] = (uint32_t)(pre[x] + kLBias);
    mp[x] = (uint32_t)(m + kLBias);
  }
  // ---- sums over this thread's gaps
  const bool has_after = d + kMsItems < cnt || has_next;
  const uint64_t after = d + kMsItems < cnt ? se[lpad(d + kMsItems)] : ss.next;
  using UT = typename std::conditional<WIDE, uint64_t, uint32_t>::type;
  UT tt[1 + NP];
  uint64_t s1[KC], s2[NP];
#pragma unroll
  for (int x = 0; x < 1 + NP; ++x) tt[x] = 0;
#pragma unroll
  for (int x = 0; x < KC; ++x) s1[x] = 0;
#pragma unroll
  for (int x = 0; x < NP; ++x) s2[x] = 0;
  constexpr bool BINS = !WIDE && MsShared<KC>::BINS;
  uint32_t* hb = &ss.bins[BINS ? t * MsShared<KC>::BW : 0];
  if (nval) sweep8<KC, !WIDE, BINS>(se, d, nval, after, has_after, lp, mp, tt, s1, s2, hb);
  if constexpr (BINS) {
    // T[x] (pair x, x) and T2[x][y] from the bins, which are cleared for the
    // next tile
    uint32_t h[1 << KC];
#pragma unroll
    for (int m = 0; m < (1 << KC); ++m) {
      h[m] = hb[m];
      hb[m] = 0;
    }
    int k = 0;
#pragma unroll
    for (int x = 0; x < KC; ++x) {
#pragma unroll
      for (int y = x; y < KC; ++y, ++k) {
        uint32_t v = 0;
#pragma unroll
        for (int m = 0; m < (1 << KC); ++m)
          if (((m >> x) & 1) && ((m >> y) & 1)) v += h[m];
        tt[1 + k] = v;
      }
    }
  }
  // ---- tile totals: waves in registers, then across waves in LDS
  if constexpr (NV <= 32) {
    uint64_t vals[NV];
    vals[0] = (uint64_t)tt[0];
#pragma unroll
    for (int x = 0; x < KC; ++x) vals[1 + x] = s1[x];
#pragma unroll
    for (int x = 0; x < NP; ++x) {
      vals[1 + KC + x] = s2[x];
      vals[1 + KC + NP + x] = (uint64_t)tt[1 + x];
    }
    uint32_t idx;
    const uint64_t r = wave_sums64<NV>(vals, &idx);
    if ((lane & 1u) == 0 && idx < (uint32_t)NV) ss.red[idx][w] = r;
  } else {
    // (rows of 16 lanes, then the four row results as scalars)
    int c = 0;
    // 32-bit sums stay exact per wave in the narrow case: a wave's gaps add
    // up to less than the tile's span
    auto put = [&](uint64_t val, bool narrow32) {
      const uint64_t r = narrow32 ? (uint64_t)rows_sum32(row_sum32((uint32_t)val))
                                  : rows_sum64(row_sum64(val));
      if (lane == 0) ss.red[c][w] = r;
      ++c;
    };
    put((uint64_t)tt[0], !WIDE);
#pragma unroll
    for (int x = 0; x < KC; ++x) put(s1[x], false);
#pragma unroll
    for (int x = 0; x < NP; ++x) put(s2[x], false);
#pragma unroll
    for (int x = 0; x < NP; ++x) put((uint64_t)tt[1 + x], !WIDE);
  }
  __syncthreads();
  if (t < (uint32_t)NV) {
    uint64_t sum = 0;
#pragma unroll
    for (int q = 0; q < NW; ++q) sum += ss.red[t][q];
    rec[1 + KC + t] = sum;
  } else if (t == (uint32_t)kMsThreads - 1) {
    // the tile's count changes and minima, again from the per-wave values
    // (not kept in registers over the sweep)
    rec[0] = head;
#pragma unroll
    for (int x = 0; x < KC; ++x) {
      int32_t agg = 0, mn = 0x7FFFFFFF;
#pragma unroll
      for (int q = 0; q < NW; ++q) {
        agg += ss.wd[q][x];
        mn = ss.wm[q][x] < mn ? ss.wm[q][x] : mn;
      }
      rec[1 + x] = (uint64_t)(uint32_t)agg | ((uint64_t)(uint32_t)mn << 32);
    }
  }
  return true;
}

// The last merge pass fused with the class-overlap sums.  Each tile of at
// most 4096 merged events belongs to one group.  Per tile: merge the input
// slices in LDS (8 consecutive outputs per thread and stage, written back in
// merged order),
// scan the class-count deltas over the block, take the tile minima, and sum
// S0, S1', S2', T over the tile's gaps into the tile's record with its
// deltas and minima.  A tile spanning 2^32 cycles or more only gets its
// record flagged here (k_merge_sweep_wide redoes it).  Tiles are independent
// (tile = block + k * grid); the loads of one block overlap the work of the
// other blocks on its compute unit.
template <int KC, bool WIDE>
__device__ __forceinline__ void merge_sweep_tiles(const MergeSweepArgs& a) {
  constexpr int RW = tile_rec_words(KC);
  const DevPlan* p = a.plan;
  if (!p->ev_merge || p->m_rounds == 0) return;
  __shared__ uint64_t s_e[kMergeLds];
  __shared__ MsShared<KC> ss;
  if constexpr (!WIDE && MsShared<KC>::BINS) {
    if (threadIdx.x < (uint32_t)kMsThreads)
      for (int m = 0; m < MsShared<KC>::BW; ++m) ss.bins[threadIdx.x * MsShared<KC>::BW + m] = 0;
  }
  const MergeRound mr = p->mr[p->m_rounds - 1];
  const uint64_t n_tiles = mr.n_tiles;
  const uint32_t end = (uint32_t)p->m_end;
  const uint32_t es = p->rec.ts_bits + kEvCodeBits;  // group bits start here
  const uint64_t* src = a.ev[mr.src];
  const uint32_t t = threadIdx.x;
  // WIDE: the block first finds the flagged tiles among kMergeThreads tiles
  // (one per thread), then processes them in order
  __shared__ uint32_t s_wide[kMergeThreads];
  __shared__ uint32_t s_nwide;
  const uint64_t step = WIDE ? (uint64_t)gridDim.x * kMergeThreads : (uint64_t)gridDim.x;
  for (uint64_t k0 = WIDE ? (uint64_t)blockIdx.x * kMergeThreads : blockIdx.x; k0 < n_tiles; k0 += step) {
    uint32_t n_here = 1;
    if (WIDE) {
      if (t == 0) s_nwide = 0;
      __syncthreads();
      const uint64_t kt = k0 + t;
      if (kt < n_tiles && ((a.rec[kt * RW] >> 33) & 1u)) s_wide[atomicAdd(&s_nwide, 1u)] = t;
      __syncthreads();
      n_here = s_nwide;
      // the order of the flagged tiles does not matter: each has its own record
    }
    for (uint32_t h = 0; h < n_here; ++h) {
      const uint64_t k = WIDE ? k0 + s_wide[h] : k0;
      uint64_t* rec = a.rec + k * RW;
      Tile tk;
      if (!tile_of(a.task, k, n_tiles, end, tk)) {
        if (WIDE) continue;  // never flagged
        // unusable task: a record that starts a segment and adds nothing
        if (t == 0) flag_internal_error(a.counters, 256);
        if (t < (uint32_t)RW) rec[t] = t == 0 ? (0xFFFFFFFFull | (1ull << 32)) : 0ull;
        continue;
      }
      uint64_t v[kMergeItems];
      load_tile(src, tk, t, v);
      uint64_t nx = 0;
      bool hnx = false;
      if (t == 0) hnx = tile_next(src, tk, &nx);
      const uint32_t cnt = tk.cnt;
      stage_tile(s_e, v, tk, t);
      if (t == 0) {
        ss.next = nx;
        ss.has_next = hnx ? 1u : 0u;
      }
      __syncthreads();
      merge_staged(s_e, tk, t);
      tile_sums<KC, WIDE>(s_e, cnt, tk.first != 0, ss, rec, es);
      __syncthreads();
    }
    if (WIDE) __syncthreads();  // s_wide is rewritten for the next tiles
  }
}

// Up to four classes: six waves per SIMD (three blocks per compute unit; the
// kernel is ALU bound and the extra waves hide the LDS latency).
template <int KC>
__global__ __launch_bounds__(kMergeThreads, KC <= 4 ? 6 : 1) void k_merge_sweep(MergeSweepArgs a) {
  merge_sweep_tiles<KC, false>(a);
}

// Tiles of the last pass flagged as spanning 2^32 cycles or more: merged
// again and summed with 64-bit gaps.
template <int KC>
__global__ __launch_bounds__(kMergeThreads) void k_merge_sweep_wide(MergeSweepArgs a) {
  merge_sweep_tiles<KC, true>(a);
}

// ------------------------------------------------------ tile records → rows

struct OvtArgs {
  const DevPlan* plan;
  const uint64_t* rec;
  int64_t* blk;    // [blocks][1 + K]: reset flag, then the block's count deltas
  uint64_t* ov_u;  // [G][36]
  uint64_t* ov_q;  // [G][36]
  uint64_t* counters;
  uint32_t G;
};

constexpr int kOvtThreads = 256;

// Per block of 256 tile records: whether a segment starts in it, and the
// class-count deltas since the last start (or of the whole block).
template <int KC>
__global__ __launch_bounds__(kOvtThreads) void k_ovt_agg(OvtArgs a) {
  constexpr int RW = tile_rec_words(KC);
  const DevPlan* p = a.plan;
  if (!p->ev_merge || p->m_rounds == 0) return;
  const uint64_t n_tiles = p->mr[p->m_rounds - 1].n_tiles;
  const uint64_t tile = (uint64_t)blockIdx.x * kOvtThreads + threadIdx.x;
  if ((uint64_t)blockIdx.x * kOvtThreads >= n_tiles) return;
  __shared__ uint32_t s_last;
  __shared__ int64_t s_sum[KC];
  if (threadIdx.x == 0) s_last = 0;
  if (threadIdx.x < KC) s_sum[threadIdx.x] = 0;
  __syncthreads();
  const bool in = tile < n_tiles;
  const bool first = in && ((a.rec[tile * RW] >> 32) & 1u);
  if (first) atomicMax(&s_last, threadIdx.x + 1);
  __syncthreads();
  const uint32_t last = s_last;  // 1 + index of the last segment start, or 0
  if (in && threadIdx.x + 1 >= last) {
#pragma unroll
    for (int x = 0; x < KC; ++x) {
      const int32_t dv = (int32_t)(uint32_t)a.rec[tile * RW + 1 + x];
      if (dv) atomicAdd((unsigned long long*)&s_sum[x], (unsigned long long)(int64_t)dv);
    }
  }
  __syncthreads();
  int64_t* b = a.blk + (uint64_t)blockIdx.x * (1 + KC);
  if (threadIdx.x == 0) b[0] = last ? 1 : 0;
  if (threadIdx.x < KC) b[1 + threadIdx.x] = s_sum[threadIdx.x];
}

// Counts entering each tile (a segmented scan over the tile records, the
// carry into a block found by walking back over the block aggregates to the
// nearest segment start), then each tile's share of U and Q added to its
// group's rows.
template <int KC>
__global__ __launch_bounds__(kOvtThreads) void k_ovt_final(OvtArgs a) {
  constexpr int KM = KC <= 2 ? 2 : (KC <= 4 ? 4 : 8);  // stride of the pair index
  constexpr int NP = KC * (KC + 1) / 2;
  constexpr int RW = tile_rec_words(KC);
  const DevPlan* p = a.plan;
  if (!p->ev_merge || p->m_rounds == 0) return;
  const uint64_t n_tiles = p->mr[p->m_rounds - 1].n_tiles;
  const uint64_t blk0 = (uint64_t)blockIdx.x * kOvtThreads;
  if (blk0 >= n_tiles) return;
  const uint32_t t = threadIdx.x, lane = t & 63, w = t >> 6;
  const uint64_t tile = blk0 + t;
  const bool in = tile < n_tiles;
  __shared__ int64_t s_carry[KC];
  __shared__ int64_t s_wsum[kOvtThreads / 64][KC];
  __shared__ uint32_t s_wfirst[kOvtThreads / 64];
  // ---- carry into this block (wave 0): blocks before it back to a reset
  if (w == 0) {
    int64_t acc[KC];
#pragma unroll
    for (int x = 0; x < KC; ++x) acc[x] = 0;
    int64_t top = (int64_t)blockIdx.x - 1;
    while (top >= 0) {
      const int64_t bb = top - (int64_t)lane;
      uint32_t reset = 1;  // before block 0: nothing
      int64_t val[KC];
#pragma unroll
      for (int x = 0; x < KC; ++x) val[x] = 0;
      if (bb >= 0) {
        const int64_t* b = a.blk + (uint64_t)bb * (1 + KC);
        reset = b[0] != 0;
#pragma unroll
        for (int x = 0; x < KC; ++x) val[x] = b[1 + x];
      }
      const uint64_t mr = __ballot(reset);
      const int jr = mr ? __ffsll((unsigned long long)mr) - 1 : 64;  // nearest reset
#pragma unroll
      for (int x = 0; x < KC; ++x) {
        int64_t vv = (int)lane <= jr ? val[x] : 0;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) vv += __shfl_xor(vv, off);
        acc[x] += vv;
      }
      if (jr < 64) break;
      top -= 64;
    }
    if (lane == 0) {
#pragma unroll
      for (int x = 0; x < KC; ++x) s_carry[x] = acc[x];
    }
  }
  // ---- segmented exclusive scan of the tile deltas within the block
  const uint64_t* r = a.rec + tile * RW;
  const bool first = in && ((r[0] >> 32) & 1u);
  int32_t dv[KC];
#pragma unroll
  for (int x = 0; x < KC; ++x) dv[x] = in ? (int32_t)(uint32_t)r[1 + x] : 0;
  // inclusive segmented scan in the wave: (reset, sums)
  uint32_t xr = first ? 1u : 0u;
  int64_t xs[KC];
#pragma unroll
  for (int x = 0; x < KC; ++x) xs[x] = dv[x];
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t yr = __shfl_up(xr, off);
    int64_t ys[KC];
#pragma unroll
    for (int x = 0; x < KC; ++x) ys[x] = __shfl_up(xs[x], off);
    if ((int)lane >= off && !xr) {
      xr = yr;
#pragma unroll
      for (int x = 0; x < KC; ++x) xs[x] += ys[x];
    }
  }
  if (lane == 63) {
    s_wfirst[w] = xr;
#pragma unroll
    for (int x = 0; x < KC; ++x) s_wsum[w][x] = xs[x];
  }
  __syncthreads();
  // exclusive value entering this tile: fold earlier waves and the carry
  int64_t cin[KC];
  {
    // inclusive minus own (own tile resets: nothing enters from before)
    bool reset = xr != 0;
#pragma unroll
    for (int x = 0; x < KC; ++x) cin[x] = xs[x] - dv[x];
    if (first) {
#pragma unroll
      for (int x = 0; x < KC; ++x) cin[x] = 0;
    }
    // a reset inside this wave before (or at) the tile cuts off everything earlier
    if (!reset) {
      for (int q = (int)w - 1; q >= 0; --q) {
#pragma unroll
        for (int x = 0; x < KC; ++x) cin[x] += s_wsum[q][x];
        if (s_wfirst[q]) {
          reset = true;
          break;
        }
      }
      if (!reset) {
#pragma unroll
        for (int x = 0; x < KC; ++x) cin[x] += s_carry[x];
      }
    }
  }
  // ---- this tile's U and Q
  uint64_t uu[NP], qq[NP];
  uint32_t g = 0xFFFFFFFFu;
  if (in) {
    g = (uint32_t)r[0];
    const uint64_t S0 = r[1 + KC];
    const uint64_t* S1 = r + 2 + KC;
    const uint64_t* S2 = r + 2 + 2 * KC;
    const uint64_t* T = r + 2 + 2 * KC + NP;  // pair order; T[x][x] = T[x]
    bool always[KC];
    int64_t av[KC];
#pragma unroll
    for (int x = 0; x < KC; ++x) {
      const int32_t m = (int32_t)(uint32_t)(r[1 + x] >> 32);
      always[x] = cin[x] + m > 0;
      av[x] = cin[x] - kLBias;
    }
    int k = 0;
#pragma unroll
    for (int x = 0; x < KC; ++x) {
#pragma unroll
      for (int y = x; y < KC; ++y, ++k) {
        const uint64_t ax = (uint64_t)av[x], ay = (uint64_t)av[y];
        const uint64_t tx = T[pair_index<KC>(x, x)], ty = T[pair_index<KC>(y, y)];
        if (x == y) {
          uu[k] = always[x] ? S0 : tx;
          const uint64_t cx2 = (uint64_t)((av[x] * (av[x] - 1)) / 2);
          qq[k] = S2[k] + ax * S1[x] + cx2 * S0;
        } else {
          uu[k] = always[x] && always[y] ? S0 : always[x] ? ty : always[y] ? tx : T[k];
          qq[k] = S2[k] + ax * S1[y] + ay * S1[x] + ax * ay * S0;
        }
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      uu[k] = 0;
      qq[k] = 0;
    }
  }
  if constexpr (2 * NP <= 32) {
    // Tiles of one group are adjacent: per group present in the wave, its
    // lanes' values are summed across the wave and added once.
    uint64_t pend = __ballot(in && g < a.G);
    while (pend) {
      const uint32_t gc = (uint32_t)__shfl((int)g, __ffsll((unsigned long long)pend) - 1);
      const uint64_t mine = __ballot(g == gc) & pend;
      pend &= ~mine;
      const bool take = (mine >> lane) & 1ull;
      uint64_t vals[2 * NP];
#pragma unroll
      for (int k = 0; k < NP; ++k) {
        vals[k] = take ? uu[k] : 0ull;
        vals[NP + k] = take ? qq[k] : 0ull;
      }
      uint32_t idx;
      const uint64_t r = wave_sums64<2 * NP>(vals, &idx);
      if ((lane & 1u) == 0 && idx < 2u * NP && r) {
        // pair idx % NP in row order, at its place in a group's rows
        const uint32_t k = idx < (uint32_t)NP ? idx : idx - NP;
        uint32_t pi = 0;
        int kk = 0;
#pragma unroll
        for (int x = 0; x < KC; ++x) {
#pragma unroll
          for (int y = x; y < KC; ++y, ++kk)
            if ((uint32_t)kk == k) pi = (uint32_t)pair_index<KM>(x, y);
        }
        uint64_t* dst = idx < (uint32_t)NP ? a.ov_u : a.ov_q;
        atomicAdd((unsigned long long*)&dst[(uint64_t)gc * kSweepQWords + pi], (unsigned long long)r);
      }
    }
    if (in && g >= a.G && g != 0xFFFFFFFFu) flag_internal_error(a.counters, 256);
    return;
  }
  // whole waves of one group add once; everything else per tile
  const uint32_t g0 = __shfl(g, 0);
  const bool uniform = __ballot(g != g0) == 0ull;
  int k = 0;
#pragma unroll
  for (int x = 0; x < KC; ++x) {
#pragma unroll
    for (int y = x; y < KC; ++y, ++k) {
      uint64_t uv = uu[k], qv = qq[k];
      if (uniform) {
        uv = wave_sum64(uv);
        qv = wave_sum64(qv);
      }
      if ((!uniform || lane == 0) && g < a.G) {
        const uint64_t at = (uint64_t)g * kSweepQWords + (uint64_t)pair_index<KM>(x, y);
        if (uv) atomicAdd((unsigned long long*)&a.ov_u[at], (unsigned long long)uv);
        if (qv) atomicAdd((unsigned long long*)&a.ov_q[at], (unsigned long long)qv);
      }
    }
  }
  if (in && g >= a.G && g != 0xFFFFFFFFu) flag_internal_error(a.counters, 256);
}

#define ARGUS_KC_SWITCH(K, F) \
  ((K) == 1 ? (const void*)F<1> : (K) == 2 ? (const void*)F<2> : (K) == 3 ? (const void*)F<3> : \
   (K) == 4 ? (const void*)F<4> : (K) == 5 ? (const void*)F<5> : (K) == 6 ? (const void*)F<6> : \
   (K) == 7 ? (const void*)F<7> : (const void*)F<8>)

hipError_t launch_merge_sweep(const RunArgs& a, hipStream_t s) {
  MergeSweepArgs m{};
  m.plan = a.w.plan;
  for (int b = 0; b < 2; ++b) m.ev[b] = a.w.key[b];
  m.task = (const MergeTask*)a.w.part;
  m.rec = a.w.mslb;
  m.counters = a.out.d_counters;
  const void* kern = ARGUS_KC_SWITCH(a.K, k_merge_sweep);
  uint64_t blocks = a.w.tiles_cap ? a.w.tiles_cap : 1;
  const uint64_t resident = persistent_blocks(kern, kMergeThreads);
  if (blocks > resident) blocks = resident;
  void* args[] = {&m};
  hipError_t e = hipLaunchKernel(kern, dim3((uint32_t)blocks), dim3(kMergeThreads), args, 0, s);
  if (e != hipSuccess) return e;
  const void* wkern = ARGUS_KC_SWITCH(a.K, k_merge_sweep_wide);
  uint64_t wblocks = a.w.tiles_cap ? a.w.tiles_cap : 1;
  const uint64_t wres = persistent_blocks(wkern, kMergeThreads);
  if (wblocks > wres) wblocks = wres;
  e = hipLaunchKernel(wkern, dim3((uint32_t)wblocks), dim3(kMergeThreads), args, 0, s);
  if (e != hipSuccess) return e;
  OvtArgs o{};
  o.plan = a.w.plan;
  o.rec = a.w.mslb;
  o.blk = (int64_t*)a.w.part;  // the merge tasks are no longer needed
  o.ov_u = a.w.ov_mask;
  o.ov_q = a.w.ov_q;
  o.counters = a.out.d_counters;
  o.G = a.G;
  const uint64_t ob = ceil_div(a.w.tiles_cap ? a.w.tiles_cap : 1, kOvtThreads);
  void* oargs[] = {&o};
  e = hipLaunchKernel(ARGUS_KC_SWITCH(a.K, k_ovt_agg), dim3((uint32_t)ob), dim3(kOvtThreads), oargs, 0, s);
  if (e != hipSuccess) return e;
  return hipLaunchKernel(ARGUS_KC_SWITCH(a.K, k_ovt_final), dim3((uint32_t)ob), dim3(kOvtThreads), oargs, 0, s);
}

}  // namespace argus
