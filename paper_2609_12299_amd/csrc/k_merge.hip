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
// Round b merges, for every prefix ctx >> (b + 1), the run of its contexts
// whose bit b is 0 with the run of those whose bit b is 1; rounds go over
// the bits b in increasing order, and only over bits in which two
// neighbouring contexts of one group first differ (no other bit has a pair to
// merge).  After the last round every group is one run in time order.
//
// A round is three launches: segment boundaries (one block), the merge-path
// split of every output tile (Green, McColl and Bader's merge path: a binary
// search on the cross diagonal), and the merge of each tile's two input
// slices in LDS.
#include "internal.h"

namespace argus {

constexpr uint32_t kNoSplit = 0xFFFFFFFFu;

// ------------------------------------------------------------------ plan

struct MPlanArgs {
  DevPlan* plan;
  const uint2* ctx_list;
  const uint64_t* counters;
  uint32_t K, G, shift;
  uint32_t force_radix;
  uint32_t max_rounds;
  uint64_t ctx_cap;
};

// Chooses between merging and the event radix sort, and plans the rounds.
// Merging applies when the event word (group, timestamp offset, code) fits
// 64 bits, the context list is complete, and the rounds are few enough.
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
  const uint32_t rounds = (uint32_t)__popc(need);
  // A round moves 8 + 8 bytes per event, a radix pass 12 + 12 plus its
  // look-back traffic: merging wins up to about twice as many rounds.
  const uint32_t radix_passes = (g_bits + ks.ts_bits + 7) / 8;
  if (rounds > a.max_rounds || rounds > 2 * radix_passes) return;
  // contexts of groups < G form a prefix of the (sorted) context list
  uint64_t lo = 0, hi = n_ctx;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) / 2;
    const uint32_t c = a.ctx_list[mid].x;
    const uint64_t g = a.shift >= 32 ? 0u : (c >> a.shift);
    if (g < a.G) lo = mid + 1;
    else hi = mid;
  }
  p->m_nctx = (uint32_t)lo;
  p->m_end = lo < n_ctx ? a.ctx_list[lo].y : p->n_valid;
  p->m_rounds = rounds;
  uint32_t buf = p->rec_final ^ 1u, r = 0;
  for (uint32_t b = 0; b < 32; ++b) {
    if (!((need >> b) & 1u)) continue;
    MergeRound& m = p->mr[r++];
    m.bit = b;
    m.src = buf;
    m.dst = buf ^ 1u;
    m.n_segs = 0;
    m.n_tiles = 0;
    buf ^= 1u;
  }
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
              a.shift < (uint32_t)kMaxMergeRounds ? a.shift : (uint32_t)kMaxMergeRounds,
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
  uint32_t* ctx_seg;
  uint32_t* seg_start;
  uint32_t* seg_split;
  uint32_t* seg_tile0;
  uint64_t stride;  // per-round stride of the segment arrays
};

// Segments of every round (block r: round r): maximal runs of contexts with
// equal ctx >> (bit + 1); the split is where bit `bit` becomes 1.  They
// depend on the context list only, so all rounds are planned at once.
__global__ __launch_bounds__(1024) void k_mseg(MSegArgs a) {
  DevPlan* p = a.plan;
  const int round = blockIdx.x;
  if (!p->ev_merge || (uint32_t)round >= p->m_rounds) return;
  a.ctx_seg += round * a.stride;
  a.seg_start += round * a.stride;
  a.seg_split += round * a.stride;
  a.seg_tile0 += round * a.stride;
  __shared__ uint32_t s_w[16];
  const uint32_t bit = p->mr[round].bit;
  const uint32_t nc = p->m_nctx;
  const uint32_t end = (uint32_t)p->m_end;
  const uint32_t t = threadIdx.x;
  auto hi_of = [&](uint32_t c) -> uint32_t { return bit >= 31 ? 0u : (c >> (bit + 1)); };

  uint32_t carry = 0;
  for (uint32_t base = 0; base < nc; base += 1024) {
    const uint32_t j = base + t;
    bool head = false;
    uint2 e = make_uint2(0, 0);
    if (j < nc) {
      e = a.ctx_list[j];
      head = j == 0 || hi_of(a.ctx_list[j - 1].x) != hi_of(e.x);
    }
    uint32_t total;
    const uint32_t incl = block_incl_scan1024(head ? 1u : 0u, s_w, &total);
    if (j < nc) {
      const uint32_t seg = carry + incl - 1;
      a.ctx_seg[j] = seg;
      if (head) {
        a.seg_start[seg] = e.y;
        a.seg_split[seg] = kNoSplit;
      }
    }
    carry += total;
  }
  const uint32_t n_segs = carry;
  __threadfence_block();
  __syncthreads();
  // first context of each segment whose bit is 1
  for (uint32_t j = t; j < nc; j += 1024) {
    const uint2 e = a.ctx_list[j];
    if (!((e.x >> bit) & 1u)) continue;
    bool first1 = j == 0;
    if (!first1) {
      const uint32_t c0 = a.ctx_list[j - 1].x;
      first1 = hi_of(c0) != hi_of(e.x) || !((c0 >> bit) & 1u);
    }
    if (first1) a.seg_split[a.ctx_seg[j]] = e.y;
  }
  __threadfence_block();
  __syncthreads();
  // merge tiles per segment, and their prefix
  carry = 0;
  for (uint32_t base = 0; base < n_segs; base += 1024) {
    const uint32_t sg = base + t;
    uint32_t tiles = 0;
    if (sg < n_segs) {
      const uint32_t s0 = a.seg_start[sg];
      const uint32_t s1 = sg + 1 < n_segs ? a.seg_start[sg + 1] : end;
      if (a.seg_split[sg] == kNoSplit) a.seg_split[sg] = s1;
      tiles = (uint32_t)ceil_div(s1 - s0, kMergeTile);
    }
    uint32_t total;
    const uint32_t incl = block_incl_scan1024(tiles, s_w, &total);
    if (sg < n_segs) a.seg_tile0[sg] = carry + incl - tiles;
    carry += total;
  }
  if (t == 0) {
    a.seg_tile0[n_segs] = carry;
    p->mr[round].n_segs = n_segs;
    p->mr[round].n_tiles = carry;
  }
}

hipError_t launch_mseg(const RunArgs& a, int rounds, hipStream_t s) {
  MSegArgs m{a.w.plan, a.w.ctx_list, a.w.ctx_seg, a.w.seg_start, a.w.seg_split, a.w.seg_tile0,
             a.w.ctx_cap + 1};
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

// One merge tile: where its slices of the two runs start, their lengths,
// and where its output starts (absolute sorted positions).
struct MergeTask {
  uint32_t a_pos, na, b_pos, nb, out_pos, pad0, pad1, pad2;
};

struct MPartArgs {
  const DevPlan* plan;
  const uint64_t* ev[2];
  const uint32_t* seg_start;
  const uint32_t* seg_split;
  const uint32_t* seg_tile0;
  MergeTask* task;
  uint64_t* counters;
  int round;
  uint64_t stride;
};

__global__ __launch_bounds__(256) void k_mpart(MPartArgs a) {
  const DevPlan* p = a.plan;
  if (!p->ev_merge || (uint32_t)a.round >= p->m_rounds) return;
  const MergeRound mr = p->mr[a.round];
  const uint32_t n_segs = (uint32_t)mr.n_segs;
  const uint64_t n_tiles = mr.n_tiles;
  const uint32_t end = (uint32_t)p->m_end;
  const uint64_t* src = a.ev[mr.src];
  const uint64_t off = (uint64_t)a.round * a.stride;
  const uint32_t* seg_start = a.seg_start + off;
  const uint32_t* seg_split = a.seg_split + off;
  const uint32_t* seg_tile0 = a.seg_tile0 + off;
  for (uint64_t k = (uint64_t)blockIdx.x * 256 + threadIdx.x; k < n_tiles;
       k += (uint64_t)gridDim.x * 256) {
    // segment of tile k: the last one whose first tile is <= k
    uint32_t lo = 0, hi = n_segs;
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (seg_tile0[mid] <= k) lo = mid;
      else hi = mid;
    }
    const uint32_t s0 = seg_start[lo], sp = seg_split[lo];
    const uint32_t s1 = lo + 1 < n_segs ? seg_start[lo + 1] : end;
    MergeTask tk{0, 0, 0, 0, 0, 0, 0, 0};
    if (s0 <= sp && sp <= s1 && s1 <= end) {
      const uint32_t L = s1 - s0, la = sp - s0, lb = s1 - sp;
      const uint64_t d0w = (k - seg_tile0[lo]) * (uint64_t)kMergeTile;
      const uint32_t d0 = d0w < L ? (uint32_t)d0w : L;
      const uint32_t d1 = d0 + kMergeTile < L ? d0 + kMergeTile : L;
      const uint64_t* A = src + s0;
      const uint64_t* B = src + sp;
      const uint32_t a0 = corank(A, la, B, lb, d0), a1 = corank(A, la, B, lb, d1);
      tk.a_pos = s0 + a0;
      tk.na = a1 - a0;
      tk.b_pos = sp + (d0 - a0);
      tk.nb = (d1 - a1) - (d0 - a0);
      tk.out_pos = s0 + d0;
    } else {
      flag_internal_error(a.counters, 256);
    }
    a.task[k] = tk;
  }
}

hipError_t launch_mpart(const RunArgs& a, int round, hipStream_t s) {
  MPartArgs m{};
  m.plan = a.w.plan;
  for (int b = 0; b < 2; ++b) m.ev[b] = a.w.key[b];
  m.seg_start = a.w.seg_start;
  m.seg_split = a.w.seg_split;
  m.seg_tile0 = a.w.seg_tile0;
  m.task = (MergeTask*)a.w.part;
  m.counters = a.out.d_counters;
  m.round = round;
  m.stride = a.w.ctx_cap + 1;
  uint64_t blocks = ceil_div(a.w.tiles_cap, 256);
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_mpart, dim3((uint32_t)blocks), dim3(256), 0, s, m);
  return hipGetLastError();
}

// ----------------------------------------------------------------- merge

struct MergeArgs {
  const DevPlan* plan;
  uint64_t* ev[2];
  const MergeTask* task;
  uint64_t* counters;
  int round;
};

// A task is usable if its slices and output lie inside the merged range.
__device__ __forceinline__ bool task_ok(const MergeTask& t, uint32_t end) {
  return t.na + t.nb <= (uint32_t)kMergeTile && t.na + t.nb > 0 && t.a_pos + t.na <= end &&
         t.b_pos + t.nb <= end && t.out_pos + t.na + t.nb <= end;
}

// Loads this thread's share of a tile's inputs (element t + 512 j; past the
// end: the last element again, never stored).
__device__ __forceinline__ void load_task(const uint64_t* src, const MergeTask& tk, uint32_t t,
                                          uint64_t* v) {
  const uint32_t cnt = tk.na + tk.nb;
#pragma unroll
  for (int j = 0; j < kMergeItems; ++j) {
    const uint32_t i0 = t + (uint32_t)j * kMergeThreads;
    const uint32_t i = i0 < cnt ? i0 : cnt - 1;
    v[j] = i < tk.na ? src[tk.a_pos + i] : src[tk.b_pos + (i - tk.na)];
  }
}

// Static tiles (tile = block + k * grid; there is no dependency between
// tiles).  Each tile's two input slices go through LDS; each thread finds
// its own split and merges 8 outputs, which are staged in LDS again so that
// the stores are contiguous.  The next tile's task and inputs are loaded
// while the current one is merged.
__global__ __launch_bounds__(kMergeThreads) void k_merge(MergeArgs a) {
  const DevPlan* p = a.plan;
  if (!p->ev_merge || (uint32_t)a.round >= p->m_rounds) return;
  __shared__ uint64_t s_e[kMergeTile + 1];  // + 1: reads past a run stay inside
  const MergeRound mr = p->mr[a.round];
  const uint64_t n_tiles = mr.n_tiles;
  const uint32_t end = (uint32_t)p->m_end;
  const uint64_t* src = a.ev[mr.src];
  uint64_t* dst = a.ev[mr.dst];
  const uint32_t t = threadIdx.x;
  uint64_t k = blockIdx.x;
  if (k >= n_tiles) return;
  MergeTask tk = a.task[k];
  bool ok = task_ok(tk, end);
  uint64_t v[kMergeItems];
  if (ok) load_task(src, tk, t, v);
  for (; k < n_tiles; k += gridDim.x) {
    const uint64_t kn = k + gridDim.x;
    MergeTask tn{0, 0, 0, 0, 0, 0, 0, 0};
    if (kn < n_tiles) tn = a.task[kn];
    if (!ok) {
      if (t == 0) flag_internal_error(a.counters, 256);
    } else {
      const uint32_t na = tk.na, nb = tk.nb, cnt = na + nb;
#pragma unroll
      for (int j = 0; j < kMergeItems; ++j) {
        const uint32_t i = t + (uint32_t)j * kMergeThreads;
        if (i < cnt) s_e[i] = v[j];
      }
      __syncthreads();
      // the next tile's inputs, in flight during this merge
      const bool okn = kn < n_tiles && task_ok(tn, end);
      if (okn) load_task(src, tn, t, v);
      uint64_t o[kMergeItems];
      const uint32_t d = t * kMergeItems;
      if (d < cnt) {
        const uint64_t* A = s_e;
        const uint64_t* B = s_e + na;
        uint32_t ia = corank(A, na, B, nb, d), ib = d - ia;
#pragma unroll
        for (int j = 0; j < kMergeItems; ++j) {
          const bool take_a = ia < na && (ib >= nb || mkey(A[ia]) <= mkey(B[ib]));
          o[j] = take_a ? A[ia] : B[ib < nb ? ib : nb];
          ia += take_a;
          ib += !take_a;
        }
      }
      __syncthreads();
      if (d < cnt) {
#pragma unroll
        for (int j = 0; j < kMergeItems; ++j)
          if (d + j < cnt) s_e[d + j] = o[j];
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kMergeItems; ++j) {
        const uint32_t i = t + (uint32_t)j * kMergeThreads;
        if (i < cnt) dst[tk.out_pos + i] = s_e[i];
      }
      __syncthreads();
      ok = okn;
    }
    tk = tn;
    if (kn < n_tiles && !ok && task_ok(tn, end)) {
      ok = true;
      load_task(src, tn, t, v);
    }
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

}  // namespace argus
