// k_scope.hip -- iteration ordinals and scoped per-region statistics.
//
// The paper's Section 3.2 separates a region (the code a developer changes)
// from its scope (which dynamic executions are reported: a warp role, an
// iteration window, an SM subset), and Section 3.3 specialises probes to one
// iteration of a loop region.  The iteration of an instance is its ordinal
// among the instances of its context with the same BEGIN region, in
// canonical (context, begin time) order.
//
// Ordinals: the instance array is already ordered by context, so within any
// stretch of it a stable sort by region alone yields (region, context,
// canonical) order, in which the instances of one (context, region) form a
// run; an instance's ordinal among them is its distance from the start of
// its run.  Up to kSoMaxRegions regions, this is done per chunk of 4096
// consecutive instances, in LDS: each chunk's ordinals are exact except for
// the context that enters it from earlier chunks, whose counts per region
// (the carry) come from a scan over the chunks' counts of their last
// context, and are added where the statistics read the ordinals.  With more
// regions the whole array is sorted: an LSD radix sort over the region's
// 8-bit digits (per 4096-element tile a digit histogram, one exclusive scan
// over the digit-major histograms, then a stable scatter that ranks each
// tile's elements with eight ballots per wave), run starts from a wave
// max-scan of the run heads with one binary search per wave for a run that
// began before it, and the ordinals scattered back to canonical order.  The
// scoped statistics are taken in canonical order.
#include <string.h>

#include <algorithm>
#include <mutex>

#include "internal.h"

namespace argus {

constexpr int kScThreads = 256;
constexpr int kScRounds = 16;
constexpr uint32_t kScTile = kScThreads * kScRounds;  // 4096 elements
constexpr uint32_t kScScanBlock = 4096;                // entries per scan block
// Ordinals reach their instances in two steps: (index, ordinal) pairs are
// gathered per bucket of 2^18 consecutive instance indices, then each bucket
// is written by blocks of one XCD, whose L2 holds the bucket's 1 MiB of
// output while they write it.
constexpr uint32_t kOrdBucketBits = 18;
constexpr uint32_t kOrdMaxBuckets = 1u << (31 - kOrdBucketBits);  // instances < 2^31
constexpr uint32_t kOrdSlices = 128;                              // blocks per bucket

// A stable LSD radix sort over 8-bit digits of 16-byte elements (two u64
// words, ping-pong buffers).  The first pass may read the instance array
// instead (word a = BEGIN region, word b = context << 32 | index).
// Device-side state of a sort whose passes on constant digits are skipped:
// over all elements, the OR and the AND of each word (bits where they
// differ mark the digits that vary).  The passes go over word a's bytes
// 0..7, then word b's bytes 4..7, in that order; a pass that runs moves the
// elements to the other buffer, so the buffer a pass reads is the parity of
// the passes before it that run.
struct SortCtl {
  uint64_t or_a, and_a, or_b, and_b;
};

struct SortBufs {
  uint64_t* a[2];
  uint64_t* b[2];
  SortCtl* ctl;    // NULL: every pass runs, buffers as the caller says
  uint32_t* hist;  // [256][tiles_max], digit-major
  uint32_t* bsum;  // scan block sums
  uint64_t tiles_max;
  const uint64_t* count_ptr;  // device element count (clamped to count_max), or NULL
  uint64_t count_max;
  const argus_instance* inst;  // source of the SRC_INST passes
};
enum { kSrcBuf = 0, kSrcInst = 1 };

// A pass whose digit is the same for every element leaves the order as it
// is: it is skipped (its kernels return at once and the buffer stays).
__device__ __forceinline__ bool sb_skip(const SortBufs& s, int word, int shift) {
  if (!s.ctl) return false;
  const uint64_t vary = word ? (s.ctl->or_b ^ s.ctl->and_b) : (s.ctl->or_a ^ s.ctl->and_a);
  return ((vary >> shift) & 0xFFu) == 0;
}
// The buffer holding the elements before the pass on (word, shift) (after
// all passes: word 1, shift 64).
__device__ __forceinline__ int sb_in(const SortBufs& s, int in, int word, int shift) {
  if (!s.ctl) return in;
  const uint64_t va = s.ctl->or_a ^ s.ctl->and_a, vb = s.ctl->or_b ^ s.ctl->and_b;
  int ran = 0;
  for (int sh = 0; sh < 64; sh += 8) {
    if (word == 0 && sh >= shift) break;
    ran += ((va >> sh) & 0xFFu) != 0;
  }
  if (word == 1)
    for (int sh = 32; sh < shift; sh += 8) ran += ((vb >> sh) & 0xFFu) != 0;
  return ran & 1;
}

__device__ __forceinline__ uint64_t sb_count(const SortBufs& s) {
  if (!s.count_ptr) return s.count_max;
  const uint64_t v = *s.count_ptr;
  return v < s.count_max ? v : s.count_max;
}

template <int SRC>
__device__ __forceinline__ void sb_load(const SortBufs& s, int in, uint64_t e, uint64_t* a,
                                        uint64_t* b) {
  if (SRC == kSrcInst) {
    const uint4 h1 = reinterpret_cast<const uint4*>(s.inst)[2 * e + 1];
    *a = h1.w & 0xFFFFu;
    *b = ((uint64_t)h1.x << 32) | e;
  } else {
    *a = s.a[in][e];
    *b = s.b[in][e];
  }
}

// Per tile: counts of each digit, written digit-major (zeros for tiles past
// the element count, so that the scan sees a complete table).
template <int SRC>
__global__ __launch_bounds__(kScThreads) void k_sort_hist(SortBufs s, int in, int word, int shift) {
  __shared__ uint32_t s_cnt[256];
  if (sb_skip(s, word, shift)) return;
  in = sb_in(s, in, word, shift);
  const uint64_t n = sb_count(s);
  const uint64_t tile = blockIdx.x;
  s_cnt[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t base = tile * kScTile;
  for (uint32_t j = 0; j < kScRounds; ++j) {
    const uint64_t e = base + (uint64_t)j * kScThreads + threadIdx.x;
    if (e < n) {
      uint64_t a, b;
      sb_load<SRC>(s, in, e, &a, &b);
      atomicAdd(&s_cnt[((word ? b : a) >> shift) & 0xFFu], 1u);
    }
  }
  __syncthreads();
  s.hist[(uint64_t)threadIdx.x * s.tiles_max + tile] = s_cnt[threadIdx.x];
}

// Exclusive scan of a u32 array in three launches: block sums, their scan
// (one block), then each block's scan plus its base.
__global__ __launch_bounds__(kScThreads) void k_scan_sums(uint32_t* data, uint64_t total,
                                                          uint32_t* bsum) {
  __shared__ uint32_t s_part[kScThreads / 64];
  const uint64_t base = (uint64_t)blockIdx.x * kScScanBlock;
  uint32_t v = 0;
  for (uint32_t j = threadIdx.x; j < kScScanBlock; j += kScThreads)
    if (base + j < total) v += data[base + j];
  v = rows_sum32(row_sum32(v));
  if ((threadIdx.x & 63) == 0) s_part[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) bsum[blockIdx.x] = s_part[0] + s_part[1] + s_part[2] + s_part[3];
}

// Exclusive scan of v over the block; *carry (LDS) holds the running total
// across calls.  Every thread of the block must call it.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* s_w, uint32_t* carry) {
  const uint32_t lane = threadIdx.x & 63, w = threadIdx.x >> 6;
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
  const uint32_t c = *carry;
  __syncthreads();
  if (threadIdx.x == NT - 1) *carry = c + wpre + x;
  __syncthreads();
  return c + wpre + x - v;
}

__global__ __launch_bounds__(1024) void k_scan_top(uint32_t* bsum, uint32_t blocks) {
  __shared__ uint32_t s_carry;
  __shared__ uint32_t s_w[16];
  if (threadIdx.x == 0) s_carry = 0;
  __syncthreads();
  for (uint32_t b0 = 0; b0 < blocks; b0 += 1024) {
    const uint32_t b = b0 + threadIdx.x;
    const uint32_t v = b < blocks ? bsum[b] : 0u;
    const uint32_t ex = block_excl_scan<1024>(v, s_w, &s_carry);
    if (b < blocks) bsum[b] = ex;
  }
}

__global__ __launch_bounds__(kScThreads) void k_scan_apply(uint32_t* data, uint64_t total,
                                                           const uint32_t* bsum) {
  __shared__ uint32_t s_w[kScThreads / 64];
  __shared__ uint32_t s_carry;
  const uint64_t base = (uint64_t)blockIdx.x * kScScanBlock;
  if (threadIdx.x == 0) s_carry = bsum[blockIdx.x];
  __syncthreads();
  for (uint32_t j0 = 0; j0 < kScScanBlock; j0 += kScThreads) {
    const uint64_t i = base + j0 + threadIdx.x;
    const uint32_t v = i < total ? data[i] : 0u;
    const uint32_t ex = block_excl_scan<kScThreads>(v, s_w, &s_carry);
    if (i < total) data[i] = ex;
  }
}

// A small table scanned by one block: staged in LDS with coalesced loads,
// each of 1024 threads sums a stretch of consecutive entries, one block scan
// places the stretches, each thread writes its stretch's exclusive prefixes
// in LDS, and the table goes back with coalesced stores.
constexpr uint64_t kScSmallMax = 32768;
__global__ __launch_bounds__(1024) void k_scan_small(uint32_t* data, uint64_t total, SortBufs s,
                                                     int word, int shift) {
  __shared__ uint32_t s_d[kScSmallMax];
  __shared__ uint32_t s_carry;
  __shared__ uint32_t s_w[16];
  if (sb_skip(s, word, shift)) return;  // the digit table of a skipped pass
  const uint32_t t = threadIdx.x, n = (uint32_t)total;
  for (uint32_t i = t; i < n; i += 1024) s_d[i] = data[i];
  if (t == 0) s_carry = 0;
  __syncthreads();
  const uint32_t per = (n + 1023) / 1024, b = t * per;
  uint32_t v = 0;
  for (uint32_t k = 0; k < per; ++k)
    if (b + k < n) v += s_d[b + k];
  uint32_t run = block_excl_scan<1024>(v, s_w, &s_carry);
  for (uint32_t k = 0; k < per; ++k) {
    if (b + k >= n) break;
    const uint32_t d = s_d[b + k];
    s_d[b + k] = run;
    run += d;
  }
  __syncthreads();
  for (uint32_t i = t; i < n; i += 1024) data[i] = s_d[i];
}

// Stable scatter of one tile.  Each wave takes 1024 consecutive elements
// (16 rounds of 64 lanes, all loaded up front) and ranks each among the
// wave's earlier elements of its digit: eight ballots find the lanes that
// share it, and per-wave digit counters in LDS carry the earlier rounds
// (wave barriers only).  One block barrier later the waves' counts give
// each digit's offset per wave and the tile-local digit starts; the tile is
// staged in LDS in digit order and written out so that a run of equal
// digits goes to consecutive addresses.
constexpr size_t kScStageBytes = 2 * sizeof(uint64_t) * kScTile;  // dynamic LDS of k_sort_scatter
template <int SRC>
__global__ __launch_bounds__(kScThreads) void k_sort_scatter(SortBufs s, int in, int out, int word,
                                                             int shift) {
  if (sb_skip(s, word, shift)) return;
  in = sb_in(s, in, word, shift);
  out = s.ctl ? in ^ 1 : out;
  extern __shared__ __align__(16) uint8_t sc_stage[];
  uint64_t* s_ta = reinterpret_cast<uint64_t*>(sc_stage);
  uint64_t* s_tb = s_ta + kScTile;
  __shared__ uint32_t s_wave[4][256];  // per-wave digit counts, then each wave's offset in the digit
  __shared__ uint32_t s_base[256];
  __shared__ uint32_t s_lstart[256];
  __shared__ uint32_t s_w[kScThreads / 64];
  __shared__ uint32_t s_carry;
  const uint64_t n = sb_count(s);
  const uint64_t tile = blockIdx.x;
  const uint32_t tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
#pragma unroll
  for (int q = 0; q < 4; ++q) s_wave[q][tid] = 0;
  s_base[tid] = s.hist[(uint64_t)tid * s.tiles_max + tile];
  if (tid == 0) s_carry = 0;
  uint64_t av[kScRounds], bv[kScRounds];
  uint32_t dg[kScRounds], rk[kScRounds];
  const uint64_t e0 = tile * kScTile + (uint64_t)w * (kScRounds * 64) + lane;
#pragma unroll
  for (int r = 0; r < kScRounds; ++r) {
    const uint64_t e = e0 + (uint64_t)r * 64;
    av[r] = 0;
    bv[r] = 0;
    if (e < n) sb_load<SRC>(s, in, e, &av[r], &bv[r]);
  }
  __syncthreads();  // counters cleared
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int r = 0; r < kScRounds; ++r) {
    const bool valid = e0 + (uint64_t)r * 64 < n;
    const uint32_t d = (uint32_t)(((word ? bv[r] : av[r]) >> shift) & 0xFFu);
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t bal = __ballot((d >> bit) & 1u);
      peers &= ((d >> bit) & 1u) ? bal : ~bal;
    }
    uint32_t rank = 0;
    if (valid) {
      const uint32_t old = s_wave[w][d];
      rank = old + (uint32_t)__popcll(peers & lt);
      __builtin_amdgcn_wave_barrier();
      if ((peers >> lane) == 1ull) s_wave[w][d] = old + (uint32_t)__popcll(peers);
    }
    __builtin_amdgcn_wave_barrier();
    dg[r] = valid ? d : 256u;
    rk[r] = rank;
  }
  __syncthreads();
  // thread tid owns digit tid: the waves' offsets within it, the tile's count
  // of it, and (scanned) where it starts in the staged tile
  uint32_t cnt = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t c = s_wave[q][tid];
    s_wave[q][tid] = cnt;
    cnt += c;
  }
  s_lstart[tid] = block_excl_scan<kScThreads>(cnt, s_w, &s_carry);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kScRounds; ++r) {
    const uint32_t d = dg[r];
    if (d >= 256u) continue;
    const uint32_t slot = s_lstart[d] + s_wave[w][d] + rk[r];
    if (slot < kScTile) {
      s_ta[slot] = av[r];
      s_tb[slot] = bv[r];
    }
  }
  __syncthreads();
  const uint32_t total = s_carry;  // the tile's elements
  uint64_t* da = s.a[out];
  uint64_t* db = s.b[out];
  for (uint32_t i = tid; i < total && i < kScTile; i += kScThreads) {
    const uint64_t a = s_ta[i], b = s_tb[i];
    const uint32_t d = (uint32_t)(((word ? b : a) >> shift) & 0xFFu);
    const uint64_t dst = (uint64_t)s_base[d] + (i - s_lstart[d]);
    if (dst < n) {
      da[dst] = a;
      db[dst] = b;
    }
  }
}

// Scope counters: slot 7 holds internal-error bits (zero unless a
// consistency check inside the library fails).
__device__ __forceinline__ void sc_flag(uint64_t* counters, uint64_t code) {
  atomicOr((unsigned long long*)&counters[ARGUS_SC_INTERNAL], (unsigned long long)code);
}

// Chunk-local ordinals (up to kSoMaxRegions regions).
constexpr uint32_t kSoMaxRegions = 4096;
constexpr uint32_t kSoCont = 1;    // the chunk's last context continues into the next chunk
constexpr uint32_t kSoWhole = 2;   // the chunk holds one context
constexpr uint32_t kSoPcont = 4;   // the chunk's first context began in an earlier chunk
constexpr uint32_t kSoPending = 0x80000000u;  // ordinal still lacks its chunk's carry
constexpr uint32_t kSoSeg = 256;   // chunks per segment of the carry scan

struct ScopeArgs {
  const argus_instance* inst;
  const uint64_t* excl;
  uint32_t R;
  argus_scope sc;
  const uint8_t* region_mask;
  uint32_t* ordinal;
  uint64_t* stats;
  uint64_t* counters;
  SortBufs s;         // count = the instances
  uint32_t* octr;     // [kOrdMaxBuckets] pairs gathered per bucket so far
  uint64_t* pairs;    // [count] ordinal << 32 | index, by bucket (a free sort buffer)
  uint32_t* hkey;     // [count] histogram key of each instance (a free sort buffer)
  // chunk-local ordinals
  uint32_t fast;      // 1: k_so_local wrote the ordinals; k_sc_stats adds the carries
  uint32_t* tail;     // [chunks][R] counts of the chunk's last context per region, then
                      // the carry entering each chunk whose first context began earlier
  uint32_t* cflag;    // [chunks] kSoCont | kSoWhole | kSoPcont
  uint32_t* segb;     // [segments][R] segment composites, then the carry entering each
  uint32_t* segm;     // [segments] 1: the segment passes its entering carry on
};

// Fill kernel for the outputs that are accumulated.
__global__ __launch_bounds__(kScThreads) void k_sc_init(ScopeArgs a) {
  const uint64_t total = (uint64_t)a.R * ARGUS_RS_WIDTH;
  for (uint64_t i = (uint64_t)blockIdx.x * kScThreads + threadIdx.x; i < total;
       i += (uint64_t)gridDim.x * kScThreads) {
    const uint32_t col = (uint32_t)(i % ARGUS_RS_WIDTH);
    a.stats[i] = (col == ARGUS_RS_INCL_MIN || col == ARGUS_RS_EXCL_MIN) ? kU64Max : 0ull;
  }
  if (blockIdx.x == 0 && threadIdx.x < ARGUS_SC_NUM_COUNTERS) a.counters[threadIdx.x] = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * kScThreads + threadIdx.x; i < kOrdMaxBuckets;
       i += (uint64_t)gridDim.x * kScThreads)
    a.octr[i] = 0;
}

// Start of the (key, ctx) run that holds sorted element e, by one wave:
// lane k probes e - 2^k (one round trip brackets the start), then 64 probes
// per step narrow the bracket.
__device__ __forceinline__ uint64_t run_start_wave(const uint64_t* ka, const uint64_t* kb, uint64_t e,
                                                   uint64_t key, uint32_t ctx) {
  const uint32_t lane = threadIdx.x & 63;
  auto same = [&](uint64_t p) { return ka[p] == key && (uint32_t)(kb[p] >> 32) == ctx; };
  // p = e - 2^lane; "outside" when p < 0 or its element is of another run
  const bool in = lane < 63 && (1ull << lane) <= e && same(e - (1ull << lane));
  const uint64_t out = __ballot(!in);
  const uint32_t j = (uint32_t)__ffsll((unsigned long long)out) - 1;  // first lane outside
  if (j == 0) return e;  // e - 1 is outside: e starts its run
  // the start lies in (e - 2^j, e - 2^(j-1)]: the first position whose element is in the run
  uint64_t lo = (1ull << j) <= e ? e - (1ull << j) + 1 : 0;  // lo .. hi may hold the start
  uint64_t hi = e - (1ull << (j - 1));
  while (lo < hi) {
    const uint64_t span = hi - lo;
    const uint64_t p = lo + span * lane / 64;
    const bool ok = same(p);
    // the smallest probe inside the run bounds the start from above; the
    // largest probe outside from below
    const uint64_t ins = __ballot(ok);
    const uint64_t outs = __ballot(!ok);
    if (ins) {
      const uint32_t f = (uint32_t)__ffsll((unsigned long long)ins) - 1;
      const uint64_t pf = lo + span * f / 64;
      uint64_t nlo = lo;
      if (outs & ((1ull << f) - 1ull)) {
        const uint32_t g = 63u - (uint32_t)__clzll(outs & ((1ull << f) - 1ull));
        nlo = lo + span * g / 64 + 1;
      }
      lo = nlo;
      hi = pf;
    } else {
      lo = lo + span * 63 / 64 + 1;
    }
  }
  return lo;
}

// Ordinal of each sorted element: its distance from the start of its
// (region, context) run.  A block takes 4096 sorted elements (16 rounds of
// 64 per wave, chunk c = 4 * round + wave).  The start of a run that began
// before an element's chunk is the last head of the chunks before it, or
// (before the tile's first head) the start of the run holding the tile's
// first element.  The (index, ordinal) pairs go to the buckets of their
// indices, each block reserving its share of a bucket once.
__global__ __launch_bounds__(kScThreads) void k_sc_ordinal(ScopeArgs a, int buf) {
  __shared__ uint32_t s_cnt[kOrdMaxBuckets];  // per bucket: count, then global base
  __shared__ int64_t s_last[4 * kScRounds];   // last head in each chunk, then the run start entering it
  __shared__ uint64_t s_tstart;
  const uint64_t n = sb_count(a.s);
  const uint64_t* ka = a.s.a[buf];
  const uint64_t* kb = a.s.b[buf];
  const uint32_t tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t nbk = (uint32_t)((n + (1ull << kOrdBucketBits) - 1) >> kOrdBucketBits);
  uint32_t best = 0;
  for (uint64_t tile = blockIdx.x; tile * kScTile < n; tile += gridDim.x) {
    const uint64_t t0 = tile * kScTile;
    for (uint32_t b = tid; b < nbk; b += kScThreads) s_cnt[b] = 0;
    if (w == 0) {
      const uint64_t st = run_start_wave(ka, kb, t0, ka[t0], (uint32_t)(kb[t0] >> 32));
      if (lane == 0) s_tstart = st;
    }
    // heads, and the last head at or before each lane within its chunk
    int64_t h[kScRounds];
    uint32_t idx[kScRounds];
#pragma unroll
    for (int r = 0; r < kScRounds; ++r) {
      const uint64_t e = t0 + (uint64_t)r * kScThreads + (uint64_t)w * 64 + lane;
      const bool valid = e < n;
      bool head = false;
      idx[r] = 0xFFFFFFFFu;
      if (valid) {
        const uint64_t key = ka[e];
        const uint64_t vv = kb[e];
        idx[r] = (uint32_t)vv;
        head = e == 0 || ka[e - 1] != key || (uint32_t)(kb[e - 1] >> 32) != (uint32_t)(vv >> 32);
      }
      int64_t x = head ? (int64_t)e : -1;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int64_t o = __shfl_up(x, d);
        if (lane >= (uint32_t)d && o > x) x = o;
      }
      h[r] = x;
      if (lane == 63) s_last[4 * r + w] = x;
    }
    __syncthreads();
    if (tid == 0) {
      int64_t run = (int64_t)s_tstart;
      for (uint32_t c = 0; c < 4 * kScRounds; ++c) {
        const int64_t l = s_last[c];
        s_last[c] = run;  // the run start entering chunk c
        if (l >= 0) run = l;
      }
    }
    __syncthreads();
    uint64_t pr[kScRounds];
    uint32_t bk[kScRounds], slot[kScRounds];
#pragma unroll
    for (int r = 0; r < kScRounds; ++r) {
      const uint64_t e = t0 + (uint64_t)r * kScThreads + (uint64_t)w * 64 + lane;
      bk[r] = 0xFFFFFFFFu;
      if (e >= n) continue;
      const int64_t hs = h[r] >= 0 ? h[r] : s_last[4 * r + w];
      if (idx[r] < n && hs >= 0 && (uint64_t)hs <= e) {
        const uint32_t ord = (uint32_t)(e - (uint64_t)hs);
        best = best > ord + 1 ? best : ord + 1;
        bk[r] = idx[r] >> kOrdBucketBits;
        slot[r] = atomicAdd(&s_cnt[bk[r]], 1u);
        pr[r] = ((uint64_t)ord << 32) | idx[r];
      } else {
        sc_flag(a.counters, 1);
      }
    }
    __syncthreads();
    for (uint32_t b = tid; b < nbk; b += kScThreads) {
      const uint32_t c = s_cnt[b];
      if (c) s_cnt[b] = atomicAdd(&a.octr[b], c);
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kScRounds; ++r) {
      if (bk[r] == 0xFFFFFFFFu) continue;
      const uint64_t at = ((uint64_t)bk[r] << kOrdBucketBits) + s_cnt[bk[r]] + slot[r];
      if (at < n) a.pairs[at] = pr[r];
      else sc_flag(a.counters, 1);
    }
    __syncthreads();
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

// Each bucket's pairs written to their instances: block k serves XCD k % 8
// (blocks are dispatched to XCDs round-robin), buckets b with b % 8 == k % 8,
// one of kOrdSlices slices of the bucket each.
__global__ __launch_bounds__(kScThreads) void k_sc_ord_place(ScopeArgs a) {
  const uint64_t n = sb_count(a.s);
  const uint32_t k = blockIdx.x, x = k % 8, j = k / 8;
  const uint64_t b = x + 8ull * (j / kOrdSlices);
  const uint32_t sl = j % kOrdSlices;
  const uint64_t b0 = b << kOrdBucketBits;
  if (b0 >= n) return;
  const uint64_t size = n - b0 < (1ull << kOrdBucketBits) ? n - b0 : (1ull << kOrdBucketBits);
  const uint64_t lo = b0 + size * sl / kOrdSlices, hi = b0 + size * (sl + 1) / kOrdSlices;
  for (uint64_t i = lo + threadIdx.x; i < hi; i += kScThreads) {
    const uint64_t pr = a.pairs[i];
    const uint32_t idx = (uint32_t)pr;
    if (idx >= b0 && idx < b0 + size) a.ordinal[idx] = (uint32_t)(pr >> 32);
    else sc_flag(a.counters, 1);
  }
}


// Inclusive maximum over the wave (unsigned; lanes past a row edge see 0).
__device__ __forceinline__ uint32_t wave_incl_max32(uint32_t v) {
  v = max(v, dpp32<kDppRowShr + 1>(v));
  v = max(v, dpp32<kDppRowShr + 2>(v));
  v = max(v, dpp32<kDppRowShr + 4>(v));
  v = max(v, dpp32<kDppRowShr + 8>(v));
  v = max(v, dpp32<kDppBcast15, 0xA>(v));
  v = max(v, dpp32<kDppBcast31, 0xC>(v));
  return v;
}

// Ordinals of one chunk of 4096 consecutive instances, exact except for the
// context that entered the chunk from earlier ones (those are written with
// kSoPending and completed in k_sc_stats), and, when the chunk's last
// context continues into the next chunk, that context's counts per region.
// One wave per chunk walks it in order, 64 elements per round.  An element's
// local ordinal is the count its (context, region) reached before the round,
// kept per region in the wave's LDS row, plus its rank among the lanes of
// the round with the same context and region (contexts are contiguous, so
// the lanes of one context form a range; the region by one ballot per
// region bit).  A counter keeps the chunk position where its context starts
// beside the count, so a context that starts inside the chunk counts from
// zero.  The loads of kSoBatch rounds are issued together.
constexpr int kSoBatch = 16;

__global__ __launch_bounds__(kScThreads) void k_so_local(ScopeArgs a) {
  extern __shared__ uint32_t so_cnt[];  // [4 waves][R]: context start << 16 | count
  const uint64_t n = sb_count(a.s);
  const uint4* inst = reinterpret_cast<const uint4*>(a.inst);
  const uint32_t w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  uint32_t* cr = so_cnt + (uint64_t)w * a.R;
  const uint32_t rbits = a.R > 1 ? 32u - (uint32_t)__clz(a.R - 1) : 1u;
  const uint64_t lt = lanemask_lt();
  const uint64_t above = lane == 63 ? 0ull : (~0ull << (lane + 1));  // lanes after this one
  const uint64_t chunks = (n + kScTile - 1) / kScTile;
  bool bad = false;
  for (uint64_t c = (uint64_t)blockIdx.x * 4 + w; c < chunks; c += (uint64_t)gridDim.x * 4) {
    const uint64_t base = c * kScTile;
    const uint32_t cnt = n - base < (uint64_t)kScTile ? (uint32_t)(n - base) : kScTile;
    // the chunk's first and last contexts and their neighbours outside it
    const uint32_t F = inst[2 * base + 1].x, L = inst[2 * (base + cnt - 1) + 1].x;
    const uint32_t ctx_before = inst[2 * (base > 0 ? base - 1 : 0) + 1].x;
    const uint32_t ctx_after = inst[2 * (base + cnt < n ? base + cnt : base) + 1].x;
    uint32_t f = F == L ? kSoWhole : 0u;
    if (base > 0 && ctx_before == F) f |= kSoPcont;
    if (base + cnt < n && ctx_after == L) f |= kSoCont;
    if (lane == 0) a.cflag[c] = f;
    for (uint32_t r = lane; r < a.R; r += 64) cr[r] = 0;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    uint32_t seg1 = 0;  // 1 + the context start of the element before the round
    uint32_t pctx = F;  // the context of that element (the first element starts one anyway)
    for (uint32_t b0 = 0; b0 < cnt; b0 += 64u * kSoBatch) {
      uint32_t cx[kSoBatch], rw[kSoBatch];
#pragma unroll
      for (int k = 0; k < kSoBatch; ++k) {
        const uint32_t e = b0 + 64u * k + lane;
        const uint4 h1 = inst[2 * (base + (e < cnt ? e : cnt - 1)) + 1];
        cx[k] = h1.x;
        rw[k] = h1.w;
      }
#pragma unroll
      for (int k = 0; k < kSoBatch; ++k) {
        const uint32_t r0 = b0 + 64u * k;  // the round's first element
        if (r0 < cnt) {
        const uint32_t e = r0 + lane;
        const bool in = e < cnt;
        const uint32_t ctx = cx[k], reg = rw[k] & 0xFFFFu;
        bad |= in && reg >= a.R;
        const bool ok = in && reg < a.R;
        const bool head = in && (e == 0 || lane_prev(ctx, pctx) != ctx);
        uint32_t x = wave_incl_max32(head ? e + 1 : 0u);
        x = x > seg1 ? x : seg1;
        const uint32_t seg = x - 1u;  // where this element's context starts in the chunk
        seg1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
        pctx = (uint32_t)__builtin_amdgcn_readlane((int)ctx, 63);
        // the lanes of this context in the round, then those of this region
        const uint64_t nxt = __ballot(head) & above;
        const uint32_t hi = nxt ? (uint32_t)__builtin_ctzll(nxt) : 64u;
        const uint32_t lo = seg > r0 ? seg - r0 : 0u;
        uint64_t peers = __ballot(ok) & (hi == 64u ? ~0ull : ((1ull << hi) - 1ull)) & (~0ull << lo);
        for (uint32_t bit = 0; bit < rbits; ++bit) {
          const bool set = (reg >> bit) & 1u;
          const uint64_t bal = __ballot(set);
          peers &= set ? bal : ~bal;
        }
        const uint32_t rc = ok ? reg : 0u;
        const uint32_t ent = ok ? cr[rc] : 0u;
        const uint32_t prior = (ent >> 16) == seg ? (ent & 0xFFFFu) : 0u;
        const uint32_t local = ok ? prior + (uint32_t)__popcll(peers & lt) : 0u;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // the last lane of each (context, region) group carries its count on
        if (ok && (peers >> lane) == 1ull) cr[rc] = (seg << 16) | (prior + (uint32_t)__popcll(peers));
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (in) {
          // the chunk's first context starts at position 0
          const bool pending = (f & kSoPcont) && seg == 0;
          a.ordinal[base + e] = pending ? (kSoPending | local) : local;
        }
        }
      }
    }
    if (f & kSoCont) {
      // the last context's counts (its start: the last element's)
      const uint32_t ls = seg1 - 1u;
      uint32_t* tail = a.tail + c * (uint64_t)a.R;
      for (uint32_t r = lane; r < a.R; r += 64) {
        const uint32_t ent = cr[r];
        tail[r] = (ent >> 16) == ls ? (ent & 0xFFFFu) : 0u;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();  // the row is cleared for the next chunk after these reads
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  if (__ballot(bad) && lane == 0) sc_flag(a.counters, 2);  // regions must lie below num_regions
}

__device__ __forceinline__ uint64_t so_chunks(uint64_t n) { return (n + kScTile - 1) / kScTile; }

// The carry entering chunk c (per region): x_{c+1} = m_c x_c + b_c, with
// m_c = 1 when the chunk is one context that continues from the chunk before
// and into the next, b_c = the chunk's last-context counts when that context
// continues (else 0); x_0 = 0.  A three-phase scan: the composite of each
// segment of kSoSeg chunks, a sequential pass over the segments per region,
// then each segment's carries.
__global__ __launch_bounds__(kScThreads) void k_so_seg(ScopeArgs a) {
  const uint64_t chunks = so_chunks(sb_count(a.s));
  const uint64_t nseg = (chunks + kSoSeg - 1) / kSoSeg;
  const uint64_t i = (uint64_t)blockIdx.x * kScThreads + threadIdx.x;
  const uint64_t sg = i / a.R;
  const uint32_t r = (uint32_t)(i % a.R);
  if (sg >= nseg) return;
  uint32_t M = 1, B = 0;
  const uint64_t c1 = (sg + 1) * kSoSeg < chunks ? (sg + 1) * kSoSeg : chunks;
  // branch-free steps, eight chunks' loads at a time (a count slot of a chunk
  // whose last context ends in it holds no count and is not used)
  for (uint64_t c0 = sg * kSoSeg; c0 < c1; c0 += 8) {
    uint32_t f[8], t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint64_t c = c0 + u;
      f[u] = c < c1 ? a.cflag[c] : kSoCont | kSoWhole | kSoPcont;
      t[u] = c < c1 ? a.tail[c * a.R + r] : 0u;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t tv = (f[u] & kSoCont) ? t[u] : 0u;
      const bool keep = (f[u] & (kSoCont | kSoWhole | kSoPcont)) == (kSoCont | kSoWhole | kSoPcont);
      M = keep ? M : 0u;
      B = keep ? B + tv : tv;
    }
  }
  a.segb[sg * a.R + r] = B;
  if (r == 0) a.segm[sg] = M;
}

__global__ __launch_bounds__(kScThreads) void k_so_top(ScopeArgs a) {
  const uint64_t chunks = so_chunks(sb_count(a.s));
  const uint64_t nseg = (chunks + kSoSeg - 1) / kSoSeg;
  const uint32_t r = blockIdx.x * kScThreads + threadIdx.x;
  if (r >= a.R) return;
  uint32_t X = 0;
  for (uint64_t sg = 0; sg < nseg; ++sg) {
    const uint32_t B = a.segb[sg * a.R + r];
    a.segb[sg * a.R + r] = X;  // the carry entering the segment
    X = a.segm[sg] ? X + B : B;
  }
}

__global__ __launch_bounds__(kScThreads) void k_so_down(ScopeArgs a) {
  const uint64_t chunks = so_chunks(sb_count(a.s));
  const uint64_t nseg = (chunks + kSoSeg - 1) / kSoSeg;
  const uint64_t i = (uint64_t)blockIdx.x * kScThreads + threadIdx.x;
  const uint64_t sg = i / a.R;
  const uint32_t r = (uint32_t)(i % a.R);
  if (sg >= nseg) return;
  uint32_t x = a.segb[sg * a.R + r];
  const uint64_t c1 = (sg + 1) * kSoSeg < chunks ? (sg + 1) * kSoSeg : chunks;
  for (uint64_t c0 = sg * kSoSeg; c0 < c1; c0 += 8) {
    uint32_t f[8], t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint64_t c = c0 + u;
      f[u] = c < c1 ? a.cflag[c] : 0u;
      t[u] = c < c1 ? a.tail[c * a.R + r] : 0u;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint64_t c = c0 + u;
      if (f[u] & kSoPcont) a.tail[c * a.R + r] = x;  // the carry entering chunk c
      const uint32_t tv = (f[u] & kSoCont) ? t[u] : 0u;
      const bool keep = (f[u] & (kSoCont | kSoWhole | kSoPcont)) == (kSoCont | kSoWhole | kSoPcont);
      x = keep ? x + tv : tv;
    }
  }
}

__device__ __forceinline__ bool in_range32(uint64_t v, uint32_t lo, uint32_t hi) {
  return lo <= v && v <= hi;
}

// Scoped statistics in canonical order.  With LDS_ROWS, each block keeps
// the twelve scalar columns of every region in LDS (LDS atomics), and adds
// them to the output once at the end; without, every column goes straight
// to the output with global atomics.  The histograms are counted afterwards
// from one key per instance (k_hist over slices of regions).
constexpr uint32_t kScLdsRegions = 1024;  // 12 x 8 B x 1024 = 96 KiB of LDS
constexpr int kScStatThreads = 1024;
constexpr int kScCols = 12;               // ARGUS_RS_COUNT .. ARGUS_RS_SELF_NESTED
constexpr int kScStatItems = 2;           // instances per thread and step

template <bool LDS_ROWS>
__global__ __launch_bounds__(kScStatThreads) void k_sc_stats(ScopeArgs a) {
  extern __shared__ __align__(16) uint8_t sc_smem[];
  unsigned long long* srow = reinterpret_cast<unsigned long long*>(sc_smem);
  const uint64_t n = sb_count(a.s);
  const uint4* inst = reinterpret_cast<const uint4*>(a.inst);
  if (LDS_ROWS) {
    for (uint32_t i = threadIdx.x; i < a.R * kScCols; i += kScStatThreads) {
      const uint32_t col = i % kScCols;
      srow[i] = (col == ARGUS_RS_INCL_MIN || col == ARGUS_RS_EXCL_MIN) ? ~0ull : 0ull;
    }
    __syncthreads();
  }
  auto col_ptr = [&](uint32_t reg, uint32_t col) -> unsigned long long* {
    return LDS_ROWS ? &srow[(uint64_t)reg * kScCols + col]
                    : (unsigned long long*)(a.stats + (uint64_t)reg * ARGUS_RS_WIDTH + col);
  };
  uint32_t c_in = 0, c_m = 0, c_mm = 0, c_u = 0, c_s = 0, best = 0;
  // kScStatItems instances per thread and step: their instance and ordinal
  // loads together, issued one step ahead; then (in scope and matched only)
  // the exclusive times and parents' regions together
  const uint64_t step = (uint64_t)gridDim.x * kScStatThreads;
  const uint64_t first = (uint64_t)blockIdx.x * kScStatThreads + threadIdx.x;
  uint4 p0[kScStatItems], p1[kScStatItems];
  uint32_t pord[kScStatItems];
  auto issue = [&](uint64_t xs) {
#pragma unroll
    for (int j = 0; j < kScStatItems; ++j) {
      const uint64_t x = xs + j * step;
      const uint64_t xc = x < n ? x : n - 1;
      p0[j] = inst[2 * xc];
      p1[j] = inst[2 * xc + 1];
      pord[j] = a.ordinal[xc];
    }
  };
  if (first < n) issue(first);
  for (uint64_t x0 = first; x0 < n; x0 += step * kScStatItems) {
    uint4 h0[kScStatItems], h1[kScStatItems];
    uint32_t ord[kScStatItems];
#pragma unroll
    for (int j = 0; j < kScStatItems; ++j) {
      h0[j] = p0[j];
      h1[j] = p1[j];
      ord[j] = pord[j];
    }
    bool in[kScStatItems];
    uint64_t exv[kScStatItems];
    uint32_t preg[kScStatItems];
#pragma unroll
    for (int j = 0; j < kScStatItems; ++j) {
      const uint64_t x = x0 + j * step;
      const uint32_t ctx = h1[j].x, reg = h1[j].w & 0xFFFFu, ereg = h1[j].w >> 16;
      if (a.fast && x < n) {
        // chunk-local ordinal: add the carry of the context entering the chunk
        if (ord[j] & kSoPending) {
          ord[j] = (ord[j] & ~kSoPending) + (reg < a.R ? a.tail[(x / kScTile) * a.R + reg] : 0u);
          a.ordinal[x] = ord[j];
        }
        best = best > ord[j] + 1 ? best : ord[j] + 1;
      }
      const uint64_t group = a.sc.group_shift >= 32 ? 0ull : (uint64_t)(ctx >> a.sc.group_shift);
      in[j] = x < n && in_range32(ctx & a.sc.role_mask, a.sc.role_lo, a.sc.role_hi) &&
              in_range32(group, a.sc.group_lo, a.sc.group_hi) &&
              in_range32(ord[j], a.sc.iter_lo, a.sc.iter_hi) && reg < a.R &&
              (!a.region_mask || a.region_mask[reg] != 0);
      const bool mt = in[j] && ereg == reg;
      exv[j] = mt ? a.excl[x] : 0ull;
      const uint32_t par = h1[j].y;
      preg[j] = mt && par != kNoParent && par < n ? (inst[2 * (uint64_t)par + 1].w & 0xFFFFu)
                                                  : 0xFFFFFFFFu;
    }
    // the next step's loads, issued after this step's dependent loads (a
    // wait for a load also waits for every load issued before it)
    if (x0 + step * kScStatItems < n) issue(x0 + step * kScStatItems);
#pragma unroll
    for (int j = 0; j < kScStatItems; ++j) {
    const uint64_t x = x0 + j * step;
    if (x >= n) continue;
    const uint32_t reg = h1[j].w & 0xFFFFu, ereg = h1[j].w >> 16;
    // the instance's histogram key (none unless matched and in scope)
    uint32_t hk = 0xFFFFFFFFu;
    if (in[j]) {
      c_in += 1;
      if (ereg == kNoEnd) {
        c_u += 1;
        atomicAdd(col_ptr(reg, ARGUS_RS_UNCLOSED), 1ull);
      } else if (ereg != reg) {
        c_mm += 1;
        atomicAdd(col_ptr(reg, ARGUS_RS_MISM_AS_BEGIN), 1ull);
        if (ereg < a.R) atomicAdd(col_ptr(ereg, ARGUS_RS_MISM_AS_END), 1ull);
      } else {
        c_m += 1;
        const uint64_t tb = (uint64_t)h0[j].x | ((uint64_t)h0[j].y << 32);
        const uint64_t te = (uint64_t)h0[j].z | ((uint64_t)h0[j].w << 32);
        const uint64_t d = te - tb, ex = exv[j];
        atomicAdd(col_ptr(reg, ARGUS_RS_COUNT), 1ull);
        atomicAdd(col_ptr(reg, ARGUS_RS_INCL_SUM), (unsigned long long)d);
        atomicAdd(col_ptr(reg, ARGUS_RS_EXCL_SUM), (unsigned long long)ex);
        atomicMin(col_ptr(reg, ARGUS_RS_INCL_MIN), (unsigned long long)d);
        atomicMax(col_ptr(reg, ARGUS_RS_INCL_MAX), (unsigned long long)d);
        atomicMin(col_ptr(reg, ARGUS_RS_EXCL_MIN), (unsigned long long)ex);
        atomicMax(col_ptr(reg, ARGUS_RS_EXCL_MAX), (unsigned long long)ex);
        hk = (reg << 16) | (bit_width64(d) << 8) | bit_width64(ex);
        if (preg[j] == reg) {
          c_s += 1;
          atomicAdd(col_ptr(reg, ARGUS_RS_SELF_NESTED), 1ull);
        }
      }
    }
    a.hkey[x] = hk;
    }
  }
  if (LDS_ROWS) {
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < a.R * kScCols; i += kScStatThreads) {
      const uint32_t col = i % kScCols, reg = i / kScCols;
      const unsigned long long v = srow[i];
      unsigned long long* g = (unsigned long long*)(a.stats + (uint64_t)reg * ARGUS_RS_WIDTH + col);
      if (col == ARGUS_RS_INCL_MIN || col == ARGUS_RS_EXCL_MIN) {
        if (v != ~0ull) atomicMin(g, v);
      } else if (col == ARGUS_RS_INCL_MAX || col == ARGUS_RS_EXCL_MAX) {
        if (v) atomicMax(g, v);
      } else if (v) {
        atomicAdd(g, v);
      }
    }
  }
  const uint32_t lane = threadIdx.x & 63;
  if (a.fast) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
      const uint32_t o = __shfl_xor(best, d);
      best = best > o ? best : o;
    }
    if (lane == 0 && best)
      atomicMax((unsigned long long*)&a.counters[ARGUS_SC_N_ITERATIONS], (unsigned long long)best);
  }
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

// ------------------------------------------------ probe <-> reference join
// Section 3.3: a probe's interval (the exposed latency of one operation at
// one iteration) is joined to the same operation's issue in the same
// iteration of the reference trace, by identity and scope rather than by
// timestamp.  The reference instances sorted by (region, context) give, for
// (operation region, context), a run in which the iteration-th element is
// the joined instance.  Joined probes are then sorted by (instance,
// latency), so each group is a run in latency order and its nearest-rank
// percentiles are read off by position.

struct ProbeArgs {
  const argus_instance* inst;
  const uint4* probes;  // two uint4 per 32-byte probe
  uint64_t np;
  uint32_t R;
  uint64_t none;        // instance code of a probe that joined nothing (= max instances)
  SortBufs ref;         // the reference sorted by (region, context)
  int ref_buf;
  SortBufs pb;          // the probes sorted by (instance, latency)
  uint32_t* ref_out;
  uint64_t* completion;
  uint32_t* flags;      // group heads, then their exclusive scan
  uint64_t* groups;     // [np][ARGUS_PG_WIDTH]
  double* mean;
  uint64_t* counters;
  uint64_t* vpart;      // [join blocks][4] each block's ORs and ANDs of the sort words
};

__global__ void k_pr_init(ProbeArgs a) {
  if (threadIdx.x < ARGUS_PR_NUM_COUNTERS) a.counters[threadIdx.x] = 0;

}

__global__ __launch_bounds__(kScThreads) void k_pr_join(ProbeArgs a) {
  const uint64_t nref = sb_count(a.ref);
  const uint64_t* ra = a.ref.a[a.ref_buf];
  const uint64_t* rb = a.ref.b[a.ref_buf];
  uint32_t bad = 0, joined = 0, unjoined = 0;
  // the OR and the AND of the sort words (latency; instance code << 32)
  uint64_t oa = 0, na = ~0ull, ob = 0, nb2 = ~0ull;
  // Two probes per thread (j and j + stride), their reference searches in
  // lockstep: each search is a chain of dependent loads, and two chains per
  // lane keep more in flight.
  const uint64_t stride = (uint64_t)gridDim.x * kScThreads;
  auto finish = [&](uint64_t j, uint64_t ts, uint64_t te, uint32_t ctx, uint32_t op, bool ok,
                    uint64_t tgt) {
    uint64_t code = a.none, lat = 0, done = kU64Max;
    if (!ok) {
      bad += 1;
    } else {
      // both words of the target loaded together (index clamped; nref == 0
      // loads nothing)
      uint64_t av = ~0ull, bv = 0;
      if (nref) {
        const uint64_t tc = tgt < nref ? tgt : nref - 1;
        av = ra[tc];
        bv = rb[tc];
      }
      if ((tgt < nref) & (av == op) & ((uint32_t)(bv >> 32) == ctx)) {
        const uint32_t x = (uint32_t)bv;
        lat = te - ts;
        const uint4 ib = reinterpret_cast<const uint4*>(a.inst)[2 * (uint64_t)x];
        done = ((uint64_t)ib.x | ((uint64_t)ib.y << 32)) + lat;
        code = x;
        joined += 1;
      } else {
        unjoined += 1;
      }
    }
    a.ref_out[j] = code == a.none ? 0xFFFFFFFFu : (uint32_t)code;
    a.completion[j] = done;
    a.pb.a[0][j] = lat;
    a.pb.b[0][j] = (code << 32) | j;
    oa |= lat;
    na &= lat;
    ob |= code << 32;
    nb2 &= code << 32;
  };
  for (uint64_t j = (uint64_t)blockIdx.x * kScThreads + threadIdx.x; j < a.np; j += 2 * stride) {
    const uint64_t j1 = j + stride;
    const bool has1 = j1 < a.np;
    const uint4 g0 = a.probes[2 * j], g1 = a.probes[2 * j + 1];
    const uint4 q0 = a.probes[2 * (has1 ? j1 : j)], q1 = a.probes[2 * (has1 ? j1 : j) + 1];
    const uint64_t ts0 = (uint64_t)g0.x | ((uint64_t)g0.y << 32), te0 = (uint64_t)g0.z | ((uint64_t)g0.w << 32);
    const uint64_t ts1 = (uint64_t)q0.x | ((uint64_t)q0.y << 32), te1 = (uint64_t)q0.z | ((uint64_t)q0.w << 32);
    const uint32_t ctx0 = g1.x, it0 = g1.y, op0 = g1.z & 0xFFFFu;
    const uint32_t ctx1 = q1.x, it1 = q1.y, op1 = q1.z & 0xFFFFu;
    const bool ok0 = !(te0 < ts0 || op0 >= a.R), ok1 = has1 && !(te1 < ts1 || op1 >= a.R);
    uint64_t lo0 = 0, hi0 = ok0 ? nref : 0, lo1 = 0, hi1 = ok1 ? nref : 0;
    while ((lo0 < hi0) | (lo1 < hi1)) {
      const bool c0 = lo0 < hi0, c1 = lo1 < hi1;
      const uint64_t m0 = (lo0 + hi0) >> 1, m1 = (lo1 + hi1) >> 1;
      const uint64_t r0 = c0 ? m0 : 0, r1 = c1 ? m1 : 0;  // a finished chain reads element 0
      const uint64_t am0 = ra[r0], am1 = ra[r1];
      const uint32_t cm0 = (uint32_t)(rb[r0] >> 32), cm1 = (uint32_t)(rb[r1] >> 32);
      const bool less0 = (am0 < op0) | ((am0 == op0) & (cm0 < ctx0));
      const bool less1 = (am1 < op1) | ((am1 == op1) & (cm1 < ctx1));
      if (c0) {
        if (less0) lo0 = m0 + 1;
        else hi0 = m0;
      }
      if (c1) {
        if (less1) lo1 = m1 + 1;
        else hi1 = m1;
      }
    }
    finish(j, ts0, te0, ctx0, op0, ok0, lo0 + it0);
    if (has1) finish(j1, ts1, te1, ctx1, op1, ok1, lo1 + it1);
  }
  {
    // the block's OR and AND, combined over the blocks by k_pr_vary
    __shared__ uint64_t s_v[kScThreads / 64][4];
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
      oa |= (uint64_t)__shfl_xor((long long)oa, d);
      na &= (uint64_t)__shfl_xor((long long)na, d);
      ob |= (uint64_t)__shfl_xor((long long)ob, d);
      nb2 &= (uint64_t)__shfl_xor((long long)nb2, d);
    }
    const uint32_t wv = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
      s_v[wv][0] = oa;
      s_v[wv][1] = na;
      s_v[wv][2] = ob;
      s_v[wv][3] = nb2;
    }
    __syncthreads();
    if (threadIdx.x < 4) {
      uint64_t v = s_v[0][threadIdx.x];
      for (int q = 1; q < kScThreads / 64; ++q)
        v = (threadIdx.x & 1) ? (v & s_v[q][threadIdx.x]) : (v | s_v[q][threadIdx.x]);
      a.vpart[4 * (uint64_t)blockIdx.x + threadIdx.x] = v;
    }
  }
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t v[3] = {bad, joined, unjoined};
  const int slot[3] = {ARGUS_PR_N_BAD, ARGUS_PR_N_JOINED, ARGUS_PR_N_UNJOINED};
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    const uint32_t t = rows_sum32(row_sum32(v[q]));
    if (lane == 0 && t) atomicAdd((unsigned long long*)&a.counters[slot[q]], (unsigned long long)t);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) a.counters[ARGUS_PR_N_PROBES] = a.np;
}

// The blocks' ORs and ANDs of the probe sort words into the sort state.
__global__ __launch_bounds__(1024) void k_pr_vary(ProbeArgs a, uint32_t blocks) {
  __shared__ uint64_t s_v[16][4];
  uint64_t v[4] = {0, ~0ull, 0, ~0ull};
  for (uint32_t b = threadIdx.x; b < blocks; b += 1024)
#pragma unroll
    for (int k = 0; k < 4; ++k)
      v[k] = (k & 1) ? (v[k] & a.vpart[4 * (uint64_t)b + k]) : (v[k] | a.vpart[4 * (uint64_t)b + k]);
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t o = (uint64_t)__shfl_xor((long long)v[k], d);
      v[k] = (k & 1) ? (v[k] & o) : (v[k] | o);
    }
  const uint32_t w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int k = 0; k < 4; ++k) s_v[w][k] = v[k];
  __syncthreads();
  if (threadIdx.x < 4) {
    const int k = threadIdx.x;
    uint64_t r = s_v[0][k];
    for (int q = 1; q < 16; ++q) r = (k & 1) ? (r & s_v[q][k]) : (r | s_v[q][k]);
    uint64_t* c = reinterpret_cast<uint64_t*>(a.pb.ctl);
    c[k] = r;  // or_a, and_a, or_b, and_b
  }
}

__device__ __forceinline__ bool pr_head(const uint64_t* b, uint64_t k, uint64_t none) {
  const uint64_t r = b[k] >> 32;
  return r != none && (k == 0 || (b[k - 1] >> 32) != r);
}

__global__ __launch_bounds__(kScThreads) void k_pr_heads(ProbeArgs a, int buf) {
  buf = sb_in(a.pb, buf, 1, 64);
  const uint64_t* b = a.pb.b[buf];
  uint32_t heads = 0;
  for (uint64_t k = (uint64_t)blockIdx.x * kScThreads + threadIdx.x; k < a.np;
       k += (uint64_t)gridDim.x * kScThreads) {
    const uint32_t h = pr_head(b, k, a.none) ? 1u : 0u;
    a.flags[k] = h;
    heads += h;
  }
  const uint32_t t = rows_sum32(row_sum32(heads));
  if ((threadIdx.x & 63) == 0 && t)
    atomicAdd((unsigned long long*)&a.counters[ARGUS_PR_N_GROUPS], (unsigned long long)t);
}

// One thread per group head: the group's count, sum, issue time, mean and
// nearest-rank percentiles (its latencies are in increasing order).
__global__ __launch_bounds__(kScThreads) void k_pr_groups(ProbeArgs a, int buf) {
  buf = sb_in(a.pb, buf, 1, 64);
  const uint64_t* la = a.pb.a[buf];
  const uint64_t* b = a.pb.b[buf];
  for (uint64_t k = (uint64_t)blockIdx.x * kScThreads + threadIdx.x; k < a.np;
       k += (uint64_t)gridDim.x * kScThreads) {
    if (!pr_head(b, k, a.none)) continue;
    const uint64_t r = b[k] >> 32;
    // end of the run: first position whose instance code exceeds r
    uint64_t lo = k + 1, hi = a.np;
    while (lo < hi) {
      const uint64_t mid = (lo + hi) >> 1;
      if ((b[mid] >> 32) > r) hi = mid;
      else lo = mid + 1;
    }
    const uint64_t cnt = lo - k;
    uint64_t sum = 0;
    for (uint64_t i = k; i < lo; ++i) sum += la[i];
    const uint64_t g = a.flags[k];
    uint64_t* row = a.groups + g * ARGUS_PG_WIDTH;
    row[ARGUS_PG_INSTANCE] = r;
    row[ARGUS_PG_COUNT] = cnt;
    row[ARGUS_PG_SUM] = sum;
    const uint4 ib = reinterpret_cast<const uint4*>(a.inst)[2 * r];
    row[ARGUS_PG_ISSUE] = (uint64_t)ib.x | ((uint64_t)ib.y << 32);
    const uint32_t q[6] = {0, 20, 40, 60, 80, 100};
#pragma unroll
    for (int t = 0; t < 6; ++t) {
      uint64_t rank = ((uint64_t)q[t] * cnt + 99) / 100;
      if (rank < 1) rank = 1;
      row[ARGUS_PG_P0 + t] = la[k + rank - 1];
    }
    a.mean[g] = (double)sum / (double)cnt;
  }
}

// ------------------------------------------------------------ phase handoffs
// Section 4.2: the time between successive cooperative phases of a
// persistent kernel is a quantity of its own.  Phases are the instances of
// one level L; y follows x when it is the next level-L child of the same
// parent (for L = 0, the next top-level instance of the context).  Between
// two such siblings lie only descendants of the first, so after compacting
// the instances of level <= L (in canonical order), a phase's predecessor is
// simply the element before it, when that one has level L, the same context
// and the same parent.

struct HandoffArgs {
  const argus_instance* inst;
  const uint64_t* n_inst;
  uint64_t max_inst;
  uint32_t R, L;
  uint32_t* comp;    // instances of level <= L in canonical order
  uint64_t* status;  // [tiles] look-back words of the compaction (count, flags)
  uint32_t* tctr;    // tile counter of the compaction
  uint64_t* mtot;    // instances compacted
  uint64_t* pairs;  // [R][R][4]: count, sum, min, max (the output)
  uint32_t* dkey;   // [dumps][kHoSlots]: each pair block's hash table keys (0: empty)
  uint64_t* dval;   // [dumps][kHoSlots][4]: and its count, sum, min, max
  uint32_t dumps;   // pair blocks launched
  uint64_t* hist;   // [65]
  uint64_t* parent_gap;  // [max_inst] or NULL
  uint64_t* counters;
};

__device__ __forceinline__ uint64_t ho_count(const HandoffArgs& a) {
  const uint64_t v = *a.n_inst;
  return v < a.max_inst ? v : a.max_inst;
}

__global__ __launch_bounds__(kScThreads) void k_ho_init(HandoffArgs a) {
  const uint64_t stride = (uint64_t)gridDim.x * kScThreads;
  const uint64_t first = (uint64_t)blockIdx.x * kScThreads + threadIdx.x;
  const uint64_t np = (uint64_t)a.R * a.R * 4;
  for (uint64_t i = first; i < np; i += stride) a.pairs[i] = (i & 3) == 2 ? kU64Max : 0ull;
  if (a.parent_gap)
    for (uint64_t i = first; i < a.max_inst; i += stride) a.parent_gap[i] = 0;
  if (first < 65) a.hist[first] = 0;
  if (first < ARGUS_HO_NUM_COUNTERS) a.counters[first] = 0;
  const uint64_t tiles = (a.max_inst + kScTile - 1) / kScTile;
  for (uint64_t i = first; i < tiles; i += stride) a.status[i] = 0;
  if (first == 0) {
    *a.tctr = 0;
    *a.mtot = 0;
  }
}

// The instances of level <= L compacted in canonical order, in one pass:
// blocks take tiles of 4096 instances in order (a counter), count the
// tile's qualifying instances (a ballot per round of 64, the waves' counts
// through LDS), publish the count, find the count before the tile by
// decoupled look-back, and write the indices.  The tile holding the last
// instance records the total.
__global__ __launch_bounds__(kScThreads) void k_ho_compact(HandoffArgs a) {
  __shared__ uint32_t s_tile, s_w[kScThreads / 64];
  __shared__ uint64_t s_base;
  const uint64_t n = ho_count(a);
  const uint64_t T = (n + kScTile - 1) / kScTile;
  const uint32_t* iw = reinterpret_cast<const uint32_t*>(a.inst);  // 8 words per instance
  const uint32_t tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint64_t lt = lanemask_lt();
  uint32_t at = 0;
  for (;;) {
    if (tid == 0) s_tile = atomicAdd(a.tctr, 1u);
    __syncthreads();
    const uint64_t tile = s_tile;
    if (tile >= T) break;
    const uint64_t base = tile * kScTile;
    uint64_t qm[kScRounds];  // ballot of the qualifying lanes of each round
    uint32_t lv[kScRounds];
    // all the tile's loads issued before the first is used (indices clamped
    // to the last instance, n >= 1 here, instead of a branch per load)
#pragma unroll
    for (int r = 0; r < kScRounds; ++r) {
      const uint64_t x = base + w * (kScRounds * 64) + (uint32_t)r * 64 + lane;
      lv[r] = iw[8 * (x < n ? x : n - 1) + 6];
    }
    uint32_t wc = 0;
#pragma unroll
    for (int r = 0; r < kScRounds; ++r) {
      const uint64_t x = base + w * (kScRounds * 64) + (uint32_t)r * 64 + lane;
      const bool in = x < n;
      const uint32_t lvl = lv[r];
      at += in && lvl == a.L;
      qm[r] = __ballot(in && lvl <= a.L);
      wc += (uint32_t)__popcll(qm[r]);
    }
    if (lane == 0) s_w[w] = wc;
    __syncthreads();
    uint32_t wpre = 0, cnt = 0;
#pragma unroll
    for (int q = 0; q < kScThreads / 64; ++q) {
      wpre += q < (int)w ? s_w[q] : 0u;
      cnt += s_w[q];
    }
    if (tid == 0) {
      uint64_t excl = 0;
      if (tile == 0) {
        st_agent(&a.status[0], kFlagIncl | cnt);
      } else {
        st_agent(&a.status[tile], kFlagAgg | cnt);
        int64_t tt = (int64_t)tile - 1;
        uint32_t spins = 0;
        while (tt >= 0) {
          const uint64_t v = ld_agent(&a.status[tt]);
          const uint64_t f = v & ~kValMask;
          if (f == 0) {
            if (++spins > kMaxSpins) {
              atomicOr((unsigned long long*)&a.counters[ARGUS_HO_INTERNAL], 1ull);
              break;
            }
            backoff();
            continue;
          }
          excl += v & kValMask;
          if (f == kFlagIncl) break;
          --tt;
        }
        st_agent(&a.status[tile], kFlagIncl | (excl + cnt));
      }
      s_base = excl;
      if (tile == T - 1) *a.mtot = excl + cnt;
    }
    __syncthreads();
    uint64_t o = s_base + wpre;
#pragma unroll
    for (int r = 0; r < kScRounds; ++r) {
      if ((qm[r] >> lane) & 1u)
        a.comp[o + (uint32_t)__popcll(qm[r] & lt)] =
            (uint32_t)(base + w * (kScRounds * 64) + (uint32_t)r * 64 + lane);
      o += (uint32_t)__popcll(qm[r]);
    }
  }
  const uint32_t tot = rows_sum32(row_sum32(at));
  if (lane == 0 && tot)
    atomicAdd((unsigned long long*)&a.counters[ARGUS_HO_N_AT_LEVEL], (unsigned long long)tot);
}

// Successive pairs, aggregated per block in an LDS hash table of (x region,
// y region) keys (linear probing from the key's home slot, keys claimed with a
// compare-and-swap): count, sum, min and max by LDS atomics.  At the end each
// block stores its table, keys and values, into its own dump with plain
// stores; k_ho_merge adds the dumps up.  A pair whose key finds no slot goes
// to the output row directly, by global atomics (such a key is never in the
// table: every insertion of a key probes the same slots from its home).  One
// block of 1024 threads per compute unit holds 4096 keys in 144 KiB of LDS.
// The histogram is in LDS, added once per block.  The loop runs in steps of
// one wave over 64 consecutive pairs, so that the histogram and the
// per-parent sums are combined across the wave first: one LDS add per
// distinct bit width and one global add per run of lanes with the same parent
// (the phases of one parent step are consecutive, so a wave holds one or two
// parents, where an add per lane would queue 64 atomics on one address).
constexpr uint32_t kHoSlots = 4096;
constexpr int kHoProbes = 16;
constexpr uint32_t kHoThreads = 1024;
constexpr uint32_t kHoHashShift = 20;  // 32 - log2(kHoSlots)
constexpr uint32_t kHoMaxDumps = 256;  // pair blocks at most: one per compute unit

__device__ __forceinline__ uint32_t ho_hash(uint32_t key) { return key * 2654435761u; }

__global__ __launch_bounds__(kHoThreads) void k_ho_pairs(HandoffArgs a) {
  __shared__ unsigned long long s_hist[65];
  __shared__ uint32_t s_key[kHoSlots];                // 1 + rx * R + ry; 0: empty
  __shared__ unsigned long long s_v[4][kHoSlots];      // count, sum, min, max
  for (int i = threadIdx.x; i < 65; i += kHoThreads) s_hist[i] = 0;
  for (uint32_t i = threadIdx.x; i < kHoSlots; i += kHoThreads) {
    s_key[i] = 0;
    s_v[0][i] = 0;
    s_v[1][i] = 0;
    s_v[2][i] = ~0ull;
    s_v[3][i] = 0;
  }
  __syncthreads();
  const uint64_t n = ho_count(a);
  const uint4* inst = reinterpret_cast<const uint4*>(a.inst);
  const uint64_t m = *a.mtot;
  const uint32_t lane = threadIdx.x & 63;
  uint64_t gaps = 0, gsum = 0;
  for (uint64_t k0 = (uint64_t)blockIdx.x * kHoThreads + (threadIdx.x & ~63u); k0 + 1 < m;
       k0 += (uint64_t)gridDim.x * kHoThreads) {
    const uint64_t k = k0 + lane;
    bool ok = k + 1 < m;
    uint64_t gap = 0;
    uint32_t par = kNoParent;
    if (ok) {
      const uint64_t x = a.comp[k], y = a.comp[k + 1];
      // both instances loaded together (y is at level L for nearly every
      // pair), not x after y's test
      const uint4 ya = inst[2 * y], yb = inst[2 * y + 1];
      const uint4 xa = inst[2 * x], xb = inst[2 * x + 1];
      asm volatile("" ::"v"(yb.z), "v"(xb.z));
      ok = yb.z == a.L;
      if (ok) {
        const uint32_t rx = xb.w & 0xFFFFu, ry = yb.w & 0xFFFFu;
        ok = xb.z == a.L && xb.x == yb.x && xb.y == yb.y &&  // level, context, parent
             (xb.w >> 16) != kNoEnd && rx < a.R && ry < a.R;
        if (ok) {
          const uint64_t te = (uint64_t)xa.z | ((uint64_t)xa.w << 32);
          const uint64_t tb = (uint64_t)ya.x | ((uint64_t)ya.y << 32);
          gap = tb - te;
          par = yb.y;
          const uint32_t key = 1u + rx * a.R + ry;
          uint32_t h = ho_hash(key) >> kHoHashShift;
          int slot = -1;
          for (int p = 0; p < kHoProbes; ++p) {
            const uint32_t cur = __hip_atomic_load(&s_key[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            if (cur == key) {
              slot = (int)h;
              break;
            }
            if (cur == 0) {
              const uint32_t prev = atomicCAS(&s_key[h], 0u, key);
              if (prev == 0u || prev == key) {
                slot = (int)h;
                break;
              }
            }
            h = (h + 1) & (kHoSlots - 1);
          }
          if (slot >= 0) {
            atomicAdd(&s_v[0][slot], 1ull);
            atomicAdd(&s_v[1][slot], (unsigned long long)gap);
            atomicMin(&s_v[2][slot], (unsigned long long)gap);
            atomicMax(&s_v[3][slot], (unsigned long long)gap);
          } else {
            unsigned long long* row = (unsigned long long*)(a.pairs + 4 * ((uint64_t)rx * a.R + ry));
            atomicAdd(&row[0], 1ull);
            atomicAdd(&row[1], (unsigned long long)gap);
            if (gap < __hip_atomic_load(&row[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
              atomicMin(&row[2], (unsigned long long)gap);
            if (gap > __hip_atomic_load(&row[3], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
              atomicMax(&row[3], (unsigned long long)gap);
          }
        }
      }
    }
    // histogram: one leader lane per distinct bit width adds the lanes that share it
    const uint32_t bin = ok ? bit_width64(gap) : 65u;
    for (uint64_t pend = __ballot(ok); pend;) {
      const uint32_t l = (uint32_t)__builtin_ctzll(pend);
      const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)bin, (int)l);
      const uint64_t same = __ballot(bin == b);
      if (lane == l) atomicAdd(&s_hist[b], (unsigned long long)__popcll(same));
      pend &= ~same;
    }
    if (a.parent_gap) {
      // segmented inclusive scan over runs of equal parents (head flag, sum),
      // then the last lane of each run adds the run's sum
      const bool pc = ok && par != kNoParent && par < n;
      const uint32_t p = pc ? par : kNoParent;
      uint32_t f = lane_prev(p, ~p) != p;
      uint64_t v = pc ? gap : 0;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint64_t vu = __shfl_up(v, d);
        const uint32_t fu = __shfl_up(f, d);
        if (lane >= (uint32_t)d) {
          if (!f) v += vu;
          f |= fu;
        }
      }
      const uint32_t pn = __shfl_down(p, 1);
      if (pc && (lane == 63 || pn != p))
        atomicAdd((unsigned long long*)&a.parent_gap[p], (unsigned long long)v);
    }
    gaps += ok ? 1 : 0;
    gsum += gap;
  }
  const uint64_t g1 = rows_sum64(row_sum64(gaps)), g2 = rows_sum64(row_sum64(gsum));
  if ((threadIdx.x & 63) == 0) {
    if (g1) atomicAdd((unsigned long long*)&a.counters[ARGUS_HO_N_GAPS], (unsigned long long)g1);
    if (g2) atomicAdd((unsigned long long*)&a.counters[ARGUS_HO_GAP_SUM], (unsigned long long)g2);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 65; i += kHoThreads)
    if (s_hist[i]) atomicAdd((unsigned long long*)&a.hist[i], s_hist[i]);
  uint32_t* dk = a.dkey + (uint64_t)blockIdx.x * kHoSlots;
  ulonglong2* dv = reinterpret_cast<ulonglong2*>(a.dval + (uint64_t)blockIdx.x * kHoSlots * 4);
  for (uint32_t i = threadIdx.x; i < kHoSlots; i += kHoThreads) {
    const uint32_t key = s_key[i];
    dk[i] = key;
    if (key) {
      dv[2 * i] = make_ulonglong2(s_v[0][i], s_v[1][i]);
      dv[2 * i + 1] = make_ulonglong2(s_v[2][i], s_v[3][i]);
    }
  }
}

// The dumps merged.  Block j owns the keys whose home slot lies in
// [j kHoSpan, (j + 1) kHoSpan): in every dump such a key sits less than
// kHoProbes slots after its home, so the block reads that window of each dump
// (kHoWin lanes per dump, several dumps at a time), adds the entries it owns
// in an LDS table and then into their output rows, which no other block
// writes (keys that overflowed there are never in a dump; keys that overflow
// the merge table are added with atomics).
constexpr uint32_t kHoSpan = 16;
constexpr uint32_t kHoWin = 32;  // lanes per dump: kHoSpan + kHoProbes - 1 of them read
constexpr uint32_t kMgSlots = 1024;
constexpr int kMgProbes = 16;
static_assert(kHoSpan + kHoProbes - 1 <= kHoWin && kHoSlots % kHoSpan == 0, "merge window");

__global__ __launch_bounds__(kScThreads) void k_ho_merge(HandoffArgs a) {
  __shared__ uint32_t s_key[kMgSlots];
  __shared__ unsigned long long s_v[4][kMgSlots];
  for (uint32_t i = threadIdx.x; i < kMgSlots; i += kScThreads) {
    s_key[i] = 0;
    s_v[0][i] = 0;
    s_v[1][i] = 0;
    s_v[2][i] = ~0ull;
    s_v[3][i] = 0;
  }
  __syncthreads();
  const uint32_t lo = blockIdx.x * kHoSpan;
  const uint32_t o = threadIdx.x % kHoWin;
  const uint32_t slot = (lo + o) & (kHoSlots - 1);
  if (o < kHoSpan + kHoProbes - 1) {
    for (uint32_t d = threadIdx.x / kHoWin; d < a.dumps; d += kScThreads / kHoWin) {
      const uint64_t e = (uint64_t)d * kHoSlots + slot;
      const uint32_t key = a.dkey[e];
      if (!key) continue;
      const uint32_t hk = ho_hash(key), home = hk >> kHoHashShift;
      if (home < lo || home >= lo + kHoSpan) continue;
      const ulonglong2* v = reinterpret_cast<const ulonglong2*>(a.dval + 4 * e);
      const ulonglong2 cs = v[0], mm = v[1];
      uint32_t h = (hk >> 10) & (kMgSlots - 1);  // the bits below the home slot's
      int at = -1;
      for (int p = 0; p < kMgProbes; ++p) {
        const uint32_t cur = __hip_atomic_load(&s_key[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (cur == key) {
          at = (int)h;
          break;
        }
        if (cur == 0) {
          const uint32_t prev = atomicCAS(&s_key[h], 0u, key);
          if (prev == 0u || prev == key) {
            at = (int)h;
            break;
          }
        }
        h = (h + 1) & (kMgSlots - 1);
      }
      if (at >= 0) {
        atomicAdd(&s_v[0][at], cs.x);
        atomicAdd(&s_v[1][at], cs.y);
        atomicMin(&s_v[2][at], mm.x);
        atomicMax(&s_v[3][at], mm.y);
      } else {
        unsigned long long* row = (unsigned long long*)(a.pairs + 4 * (uint64_t)(key - 1u));
        atomicAdd(&row[0], cs.x);
        atomicAdd(&row[1], cs.y);
        atomicMin(&row[2], mm.x);
        atomicMax(&row[3], mm.y);
      }
    }
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < kMgSlots; i += kScThreads) {
    const uint32_t key = s_key[i];
    if (!key) continue;
    uint64_t* row = a.pairs + 4 * (uint64_t)(key - 1u);
    row[0] += s_v[0][i];
    row[1] += s_v[1][i];
    row[2] = s_v[2][i] < row[2] ? s_v[2][i] : row[2];
    row[3] = s_v[3][i] > row[3] ? s_v[3][i] : row[3];
  }
}

}  // namespace argus

using namespace argus;

namespace {

constexpr size_t kScAlign = 256;
size_t sc_align(size_t v) { return (v + kScAlign - 1) & ~(kScAlign - 1); }

struct Carver {
  size_t o = 0;
  size_t take(size_t b) {
    const size_t at = o;
    o = sc_align(o + (b ? b : 1));
    return at;
  }
};

uint64_t tiles_for(uint64_t n) { return ((n ? n : 1) + kScTile - 1) / kScTile; }
uint64_t scan_blocks_for(uint64_t entries) { return (entries + kScScanBlock - 1) / kScScanBlock; }

// Workspace of one 16-byte-element sort of up to m elements (its buffers);
// the digit table and scan sums are shared and sized by the caller.
struct SortLayout {
  size_t a[2], b[2];
};
SortLayout carve_sort(Carver& c, uint64_t m) {
  SortLayout L{};
  const uint64_t mm = m ? m : 1;
  for (int k = 0; k < 2; ++k) {
    L.a[k] = c.take(sizeof(uint64_t) * mm);
    L.b[k] = c.take(sizeof(uint64_t) * mm);
  }
  return L;
}

struct ScLayout {
  SortLayout ref;
  size_t hist, bsum, octr, tail, cflag, segb, segm, total;
};
ScLayout sc_layout(uint64_t max_inst) {
  Carver c;
  ScLayout L{};
  L.ref = carve_sort(c, max_inst);
  L.hist = c.take(sizeof(uint32_t) * 256 * tiles_for(max_inst));
  L.bsum = c.take(sizeof(uint32_t) * scan_blocks_for(256 * tiles_for(max_inst)));
  L.octr = c.take(sizeof(uint32_t) * kOrdMaxBuckets);
  // chunk-local ordinals: per chunk (tile) and region up to kSoMaxRegions
  const uint64_t chunks = tiles_for(max_inst), segs = (chunks + kSoSeg - 1) / kSoSeg;
  L.tail = c.take(sizeof(uint32_t) * chunks * kSoMaxRegions);
  L.cflag = c.take(sizeof(uint32_t) * chunks);
  L.segb = c.take(sizeof(uint32_t) * segs * kSoMaxRegions);
  L.segm = c.take(sizeof(uint32_t) * segs);
  L.total = c.o;
  return L;
}

struct PrLayout {
  SortLayout ref, pr;
  size_t hist, bsum, flags, ctl, vpart, total;
};
PrLayout pr_layout(uint64_t max_inst, uint64_t np) {
  Carver c;
  PrLayout L{};
  L.ref = carve_sort(c, max_inst);
  L.pr = carve_sort(c, np);
  const uint64_t tiles = std::max(tiles_for(max_inst), tiles_for(np));
  L.hist = c.take(sizeof(uint32_t) * 256 * tiles);
  const uint64_t sb = std::max(scan_blocks_for(256 * tiles), scan_blocks_for(np));
  L.bsum = c.take(sizeof(uint32_t) * sb);
  L.flags = c.take(sizeof(uint32_t) * (np ? np : 1));
  L.ctl = c.take(sizeof(SortCtl));
  L.vpart = c.take(sizeof(uint64_t) * 4 * 4096);  // the join's blocks (at most 4096)
  L.total = c.o;
  return L;
}

SortBufs make_bufs(char* base, const SortLayout& L, size_t hist, size_t bsum, uint64_t count_max,
                   const uint64_t* count_ptr, const argus_instance* inst) {
  SortBufs s{};
  for (int k = 0; k < 2; ++k) {
    s.a[k] = (uint64_t*)(base + L.a[k]);
    s.b[k] = (uint64_t*)(base + L.b[k]);
  }
  s.hist = (uint32_t*)(base + hist);
  s.bsum = (uint32_t*)(base + bsum);
  s.tiles_max = tiles_for(count_max);
  s.count_ptr = count_ptr;
  s.count_max = count_max;
  s.inst = inst;
  return s;
}

void scan_u32(uint32_t* data, uint64_t total, uint32_t* bsum, hipStream_t st,
              const SortBufs* sk = nullptr, int word = 0, int shift = 0) {
  if (total <= kScSmallMax) {
    SortBufs none{};
    hipLaunchKernelGGL(k_scan_small, dim3(1), dim3(1024), 0, st, data, total, sk ? *sk : none,
                       word, shift);
    return;
  }
  const uint32_t blocks = (uint32_t)scan_blocks_for(total ? total : 1);
  hipLaunchKernelGGL(k_scan_sums, dim3(blocks), dim3(kScThreads), 0, st, data, total, bsum);
  hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(1024), 0, st, bsum, blocks);
  hipLaunchKernelGGL(k_scan_apply, dim3(blocks), dim3(kScThreads), 0, st, data, total, bsum);
}

// One stable pass on digit (word, shift), reading buffer `in` (or the
// instances) and writing buffer `out`.
void sort_pass(const SortBufs& s, bool from_inst, int in, int out, int word, int shift,
               hipStream_t st) {
  const uint32_t tiles = (uint32_t)s.tiles_max;
  if (from_inst)
    hipLaunchKernelGGL(k_sort_hist<kSrcInst>, dim3(tiles), dim3(kScThreads), 0, st, s, in, word,
                       shift);
  else
    hipLaunchKernelGGL(k_sort_hist<kSrcBuf>, dim3(tiles), dim3(kScThreads), 0, st, s, in, word,
                       shift);
  scan_u32(s.hist, 256ull * s.tiles_max, s.bsum, st, &s, word, shift);
  if (from_inst)
    hipLaunchKernelGGL(k_sort_scatter<kSrcInst>, dim3(tiles), dim3(kScThreads), kScStageBytes, st, s,
                       in, out, word, shift);
  else
    hipLaunchKernelGGL(k_sort_scatter<kSrcBuf>, dim3(tiles), dim3(kScThreads), kScStageBytes, st, s,
                       in, out, word, shift);
}

// The instances sorted by (BEGIN region, context), canonical order kept
// within; returns the buffer holding the result.
int sort_reference(const SortBufs& s, uint32_t R, hipStream_t st) {
  sort_pass(s, true, 0, 0, 0, 0, st);
  if (R <= 256) return 0;
  sort_pass(s, false, 0, 1, 0, 8, st);
  return 1;
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
    // the sort scatter stages a whole tile (64 KiB of dynamic LDS)
    for (const void* f : {(const void*)k_sort_scatter<kSrcInst>, (const void*)k_sort_scatter<kSrcBuf>})
      if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kScStageBytes) !=
          hipSuccess)
        return ARGUS_E_HIP;
    g_sc_dev_ok[dev] = 1;
  }
  return ARGUS_OK;
}

uint32_t sc_grid(uint64_t items, uint64_t per_block, uint32_t cap) {
  uint64_t g = (items + per_block - 1) / per_block;
  if (g > cap) g = cap;
  return g < 1 ? 1u : (uint32_t)g;
}

bool misaligned(const void* p, uintptr_t to) { return ((uintptr_t)p & (to - 1)) != 0; }

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
  if (misaligned(io->d_instances, 16) || misaligned(io->d_instance_excl, 8) ||
      misaligned(io->d_n_instances, 8) || misaligned(io->d_ordinal, 4) ||
      misaligned(io->d_stats, 8) || misaligned(io->d_counters, 8) ||
      misaligned(d_workspace, kScAlign))
    return ARGUS_E_ALIGN;
  const ScLayout L = sc_layout(io->max_instances);
  if (workspace_bytes < L.total) return ARGUS_E_CAPACITY;
  const int dc = sc_check_device();
  if (dc != ARGUS_OK) return dc;

  char* base = (char*)d_workspace;
  ScopeArgs a{};
  a.inst = io->d_instances;
  a.excl = io->d_instance_excl;
  a.R = cfg->num_regions;
  a.sc = cfg->scope;
  a.region_mask = io->d_region_mask;
  a.ordinal = io->d_ordinal;
  a.stats = io->d_stats;
  a.counters = io->d_counters;
  a.s = make_bufs(base, L.ref, L.hist, L.bsum, io->max_instances, io->d_n_instances,
                  io->d_instances);
  a.octr = (uint32_t*)(base + L.octr);
  a.tail = (uint32_t*)(base + L.tail);
  a.cflag = (uint32_t*)(base + L.cflag);
  a.segb = (uint32_t*)(base + L.segb);
  a.segm = (uint32_t*)(base + L.segm);
  a.fast = a.R <= kSoMaxRegions ? 1u : 0u;
  hipStream_t st = (hipStream_t)stream_v;
  hipLaunchKernelGGL(k_sc_init, dim3(sc_grid((uint64_t)a.R * ARGUS_RS_WIDTH, kScThreads, 1024)),
                     dim3(kScThreads), 0, st, a);
  if (a.fast) {
    const uint64_t chunks = tiles_for(io->max_instances);
    const uint64_t segs = (chunks + kSoSeg - 1) / kSoSeg;
    // four chunks at a time per block (a wave each), each wave with its row
    // of R counters
    const size_t so_lds = (size_t)4 * a.R * sizeof(uint32_t);
    (void)hipFuncSetAttribute((const void*)k_so_local, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)so_lds);
    hipLaunchKernelGGL(k_so_local,
                       dim3((uint32_t)std::min<uint64_t>((chunks + 3) / 4,
                                                         persistent_blocks((const void*)k_so_local,
                                                                           kScThreads))),
                       dim3(kScThreads), so_lds, st, a);
    const uint64_t cells = segs * a.R;
    hipLaunchKernelGGL(k_so_seg, dim3((uint32_t)((cells + kScThreads - 1) / kScThreads)),
                       dim3(kScThreads), 0, st, a);
    hipLaunchKernelGGL(k_so_top, dim3((a.R + kScThreads - 1) / kScThreads), dim3(kScThreads), 0, st, a);
    hipLaunchKernelGGL(k_so_down, dim3((uint32_t)((cells + kScThreads - 1) / kScThreads)),
                       dim3(kScThreads), 0, st, a);
    a.hkey = reinterpret_cast<uint32_t*>(a.s.b[1]);  // the sort buffers are free
  } else {
    const int buf = sort_reference(a.s, a.R, st);
    a.pairs = a.s.a[buf ^ 1];  // free once the sort is done
    hipLaunchKernelGGL(k_sc_ordinal, dim3(sc_grid(io->max_instances, kScTile, 2048)),
                       dim3(kScThreads), 0, st, a, buf);
    const uint64_t nbk = (io->max_instances + (1ull << kOrdBucketBits) - 1) >> kOrdBucketBits;
    const uint64_t blocks = 8ull * ((nbk + 7) / 8) * kOrdSlices;
    hipLaunchKernelGGL(k_sc_ord_place, dim3((uint32_t)(blocks ? blocks : 1)), dim3(kScThreads), 0, st, a);
    a.hkey = reinterpret_cast<uint32_t*>(a.s.b[buf ^ 1]);  // free once the sort is done
  }
  if (a.R <= kScLdsRegions) {
    const size_t lds = (size_t)a.R * kScCols * sizeof(uint64_t);
    (void)hipFuncSetAttribute((const void*)k_sc_stats<true>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    // one block per compute unit: each flushes its rows once
    hipLaunchKernelGGL(k_sc_stats<true>,
                       dim3((uint32_t)std::min<uint64_t>(persistent_blocks((const void*)k_sc_stats<true>,
                                                                           kScStatThreads),
                                                         sc_grid(io->max_instances, kScStatThreads, 4096))),
                       dim3(kScStatThreads), lds, st, a);
  } else {
    hipLaunchKernelGGL(k_sc_stats<false>, dim3(sc_grid(io->max_instances, kScStatThreads, 4096)),
                       dim3(kScStatThreads), 0, st, a);
  }
  if (io->max_instances > 0 &&
      launch_hist_keys(a.hkey, io->d_n_instances, io->max_instances, a.stats, a.R, st) != hipSuccess)
    return ARGUS_E_HIP;
  return hipGetLastError() == hipSuccess ? ARGUS_OK : ARGUS_E_HIP;
}

extern "C" size_t argus_attr_probes_workspace_bytes(uint64_t max_instances, uint64_t n_probes) {
  if (max_instances >= (1ull << 31) || n_probes >= (1ull << 31)) return 0;
  return pr_layout(max_instances, n_probes).total;
}

extern "C" int argus_attr_probes(const argus_probes_config* cfg, const argus_probes_io* io,
                                 void* d_workspace, size_t workspace_bytes, void* stream_v) {
  if (!cfg || !io) return ARGUS_E_INVAL;
  if (cfg->abi_version != ARGUS_ATTR_ABI_VERSION) return ARGUS_E_ABI;
  if (cfg->num_regions < 1 || cfg->num_regions > 65535) return ARGUS_E_INVAL;
  if (io->max_instances >= (1ull << 31) || io->n_probes >= (1ull << 31)) return ARGUS_E_CAPACITY;
  if (!io->d_n_instances || !io->d_counters) return ARGUS_E_INVAL;
  if (io->max_instances > 0 && !io->d_instances) return ARGUS_E_INVAL;
  if (io->n_probes > 0 && (!io->d_probes || !io->d_ref || !io->d_completion || !io->d_groups ||
                           !io->d_mean))
    return ARGUS_E_INVAL;
  if (!d_workspace) return ARGUS_E_INVAL;
  if (misaligned(io->d_instances, 16) || misaligned(io->d_probes, 16) ||
      misaligned(io->d_n_instances, 8) || misaligned(io->d_ref, 4) ||
      misaligned(io->d_completion, 8) || misaligned(io->d_groups, 8) ||
      misaligned(io->d_mean, 8) || misaligned(io->d_counters, 8) ||
      misaligned(d_workspace, kScAlign))
    return ARGUS_E_ALIGN;
  const PrLayout L = pr_layout(io->max_instances, io->n_probes);
  if (workspace_bytes < L.total) return ARGUS_E_CAPACITY;
  const int dc = sc_check_device();
  if (dc != ARGUS_OK) return dc;

  char* base = (char*)d_workspace;
  ProbeArgs a{};
  a.inst = io->d_instances;
  a.probes = reinterpret_cast<const uint4*>(io->d_probes);
  a.np = io->n_probes;
  a.R = cfg->num_regions;
  a.none = io->max_instances;
  a.ref = make_bufs(base, L.ref, L.hist, L.bsum, io->max_instances, io->d_n_instances,
                    io->d_instances);
  a.pb = make_bufs(base, L.pr, L.hist, L.bsum, io->n_probes, nullptr, io->d_instances);
  a.pb.ctl = reinterpret_cast<SortCtl*>(base + L.ctl);  // passes on constant digits are skipped
  a.vpart = reinterpret_cast<uint64_t*>(base + L.vpart);
  a.ref_out = io->d_ref;
  a.completion = io->d_completion;
  a.flags = (uint32_t*)(base + L.flags);
  a.groups = io->d_groups;
  a.mean = io->d_mean;
  a.counters = io->d_counters;
  hipStream_t st = (hipStream_t)stream_v;
  hipLaunchKernelGGL(k_pr_init, dim3(1), dim3(64), 0, st, a);
  if (a.np > 0) {
    a.ref_buf = sort_reference(a.ref, a.R, st);
    const uint32_t jb = sc_grid(a.np, 2 * kScThreads, 4096);  // two probes per thread
    hipLaunchKernelGGL(k_pr_join, dim3(jb), dim3(kScThreads), 0, st, a);
    hipLaunchKernelGGL(k_pr_vary, dim3(1), dim3(1024), 0, st, a, jb);
    // (instance, latency) order: the latency's eight bytes, then the
    // instance code's bytes (stable LSD)
    int in = 0;
    for (int byte = 0; byte < 8; ++byte, in ^= 1) sort_pass(a.pb, false, in, in ^ 1, 0, 8 * byte, st);
    const uint32_t code_bits = 64u - (uint32_t)__builtin_clzll(a.none | 1ull);
    for (uint32_t byte = 0; 8 * byte < code_bits; ++byte, in ^= 1)
      sort_pass(a.pb, false, in, in ^ 1, 1, 32 + 8 * (int)byte, st);
    hipLaunchKernelGGL(k_pr_heads, dim3(sc_grid(a.np, kScThreads, 4096)), dim3(kScThreads), 0, st,
                       a, in);
    scan_u32(a.flags, a.np, a.pb.bsum, st);
    hipLaunchKernelGGL(k_pr_groups, dim3(sc_grid(a.np, kScThreads, 4096)), dim3(kScThreads), 0,
                       st, a, in);
  }
  return hipGetLastError() == hipSuccess ? ARGUS_OK : ARGUS_E_HIP;
}

namespace {

struct HoLayout {
  size_t comp, status, tctr, mtot, dkey, dval, total;
};
HoLayout ho_layout(uint64_t max_instances, uint32_t R) {
  Carver c;
  HoLayout L{};
  const uint64_t m = max_instances ? max_instances : 1;
  L.comp = c.take(sizeof(uint32_t) * m);
  L.status = c.take(sizeof(uint64_t) * tiles_for(m));
  L.tctr = c.take(sizeof(uint32_t));
  L.mtot = c.take(sizeof(uint64_t));
  L.dkey = c.take(sizeof(uint32_t) * (uint64_t)kHoMaxDumps * kHoSlots);
  L.dval = c.take(sizeof(uint64_t) * 4 * (uint64_t)kHoMaxDumps * kHoSlots);
  L.total = c.o;
  return L;
}

}  // namespace

extern "C" size_t argus_attr_handoffs_workspace_bytes(uint64_t max_instances,
                                                      uint32_t num_regions) {
  if (max_instances >= (1ull << 31) || num_regions < 1 || num_regions > 4096) return 0;
  return ho_layout(max_instances, num_regions).total;
}

extern "C" int argus_attr_handoffs(const argus_handoffs_config* cfg, const argus_handoffs_io* io,
                                   void* d_workspace, size_t workspace_bytes, void* stream_v) {
  if (!cfg || !io) return ARGUS_E_INVAL;
  if (cfg->abi_version != ARGUS_ATTR_ABI_VERSION) return ARGUS_E_ABI;
  if (cfg->num_regions < 1 || cfg->num_regions > 4096) return ARGUS_E_INVAL;
  if (io->max_instances >= (1ull << 31)) return ARGUS_E_CAPACITY;
  if (!io->d_n_instances || !io->d_pairs || !io->d_hist || !io->d_counters) return ARGUS_E_INVAL;
  if (io->max_instances > 0 && !io->d_instances) return ARGUS_E_INVAL;
  if (!d_workspace) return ARGUS_E_INVAL;
  if (misaligned(io->d_instances, 16) || misaligned(io->d_n_instances, 8) ||
      misaligned(io->d_pairs, 8) || misaligned(io->d_hist, 8) ||
      misaligned(io->d_parent_gap, 8) || misaligned(io->d_counters, 8) ||
      misaligned(d_workspace, kScAlign))
    return ARGUS_E_ALIGN;
  const HoLayout HL = ho_layout(io->max_instances, cfg->num_regions);
  if (workspace_bytes < HL.total) return ARGUS_E_CAPACITY;
  const int dc = sc_check_device();
  if (dc != ARGUS_OK) return dc;

  char* base = (char*)d_workspace;
  HandoffArgs a{};
  a.inst = io->d_instances;
  a.n_inst = io->d_n_instances;
  a.max_inst = io->max_instances;
  a.R = cfg->num_regions;
  a.L = cfg->level;
  a.comp = (uint32_t*)(base + HL.comp);
  a.status = (uint64_t*)(base + HL.status);
  a.tctr = (uint32_t*)(base + HL.tctr);
  a.mtot = (uint64_t*)(base + HL.mtot);
  a.dkey = (uint32_t*)(base + HL.dkey);
  a.dval = (uint64_t*)(base + HL.dval);
  a.pairs = io->d_pairs;
  a.hist = io->d_hist;
  a.parent_gap = io->d_parent_gap;
  a.counters = io->d_counters;
  hipStream_t st = (hipStream_t)stream_v;
  const uint64_t init_items =
      std::max<uint64_t>((uint64_t)a.R * a.R * 4, io->max_instances);
  hipLaunchKernelGGL(k_ho_init, dim3(sc_grid(std::max<uint64_t>(init_items, 65), kScThreads, 4096)),
                     dim3(kScThreads), 0, st, a);
  if (io->max_instances > 0) {
    const uint32_t g = sc_grid(io->max_instances, kScThreads, 4096);
    // resident blocks only: they take the tiles in order
    hipLaunchKernelGGL(k_ho_compact,
                       dim3((uint32_t)std::min<uint64_t>(tiles_for(io->max_instances),
                                                         persistent_blocks((const void*)k_ho_compact,
                                                                           kScThreads))),
                       dim3(kScThreads), 0, st, a);
    // resident blocks only (one per compute unit): each stores its table once
    a.dumps = (uint32_t)std::min<uint64_t>(
        std::min<uint64_t>(g, persistent_blocks((const void*)k_ho_pairs, kHoThreads)), kHoMaxDumps);
    hipLaunchKernelGGL(k_ho_pairs, dim3(a.dumps), dim3(kHoThreads), 0, st, a);
    hipLaunchKernelGGL(k_ho_merge, dim3(kHoSlots / kHoSpan), dim3(kScThreads), 0, st, a);
  }
  return hipGetLastError() == hipSuccess ? ARGUS_OK : ARGUS_E_HIP;
}
