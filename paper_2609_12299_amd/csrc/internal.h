// internal.h -- shared definitions of the HIP implementation (not part of the
// public ABI).  Every kernel of the library runs on gfx950: 64-lane
// wavefronts, 160 KiB of LDS per CU, 8 XCDs with private L2 caches (so all
// cross-workgroup communication inside a kernel goes through agent-scope
// atomics).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/argus_attr.h"

namespace argus {

// ------------------------------------------------------------------ sizes
constexpr int kSortThreads = 256;
constexpr int kSortItems = 16;
constexpr int kSortTile = kSortThreads * kSortItems;  // 4096 elements
constexpr int kRadixBins = 256;
constexpr int kDigitPositions = 12;  // 4 context digits, then 8 timestamp digits
constexpr int kSlots = 16;           // sort passes planned per sort
constexpr int kPhase2Slot = 4;       // first slot of the full-sort phase
constexpr int kChunk = 256;          // input records per chunk of the run detection

constexpr int kMatchThreads = 256;
constexpr int kMatchItems = 8;
constexpr int kMatchTile = kMatchThreads * kMatchItems;  // 2048 elements

constexpr int kSweepThreads = 256;
constexpr int kSweepItems = 8;
constexpr int kSweepTile = kSweepThreads * kSweepItems;  // 2048 events
constexpr int kSweepSlots = 8;  // groups of one tile aggregated in LDS

// Ordering overlap events by merging per-context runs (see k_merge.hip).
constexpr int kMergeThreads = 512;
constexpr int kMergeItems = 8;
constexpr int kMergeTile = kMergeThreads * kMergeItems;  // 4096 events
constexpr int kMaxMergeBits = 8;   // context bits merged (two per pass at most)
constexpr int kMaxMergePasses = 4;   // merge passes: pairs of bits, then a single one
// Four-way passes cut each segment at every 28th of its samples in merged
// order, a sample being every 127th event of a run: a tile then holds at
// most (28 + 4) * 127 - 4 events, which leaves room for the second pair of
// runs to start at a multiple of 8 in LDS.
constexpr uint32_t kSampStride = 127;
constexpr uint32_t kSampPerTile = 28;
static_assert((kSampPerTile + 4) * kSampStride - 4 + 7 <= (uint32_t)kMergeTile, "four-way tile bound");
constexpr uint32_t kNoBit = 0xFFFFFFFFu;  // second bit of a two-way pass
// Bit of a round that merges nothing: every group holds one context, so the
// last (only) round takes each group as one run (segments = groups).
constexpr uint32_t kSegByGroup = 0xFFFFFFFFu;
constexpr uint64_t kCtxCap = 1ull << 20;  // contexts the merge path handles
constexpr int kEvCodeBits = 5;           // event code: 0 none, 1 + 2 * class + is_end

constexpr int kMaxClasses = 8;
constexpr int kQPairs = kMaxClasses * (kMaxClasses + 1) / 2;  // 36
constexpr int kMasks = 1 << kMaxClasses;                      // 256

// Payload of a packed record: region | (kind - 1) << 16 | overlap class << 24.
// The class is 0xFF for a record whose region has none or whose group is not
// swept (group >= G), so that matching needs no class table.
constexpr uint32_t kPayClsShift = 24;
// Set by the run scatter on the first record of each context (only the tile
// sums of that path read it).
constexpr uint32_t kPayStart = 1u << 17;
__device__ __forceinline__ uint32_t pack_payload(uint32_t region, uint32_t kind, uint32_t cls) {
  return region | ((kind - 1u) << 16) | (cls << kPayClsShift);
}
// Whether the records of a context take part in the overlap sweep.
__device__ __forceinline__ bool swept_ctx(uint32_t raw_ctx, uint32_t K, uint32_t G, uint32_t shift) {
  return K && (shift >= 32 ? 0u : (raw_ctx >> shift)) < G;
}
constexpr uint32_t kClsLds = 4096;  // region-class tables up to this size are staged in LDS

constexpr uint32_t kNoParent = 0xFFFFFFFFu;
constexpr uint32_t kParentPending = 0x80000000u;  // | tile: parent lies in an earlier tile
constexpr uint16_t kNoEnd = 0xFFFF;
constexpr uint64_t kU64Max = ~0ull;

// Source of the elements read by a sort pass.
enum SrcKind : uint32_t { kSrcPacked = 0, kSrcRecords = 1, kSrcInstances = 2 };

// How packed sort keys are laid out.  key = (ctx_rel << ts_bits) | ts_off
// when ctx_bits + ts_bits <= 64, else ("wide") key = ts_off and ctx_rel lives
// in a separate 32-bit array.  ts_off = ts - ts_min, ctx_rel = ctx - ctx_min.
struct KeySpace {
  uint64_t ts_min;
  uint64_t ts_mask;  // (1 << ts_bits) - 1, all ones for 64
  uint64_t ctx_min;
  uint32_t ts_bits;
  uint32_t ctx_bits;
  uint32_t wide;
  uint32_t pad;
};

struct SlotPlan {
  uint32_t active;
  uint32_t pos;    // digit position: 0..3 context digit, 4..11 timestamp digit
  uint32_t src;    // buffer index 0/1, or 2 = raw source
  uint32_t dst;    // buffer index 0/1
  uint32_t lb;     // look-back status array used (0/1)
  uint32_t n_out;  // valid elements written (destination bound)
  uint64_t n_elems;  // elements read (raw sources include the invalid ones)
  uint64_t tiles;
};

struct MergeRound {
  uint32_t bit;   // (lower) context bit merged in this pass
  uint32_t src;   // event buffer read (0/1)
  uint32_t dst;   // event buffer written
  uint32_t bit2;  // upper bit of a four-way pass, kNoBit for a two-way one
  uint64_t n_segs;
  uint64_t n_tiles;
};

// Written on the device by the planning kernels; read by everything else.
struct DevPlan {
  // ingest
  uint64_t n_records;
  uint64_t n_valid;
  uint64_t n_begin;
  KeySpace rec;   // record sort keys
  KeySpace ev;    // overlap event keys (context = group)
  uint32_t unsorted;     // the context-only sort left some context out of time order
  uint32_t force_full;   // ARGUS_FORCE_FULL_SORT
  uint32_t rec_final;    // buffer holding the sorted records
  uint32_t ev_final;     // buffer holding the sorted events
  uint32_t rec_active;   // active record passes so far (look-back parity)
  uint32_t pad0;
  uint64_t n_ev;         // valid overlap events
  uint64_t ev_slots;     // 2 * n_begin
  SlotPlan rs[kSlots];   // record sort
  SlotPlan es[kSlots];   // event sort
  // matching
  uint64_t match_tiles;
  // overlap events ordered by merging per-context runs
  uint32_t ev_merge;   // 1: merge path chosen (else the event radix sort)
  uint32_t m_need;     // bit b: two contexts of one group first differ in bit b
  uint32_t m_rounds;   // merge passes (set bits of m_need, taken in pairs)
  uint32_t m_nctx;     // contexts of groups < G (a prefix of the context list)
  uint64_t m_end;      // sorted position where groups >= G start (or n_valid)
  MergeRound mr[kMaxMergeBits];  // one per pass (at most kMaxMergePasses; the size keeps the layout)
  // context sort over runs of one context in the input
  uint32_t runs;       // 1: records are sorted as runs (else radix passes over records)
  uint32_t pad1;
  uint64_t n_runs;     // runs of one context in the 256-record input chunks
};

// The Python binding reads the plan back for measurement (PLAN_FIELDS in
// attr.py, checked against these lines by a test): keep its layout.
static_assert(sizeof(KeySpace) == 40, "KeySpace layout");
static_assert(sizeof(SlotPlan) == 40, "SlotPlan layout");
static_assert(sizeof(MergeRound) == 32, "MergeRound layout");
static_assert(offsetof(DevPlan, n_records) == 0, "DevPlan layout");
static_assert(offsetof(DevPlan, n_valid) == 8, "DevPlan layout");
static_assert(offsetof(DevPlan, n_begin) == 16, "DevPlan layout");
static_assert(offsetof(DevPlan, rec.ts_bits) == 48, "DevPlan layout");
static_assert(offsetof(DevPlan, rec.ctx_bits) == 52, "DevPlan layout");
static_assert(offsetof(DevPlan, rec.wide) == 56, "DevPlan layout");
static_assert(offsetof(DevPlan, unsorted) == 104, "DevPlan layout");
static_assert(offsetof(DevPlan, n_ev) == 128, "DevPlan layout");
static_assert(offsetof(DevPlan, rs) == 144, "DevPlan layout");
static_assert(offsetof(DevPlan, es) == 784, "DevPlan layout");
static_assert(offsetof(DevPlan, ev_merge) == 1432, "DevPlan layout");
static_assert(offsetof(DevPlan, m_rounds) == 1440, "DevPlan layout");
static_assert(offsetof(DevPlan, m_end) == 1448, "DevPlan layout");
static_assert(offsetof(DevPlan, mr) == 1456, "DevPlan layout");
static_assert(offsetof(DevPlan, runs) == 1712, "DevPlan layout");
static_assert(offsetof(DevPlan, n_runs) == 1720, "DevPlan layout");
static_assert(sizeof(DevPlan) == 1728, "DevPlan layout");

// Per-tile summary written by the matching kernel, read by the resolver.
struct TileDesc {
  int64_t key;       // -1 if the tile holds a context start, else lowest depth seen
  uint32_t s_in;     // depth before the tile's first element (0 if it starts a context)
  uint32_t lo_head;  // lowest depth in the part before the first context start
  uint32_t s_out;    // depth after the last element
  uint32_t lo_tail;  // lowest depth in the part after the last context start
  uint32_t op_lo;    // lowest level of an enclosing instance referenced from this tile
  uint32_t pop_base;
  uint32_t push_base;
  uint32_t op_base;
  uint32_t n_pop;    // s_in - lo_head
  uint32_t n_push;   // s_out - lo_tail
  uint32_t n_op;     // s_in - op_lo (if s_in > op_lo)
  uint32_t pad;
};

// A prefix of the records maps the depth before it to the depth after it:
// s -> max(c, s + a), or the constant c once a context starts inside.  The
// identity is {0, 0, 0} on depths >= 0.  All fields fit 32 bits (n < 2^31).
struct Fn {
  uint32_t reset;  // 1: output is the constant c (a context starts inside)
  int32_t a;
  int32_t c;       // else output is max(c, s + a)
};

// A run of matching tiles composed (one per block of the tile-sum pass).
struct BlockSum {
  Fn f;
  uint32_t nb;  // BEGINs
  uint32_t nh;  // context starts
};
constexpr uint32_t kMaxScanBlocks = 2048;  // blocks of the tile-sum pass

// Entering values of one matching tile, from a scan over the tile sums.
struct TileCarry {
  uint32_t s_in;   // depth before the tile's first record
  uint32_t hpre;   // context starts before the tile
  uint64_t nbpre;  // BEGINs before the tile
};

// Device pointers of one run (workspace carved on the host).
struct Work {
  DevPlan* plan;
  uint32_t* rec_hist;   // [12][256]
  uint32_t* rec_off;    // [12][256]
  uint32_t* ev_hist;    // [12][256]
  uint32_t* ev_off;     // [12][256]
  uint32_t* tile_ctr;   // [64] dynamic tile counters (one per launch that needs one)
  uint64_t* key[2];
  uint32_t* pay[2];
  uint32_t* ctxw[2];
  uint64_t* lb[2];      // radix look-back status, [tiles][256]
  uint64_t* tsum;       // matching tile sums, [tiles]
  TileCarry* carry;     // matching tile entering values, [tiles]
  BlockSum* bsum;       // [kMaxScanBlocks]
  uint32_t* chunk_runs; // [chunks] runs of one context in each input chunk
  uint32_t* run_base;   // [chunks] index of each chunk's first run
  uint32_t* run_cnt;    // [run_cap] valid records of each run
  uint32_t* run_pos;    // [run_cap] sorted position of each run's first valid record | starts its context << 31
  uint32_t* run_hist;   // [4][256] context-digit histograms over runs
  uint64_t* scan_bsum;  // [kMaxScanBlocks] block sums of the run scans
  uint64_t chunks;      // ceil(n / kChunk)
  uint64_t run_cap;     // runs the run path accepts
  uint64_t* slb;        // sweep look-back status, [tiles][8]
  uint64_t* mslb;       // last merge round tile records, [tiles_cap][2 + 2K + K(K + 1)]
  TileDesc* tiles;      // [match tiles]
  int64_t* tree;        // [2 * tree_leaves]
  uint64_t* pop_ts;     // per matching tile, kMatchTile entries each
  uint32_t* pop_reg;
  uint32_t* pushes;
  uint32_t* op_parent;
  uint64_t* op_sum;
  argus_instance* inst;
  uint64_t* excl;       // [n_begin] exclusive times, accumulated in place (the caller's
                        // output when it asks for them)
  uint32_t* hist_key;   // [n_begin]
  uint64_t* agg_part;   // per-block region statistics of k_agg (NULL: flushed atomically)
  uint64_t* ov_mask;    // [G][256]
  uint64_t* ov_q;       // [G][36]
  uint32_t* push_pos;   // sorted position of each pushed BEGIN (pool layout)
  uint32_t* pop_pos;    // sorted position of each popping END (pool layout)
  uint2* ctx_list;      // [ctx_cap] (context key, first sorted position)
  uint4* seg_run;       // [passes][ctx_cap + 1] starts of the segment's four runs
  uint32_t* seg_tile0;  // [passes][ctx_cap + 1] first merge tile of each segment
  uint32_t* seg_samp0;  // [passes][ctx_cap + 1] first sample of each segment (four-way)
  uint32_t* part;       // [tiles_cap] merge tasks, 48 B each (k_merge.hip)
  uint64_t ctx_cap;
  uint64_t tiles_cap;
  uint64_t lb_words;    // capacity of each lb array in words
  uint64_t tree_leaves; // power of two >= max match tiles
  uint64_t match_tiles; // upper bound (from n_records)
  uint64_t pool_cap;
};

// Run parameters shared by all launches.
struct RunArgs {
  const argus_record* rec;
  uint64_t n;
  uint32_t R, K, G, shift;
  uint32_t flags;
  const uint8_t* region_class;
  argus_attr_outputs out;
  Work w;
};

// Tile counter slots.
enum CtrSlot {
  kCtrRec = 0,     // 16 record passes
  kCtrEv = 16,     // 16 event passes
  kCtrMatch = 32,
  kCtrSweep = 33,
  kCtrMerge = 34,  // 8 merge rounds
  kCtrCount = 64
};

// Run lists of the input chunks.  The ingest's waves take chunks g, g + W,
// g + 2W, ... (W waves); each wave stages its chunks' lists and writes them
// out in bursts, one wave's after another's: a chunk's list count and place
// go to the entry at chunk_slot(c) of the chunk table, its runs to the run
// buffer from 256 * wave_slot0(g) on.  With chunks = q W + r, wave g takes
// q + (g < r) chunks.
struct ChunkWaves {
  uint32_t W;
  uint64_t q, r;
};
__host__ __device__ inline ChunkWaves chunk_waves(uint64_t chunks, uint32_t W) {
  return ChunkWaves{W, chunks / W, chunks % W};
}
__host__ __device__ inline uint64_t wave_slot0(const ChunkWaves& cw, uint64_t g) {
  return g * cw.q + (g < cw.r ? g : cw.r);
}
__host__ __device__ inline uint64_t chunk_slot(const ChunkWaves& cw, uint64_t c) {
  return wave_slot0(cw, c % cw.W) + c / cw.W;
}
// chunk table entry: run count (<= 256) | first run's place in the wave's list << 9
constexpr uint32_t kChunkCountBits = 9;
// run position word (by run id): first sorted position | starts its context << 31
constexpr uint32_t kRunPosMask = 0x7FFFFFFFu;
// the ingest's grid for n records (four waves per block)
__host__ __device__ inline uint32_t ingest_blocks(uint64_t n) {
  uint64_t blocks = (n + 256 * 4 * 4 - 1) / (256 * 4 * 4);
  if (blocks > 1024) blocks = 1024;
  return blocks < 1 ? 1u : (uint32_t)blocks;
}

// ------------------------------------------------------- device helpers
#if defined(__HIP_DEVICE_COMPILE__)
#define ARGUS_DEV __device__ __forceinline__
#else
#define ARGUS_DEV __device__ inline
#endif

ARGUS_DEV uint64_t ld_agent(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
ARGUS_DEV void st_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
ARGUS_DEV void backoff() { __builtin_amdgcn_s_sleep(1); }

// Look-back waits are bounded: a predecessor tile always publishes within
// microseconds, so running out of spins means an internal error.  The wait
// then gives up (the kernel finishes, results are wrong) and the error is
// reported in counter ARGUS_C_INTERNAL_ERROR instead of hanging the GPU.
constexpr uint32_t kMaxSpins = 1u << 24;
ARGUS_DEV void flag_internal_error(uint64_t* counters, uint64_t code) {
  atomicOr((unsigned long long*)&counters[31], (unsigned long long)code);
}

ARGUS_DEV unsigned lane_id() { return __lane_id(); }
ARGUS_DEV uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

ARGUS_DEV uint32_t bit_width64(uint64_t v) { return v ? 64u - (uint32_t)__clzll(v) : 0u; }

// ------------------------------------------------- cross-lane (DPP) helpers
// gfx9 DPP controls: quad permutations, mirrors inside a row of 16 lanes,
// shifts inside a row, and broadcasts of a row's lane 15 to the next rows.
constexpr int kDppQuad1032 = 0xB1;    // quad_perm:[1,0,3,2]
constexpr int kDppQuad2301 = 0x4E;    // quad_perm:[2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror
constexpr int kDppMirror = 0x140;      // row_mirror
constexpr int kDppRowShr = 0x110;      // row_shr:n is kDppRowShr + n
constexpr int kDppBcast15 = 0x142;     // row_bcast:15
constexpr int kDppBcast31 = 0x143;     // row_bcast:31
constexpr int kDppWaveShr1 = 0x138;    // wave_shr:1 (whole wave, one lane up)

template <int CTRL, int ROWS = 0xF>
ARGUS_DEV uint32_t dpp32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xF, false);
}

// The value of lane i - 1 in lane i, and `first` in lane 0 (one DPP move).
ARGUS_DEV uint32_t lane_prev(uint32_t v, uint32_t first) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)first, (int)v, kDppWaveShr1, 0xF, 0xF, false);
}

// Sum over each row of 16 lanes, in every lane of the row.
ARGUS_DEV uint32_t row_sum32(uint32_t v) {
  v += dpp32<kDppQuad1032>(v);
  v += dpp32<kDppQuad2301>(v);
  v += dpp32<kDppHalfMirror>(v);
  v += dpp32<kDppMirror>(v);
  return v;
}
ARGUS_DEV uint64_t row_sum64(uint64_t v) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
#define ARGUS_ROW_STEP(C)                                              \
  {                                                                    \
    const uint64_t o = (uint64_t)dpp32<C>(lo) | ((uint64_t)dpp32<C>(hi) << 32); \
    const uint64_t r = ((uint64_t)lo | ((uint64_t)hi << 32)) + o;      \
    lo = (uint32_t)r;                                                  \
    hi = (uint32_t)(r >> 32);                                          \
  }
  ARGUS_ROW_STEP(kDppQuad1032)
  ARGUS_ROW_STEP(kDppQuad2301)
  ARGUS_ROW_STEP(kDppHalfMirror)
  ARGUS_ROW_STEP(kDppMirror)
#undef ARGUS_ROW_STEP
  return (uint64_t)lo | ((uint64_t)hi << 32);
}
ARGUS_DEV int32_t row_min32(int32_t v) {
  int32_t o;
  o = (int32_t)dpp32<kDppQuad1032>((uint32_t)v); v = o < v ? o : v;
  o = (int32_t)dpp32<kDppQuad2301>((uint32_t)v); v = o < v ? o : v;
  o = (int32_t)dpp32<kDppHalfMirror>((uint32_t)v); v = o < v ? o : v;
  o = (int32_t)dpp32<kDppMirror>((uint32_t)v); v = o < v ? o : v;
  return v;
}
// Wave-wide results from per-row results (lanes 0, 16, 32, 48), as scalars.
ARGUS_DEV uint32_t rows_sum32(uint32_t v) {
  return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16) +
         __builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48);
}
ARGUS_DEV uint64_t rows_sum64(uint64_t v) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  uint64_t r = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    r += (uint64_t)(uint32_t)__builtin_amdgcn_readlane(lo, 16 * q) |
         ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(hi, 16 * q) << 32);
  return r;
}
ARGUS_DEV int32_t rows_min32(int32_t v) {
  int32_t a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
  int32_t c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
  a = a < b ? a : b;
  c = c < d ? c : d;
  return a < c ? a : c;
}

// Wave sums of many 64-bit values at once, by halving: at each of five
// levels the lanes pair up across a distance (32, 16, 8, 4, 2), each pair of
// values becomes one whose sum runs over both lanes, and each lane keeps the
// half selected by its bit of that distance; a last step adds lanes 2k and
// 2k + 1.  Lane l then holds the total of value bitrev5(l >> 1) (five bits).
// The distances 32 and 16 use the gfx950 lane-half swaps, the others DPP.
constexpr int kDppRowRor8 = 0x128;  // row_ror:8 (lane i ^ 8 inside a row)
ARGUS_DEV uint64_t join64(uint32_t lo, uint32_t hi) { return (uint64_t)lo | ((uint64_t)hi << 32); }
template <int N, bool HALF32>
ARGUS_DEV void sums_level_swap(const uint64_t (&a)[N], uint64_t (&o)[(N + 1) / 2]) {
#pragma unroll
  for (int k = 0; k < (N + 1) / 2; ++k) {
    const uint64_t x = a[2 * k], y = 2 * k + 1 < N ? a[2 * k + 1] : 0ull;
    const uint32_t xl = (uint32_t)x, xh = (uint32_t)(x >> 32), yl = (uint32_t)y, yh = (uint32_t)(y >> 32);
    if constexpr (HALF32) {
      // lanes 32..63 of x trade places with lanes 0..31 of y
      const auto l = __builtin_amdgcn_permlane32_swap(xl, yl, false, false);
      const auto h = __builtin_amdgcn_permlane32_swap(xh, yh, false, false);
      o[k] = join64(l[0], h[0]) + join64(l[1], h[1]);
    } else {
      // the odd rows of x trade places with the even rows of y
      const auto l = __builtin_amdgcn_permlane16_swap(xl, yl, false, false);
      const auto h = __builtin_amdgcn_permlane16_swap(xh, yh, false, false);
      o[k] = join64(l[0], h[0]) + join64(l[1], h[1]);
    }
  }
}
template <int N, int CTRL>
ARGUS_DEV void sums_level_dpp(const uint64_t (&a)[N], uint64_t (&o)[(N + 1) / 2], bool odd) {
#pragma unroll
  for (int k = 0; k < (N + 1) / 2; ++k) {
    const uint64_t x = a[2 * k], y = 2 * k + 1 < N ? a[2 * k + 1] : 0ull;
    const uint64_t keep = odd ? y : x, send = odd ? x : y;
    o[k] = keep + join64(dpp32<CTRL>((uint32_t)send), dpp32<CTRL>((uint32_t)(send >> 32)));
  }
}
template <int V>
ARGUS_DEV uint64_t wave_sums64(const uint64_t (&v)[V], uint32_t* idx) {
  static_assert(V >= 1 && V <= 32, "at most 32 values");
  constexpr int N1 = (V + 1) / 2, N2 = (N1 + 1) / 2, N3 = (N2 + 1) / 2, N4 = (N3 + 1) / 2;
  constexpr int N5 = (N4 + 1) / 2;
  const uint32_t lane = __lane_id();
  uint64_t a1[N1], a2[N2], a3[N3], a4[N4], a5[N5];
  sums_level_swap<V, true>(v, a1);
  sums_level_swap<N1, false>(a1, a2);
  sums_level_dpp<N2, kDppRowRor8>(a2, a3, (lane >> 3) & 1u);
  sums_level_dpp<N3, kDppHalfMirror>(a3, a4, (lane >> 2) & 1u);  // partner 7 - i: bit 2 differs
  sums_level_dpp<N4, kDppQuad2301>(a4, a5, (lane >> 1) & 1u);
  uint64_t r = a5[0];
  r += join64(dpp32<kDppQuad1032>((uint32_t)r), dpp32<kDppQuad1032>((uint32_t)(r >> 32)));
  *idx = ((lane >> 1) & 1u) << 4 | ((lane >> 2) & 1u) << 3 | ((lane >> 3) & 1u) << 2 |
         ((lane >> 4) & 1u) << 1 | ((lane >> 5) & 1u);
  return r;
}

// Inclusive prefix sum over the 64 lanes of the wave.
ARGUS_DEV int32_t wave_incl_scan32(int32_t v) {
  v += (int32_t)dpp32<kDppRowShr + 1>((uint32_t)v);
  v += (int32_t)dpp32<kDppRowShr + 2>((uint32_t)v);
  v += (int32_t)dpp32<kDppRowShr + 4>((uint32_t)v);
  v += (int32_t)dpp32<kDppRowShr + 8>((uint32_t)v);
  v += (int32_t)dpp32<kDppBcast15, 0xA>((uint32_t)v);
  v += (int32_t)dpp32<kDppBcast31, 0xC>((uint32_t)v);
  return v;
}

// ------------------------------------------------- clamped depth maps

ARGUS_DEV Fn fn_id() { return Fn{0u, 0, 0}; }
// g after f
ARGUS_DEV Fn compose(const Fn& f, const Fn& g) {
  Fn r;
  r.reset = g.reset | f.reset;
  r.a = g.reset ? g.a : (f.reset ? 0 : f.a + g.a);
  r.c = g.reset ? g.c : (f.c + g.a > g.c ? f.c + g.a : g.c);
  return r;
}
ARGUS_DEV int64_t apply(const Fn& f, int64_t s) {
  if (f.reset) return f.c;
  return s + f.a > f.c ? s + f.a : f.c;
}
template <int CTRL, int ROWS = 0xF>
ARGUS_DEV Fn dpp_fn(const Fn& f) {
  return Fn{dpp32<CTRL, ROWS>(f.reset), (int32_t)dpp32<CTRL, ROWS>((uint32_t)f.a),
            (int32_t)dpp32<CTRL, ROWS>((uint32_t)f.c)};
}
ARGUS_DEV Fn shfl_down_fn(const Fn& f, int o) {
  return Fn{(uint32_t)__shfl_down((int)f.reset, o), __shfl_down(f.a, o), __shfl_down(f.c, o)};
}
ARGUS_DEV Fn shfl_fn(const Fn& f, int src) {
  return Fn{(uint32_t)__shfl((int)f.reset, src), __shfl(f.a, src), __shfl(f.c, src)};
}
// Inclusive scan of the maps over the wave (lane order = record order).
ARGUS_DEV Fn wave_scan_fn(Fn x) {
  x = compose(dpp_fn<kDppRowShr + 1>(x), x);
  x = compose(dpp_fn<kDppRowShr + 2>(x), x);
  x = compose(dpp_fn<kDppRowShr + 4>(x), x);
  x = compose(dpp_fn<kDppRowShr + 8>(x), x);
  x = compose(dpp_fn<kDppBcast15, 0xA>(x), x);
  x = compose(dpp_fn<kDppBcast31, 0xC>(x), x);
  return x;
}

// Summary of one matching tile (2048 records) in one word: number of
// BEGINs (12 bits), c (12 bits), a + 2048 (13 bits), reset (1 bit), number
// of context starts (12 bits).  BEGIN and start counts travel packed as
// nb | starts << 16.
ARGUS_DEV uint64_t pack_tile_sum(const Fn& f, uint32_t nbh) {
  return ((uint64_t)(nbh >> 16) << 41) | ((uint64_t)f.reset << 40) |
         ((uint64_t)(uint32_t)(f.a + 2048) << 24) | ((uint64_t)(uint32_t)f.c << 12) |
         (uint64_t)(nbh & 0xFFFFu);
}
ARGUS_DEV void unpack_tile_sum(uint64_t v, Fn* f, uint32_t* nbh) {
  f->reset = (uint32_t)(v >> 40) & 1u;
  f->a = (int32_t)((v >> 24) & 0x1FFFull) - 2048;
  f->c = (int32_t)((v >> 12) & 0xFFFull);
  *nbh = (uint32_t)(v & 0xFFFull) | ((uint32_t)((v >> 41) & 0xFFFull) << 16);
}

// Look-back status words: bits 62..63 hold the state, bits 0..61 the value.
constexpr uint64_t kFlagAgg = 1ull << 62;
constexpr uint64_t kFlagIncl = 2ull << 62;
constexpr uint64_t kValMask = (1ull << 62) - 1;

// ------------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error.
hipError_t launch_init(const RunArgs& a, hipStream_t s);
hipError_t launch_ingest(const RunArgs& a, hipStream_t s);
hipError_t launch_plan(const RunArgs& a, hipStream_t s);
hipError_t launch_radix_pass(const RunArgs& a, int which /*0 rec, 1 ev*/, int slot,
                             uint64_t max_elems, hipStream_t s);
hipError_t launch_tsum(const RunArgs& a, int mode, hipStream_t s);
hipError_t launch_runs_base(const RunArgs& a, hipStream_t s);
hipError_t launch_runs_compact(const RunArgs& a, hipStream_t s);
hipError_t launch_runs_plan(const RunArgs& a, hipStream_t s);
hipError_t launch_runs_pos(const RunArgs& a, hipStream_t s);
hipError_t launch_runs_scatter(const RunArgs& a, hipStream_t s);
hipError_t launch_lb_clear(const RunArgs& a, hipStream_t s);
hipError_t launch_mscan(const RunArgs& a, hipStream_t s);
hipError_t launch_ts_hist(const RunArgs& a, hipStream_t s);
hipError_t launch_plan2(const RunArgs& a, hipStream_t s);
hipError_t launch_match(const RunArgs& a, hipStream_t s);
hipError_t launch_tree(const RunArgs& a, hipStream_t s);
hipError_t launch_resolve(const RunArgs& a, hipStream_t s);
hipError_t launch_runs_check(const RunArgs& a, hipStream_t s);
hipError_t launch_tsum_codes(const RunArgs& a, hipStream_t s);
hipError_t launch_agg(const RunArgs& a, hipStream_t s);
// Words of the per-block statistics buffer of k_agg for n records (0: none).
uint64_t agg_part_words(uint64_t n, uint32_t R);
hipError_t launch_hist(const RunArgs& a, hipStream_t s);
// Log2 histograms of instances from their keys (region << 16 | incl bin << 8
// | excl bin, 0xFFFFFFFF: none), *d_count of them (at most count_max), added
// into the region rows (k_agg.hip).
hipError_t launch_hist_keys(const uint32_t* keys, const uint64_t* d_count, uint64_t count_max,
                            uint64_t* rstats, uint32_t R, hipStream_t s);
hipError_t launch_ev_plan(const RunArgs& a, hipStream_t s);
hipError_t launch_ev_clear(const RunArgs& a, hipStream_t s);
hipError_t launch_mplan(const RunArgs& a, hipStream_t s);
hipError_t launch_mseg(const RunArgs& a, int rounds, hipStream_t s);
hipError_t launch_mpart(const RunArgs& a, int round, hipStream_t s);
hipError_t launch_merge(const RunArgs& a, int round, hipStream_t s);
hipError_t launch_merge_sweep(const RunArgs& a, hipStream_t s);
hipError_t launch_sweep(const RunArgs& a, hipStream_t s);
hipError_t launch_ov_final(const RunArgs& a, hipStream_t s);

// Number of blocks of `kernel` that fit on the device at once (all CUs at
// the kernel's occupancy): the grid of a persistent kernel.
uint64_t persistent_blocks(const void* kernel, int threads);

// Launch geometry helpers shared by host code.
__host__ __device__ inline uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

}  // namespace argus
