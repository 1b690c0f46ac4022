// k_ingest.hip -- run initialisation, record validation and the sort plans.
//
// Validation follows the definition of a marker record: only BEGIN (1) and
// END (2) transitions of known regions (id < R) carry region identity (the
// paper's Section 3.2); anything else is counted and dropped.
#include "internal.h"

namespace argus {

// ---------------------------------------------------------------- helpers

// Lanes of the wave whose 8-bit value equals this lane's (restricted to
// `valid`): eight ballots, one per bit.
__device__ __forceinline__ uint64_t peers8(uint32_t d, uint64_t valid) {
  uint64_t m = valid;
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const uint32_t bit = (d >> b) & 1u;
    const uint64_t v = __ballot(bit);
    m &= bit ? v : ~v;
  }
  return m;
}

// Add this wave's values of digit `d` (for lanes in `valid`) into an LDS
// histogram with one atomic per distinct digit.
__device__ __forceinline__ void wave_hist_add(uint32_t* hist, uint32_t d, bool valid) {
  const uint64_t vm = __ballot(valid);
  if (vm == 0) return;
  const uint64_t peers = peers8(d, vm);
  if (valid && (peers >> lane_id()) == 1ull) atomicAdd(&hist[d], (uint32_t)__popcll(peers));
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
template <typename T>
__device__ __forceinline__ T wave_min(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    T u = __shfl_xor(v, o);
    v = u < v ? u : v;
  }
  return v;
}
template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    T u = __shfl_xor(v, o);
    v = u > v ? u : v;
  }
  return v;
}

// Exclusive prefix sum over 256 values held one per thread of a 256-thread
// block; returns the exclusive prefix, writes the total to *total.
__device__ __forceinline__ uint32_t block_excl_scan256(uint32_t v, uint32_t* scratch4,
                                                       uint32_t* total) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) scratch4[w] = x;
  __syncthreads();
  uint32_t pre = 0, tot = 0;
  for (int k = 0; k < 4; ++k) {
    if (k < w) pre += scratch4[k];
    tot += scratch4[k];
  }
  __syncthreads();
  *total = tot;
  return pre + x - v;
}

// ------------------------------------------------- runs of one context
// A wave holds one input chunk of 256 records as 4 rows of 64 lanes (record
// 64 j + lane of the chunk in row j); masks over the chunk have bit
// p = 64 j + lane in word j.
static_assert(kChunk == 256, "a chunk is 4 rows of a wave");

// Run heads (a record whose predecessor in the chunk has another context,
// or the chunk's first record) and valid records of the chunk.
__device__ __forceinline__ void chunk_masks(const uint32_t (&ctx)[4], const bool (&in)[4],
                                            const bool (&valid)[4], uint64_t (&H)[4],
                                            uint64_t (&V)[4]) {
  const uint32_t lane = lane_id();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    // previous record: the previous lane, or the last lane of the row before
    const uint32_t prev =
        lane_prev(ctx[j], j > 0 ? (uint32_t)__builtin_amdgcn_readlane((int)ctx[j > 0 ? j - 1 : 0], 63) : ctx[j]);
    const bool head = in[j] && ((j == 0 && lane == 0) || prev != ctx[j]);
    H[j] = __ballot(head);
    V[j] = __ballot(valid[j]);
  }
}

// ------------------------------------------------------------------ init

struct Fill {
  uint64_t* p;
  uint64_t n;
  uint64_t v;
};
constexpr int kMaxFill = 16;
struct FillList {
  Fill f[kMaxFill];
  int count;
  uint64_t n_records;
  uint32_t R;
  uint32_t force_full;
  uint64_t* counters;
  uint64_t* rstats;
  DevPlan* plan;
};

// Initialises every output and the parts of the workspace that a run needs
// zeroed.  A fill kernel rather than hipMemsetAsync keeps the run
// capturable into a HIP graph.
__global__ __launch_bounds__(256) void k_init(FillList fl) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t tid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int s = 0; s < fl.count; ++s) {
    const Fill f = fl.f[s];
    for (uint64_t i = tid; i < f.n; i += stride) f.p[i] = f.v;
  }
  // counters
  if (tid < ARGUS_NUM_COUNTERS) {
    uint64_t v = 0;
    if (tid == ARGUS_C_N_RECORDS) v = fl.n_records;
    if (tid == ARGUS_C_TS_MIN || tid == ARGUS_C_CTX_MIN) v = kU64Max;
    fl.counters[tid] = v;
  }
  // region statistics: zero, except the minima
  const uint64_t nrs = (uint64_t)fl.R * ARGUS_RS_WIDTH;
  for (uint64_t i = tid; i < nrs; i += stride) {
    const uint32_t col = (uint32_t)(i % ARGUS_RS_WIDTH);
    fl.rstats[i] = (col == ARGUS_RS_INCL_MIN || col == ARGUS_RS_EXCL_MIN) ? kU64Max : 0;
  }
  if (tid == 0) {
    fl.plan->n_records = fl.n_records;
    fl.plan->force_full = fl.force_full;
  }
}

hipError_t launch_init(const RunArgs& a, hipStream_t s) {
  FillList fl{};
  const Work& w = a.w;
  auto add = [&](void* p, uint64_t bytes, uint64_t v) {
    if (fl.count < kMaxFill && bytes >= 8) fl.f[fl.count++] = Fill{(uint64_t*)p, bytes / 8, v};
  };
  add(w.plan, sizeof(DevPlan), 0);
  add(w.rec_hist, sizeof(uint32_t) * kDigitPositions * kRadixBins, 0);
  add(w.ev_hist, sizeof(uint32_t) * kDigitPositions * kRadixBins, 0);
  add(w.tile_ctr, sizeof(uint32_t) * kCtrCount, 0);
  add(w.run_hist, sizeof(uint32_t) * 4 * kRadixBins, 0);
  // look-back status of the first record pass (its tiles cover every record)
  add(w.lb[0], sizeof(uint64_t) * ceil_div(a.n ? a.n : 1, kSortTile) * kRadixBins, 0);
  add(w.slb, sizeof(uint64_t) * 8 * ceil_div(a.n ? a.n : 1, kSweepTile), 0);
  if (a.K > 0) {
    add(w.ov_mask, sizeof(uint64_t) * kMasks * a.G, 0);
    add(w.ov_q, sizeof(uint64_t) * kQPairs * a.G, 0);
    add(a.out.d_overlap_group, sizeof(uint64_t) * 2ull * a.K * a.K * a.G, 0);
    add(a.out.d_overlap_global, sizeof(uint64_t) * 2ull * a.K * a.K, 0);
  }
  fl.n_records = a.n;
  fl.R = a.R;
  fl.force_full = (a.flags & ARGUS_FORCE_FULL_SORT) ? 1u : 0u;
  fl.counters = a.out.d_counters;
  fl.rstats = a.out.d_region_stats;
  fl.plan = w.plan;
  uint64_t most = (uint64_t)a.R * ARGUS_RS_WIDTH;
  for (int i = 0; i < fl.count; ++i) most = most > fl.f[i].n ? most : fl.f[i].n;
  uint64_t blocks = ceil_div(most, 256 * 4);
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_init, dim3((uint32_t)blocks), dim3(256), 0, s, fl);
  return hipGetLastError();
}

// ---------------------------------------------------------------- ingest

struct IngestArgs {
  const uint4* rec;
  uint64_t n;
  uint32_t R;
  uint64_t* counters;
  uint32_t* hist;        // rec_hist: positions 0..3 (raw context digits)
  DevPlan* plan;         // n_runs
  uint64_t* runs_raw;    // [chunk * 256 + j]: context | valid records << 32 of run j
  uint32_t* chunk_runs;  // [chunk slot]: count | place << kChunkCountBits
};

// Staged run lists per wave (entries; chunk table words).
constexpr uint32_t kStageRuns = 512;
constexpr uint32_t kStageChunks = 256;
static_assert(kStageRuns >= kChunk, "a chunk's runs fit the stage");

// One coalesced 16-byte load per record.  Counts kinds and regions, reduces
// the timestamp and context ranges of valid records, and builds the 256-bin
// histograms of the four raw context digits (used by the context passes of
// the sort).  Each wave step covers one 256-record chunk, whose runs of one
// context (and their valid records) are recorded for the context sort over
// runs; the histograms and the context range are added per run.
__global__ __launch_bounds__(256) void k_ingest(IngestArgs a) {
  __shared__ uint32_t s_hist[4][kRadixBins];
  __shared__ uint64_t s_red[4][8];
  __shared__ unsigned long long s_runs;
  __shared__ uint64_t s_stage[4][kStageRuns];
  __shared__ uint32_t s_ctab[4][kStageChunks];
  if (threadIdx.x == 0) s_runs = 0;
  for (int i = threadIdx.x; i < 4 * kRadixBins; i += 256) (&s_hist[0][0])[i] = 0;
  __syncthreads();

  // Counts are wave-uniform (from ballots); extremes are per lane.
  uint64_t n_valid = 0, n_badk = 0, n_badr = 0, n_begin = 0;
  uint64_t ts_min = kU64Max, ts_max = 0;
  uint64_t ctx_min = kU64Max, ctx_max = 0;
  // Each wave takes 4 x 64 consecutive records per step (4 loads in flight
  // per lane); every lane of a wave iterates the same number of times.
  constexpr int kPer = 4;
  const uint64_t stride = (uint64_t)gridDim.x * 256 * kPer;
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t first = ((uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * (64 * kPer);
  static_assert(kPer * 64 == kChunk, "a wave step is one chunk");
  uint64_t wave_runs = 0;
  // this wave's run list and chunk table words: staged, then written out
  const uint32_t wv = threadIdx.x >> 6;
  const ChunkWaves cw = chunk_waves((a.n + kChunk - 1) / kChunk, gridDim.x * 4);
  const uint64_t slot0 = wave_slot0(cw, (uint64_t)blockIdx.x * 4 + wv);
  uint64_t* const list = a.runs_raw + slot0 * kChunk;
  uint32_t n_out = 0, n_staged = 0;  // runs written out, runs staged
  uint32_t c_out = 0, c_staged = 0;  // chunk words written out, staged
  auto wave_sync = [] {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  auto flush_runs = [&] {
    wave_sync();
    for (uint32_t i = lane; i < n_staged; i += 64) list[n_out + i] = s_stage[wv][i];
    n_out += n_staged;
    n_staged = 0;
    wave_sync();
  };
  auto flush_chunks = [&] {
    wave_sync();
    for (uint32_t i = lane; i < c_staged; i += 64) a.chunk_runs[slot0 + c_out + i] = s_ctab[wv][i];
    c_out += c_staged;
    c_staged = 0;
    wave_sync();
  };
  uint4 nr_[kPer];  // the next chunk, loaded while this one is processed
  auto issue = [&](uint64_t b) {
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint64_t i = b + (uint64_t)j * 64 + lane;
      nr_[j] = a.rec[i < a.n ? i : a.n - 1];
    }
  };
  if (first < a.n) issue(first);
  for (uint64_t base = first; base < a.n; base += stride) {
    uint4 r[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) r[j] = nr_[j];
    if (base + stride < a.n) issue(base + stride);
    uint32_t cx[kPer];
    bool inr[kPer], vl[kPer];
    const uint32_t rem = a.n - base < (uint64_t)kChunk ? (uint32_t)(a.n - base) : (uint32_t)kChunk;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint32_t kind = (r[j].w >> 16) & 0xFFu;
      const uint32_t region = r[j].w & 0xFFFFu;
      const bool kind_ok = kind == 1 || kind == 2;
      cx[j] = r[j].z;
      inr[j] = 64u * j + lane < rem;
      vl[j] = inr[j] && kind_ok && region < a.R;
      n_badk += (uint64_t)__popcll(__ballot(inr[j] && !kind_ok));
      n_badr += (uint64_t)__popcll(__ballot(inr[j] && kind_ok && region >= a.R));
      n_begin += (uint64_t)__popcll(__ballot(vl[j] && kind == 1));
      const uint64_t ts = (uint64_t)r[j].x | ((uint64_t)r[j].y << 32);
      ts_min = vl[j] && ts < ts_min ? ts : ts_min;
      ts_max = vl[j] && ts > ts_max ? ts : ts_max;
    }
    // runs of one context in this chunk
    uint64_t H[4], V[4];
    chunk_masks(cx, inr, vl, H, V);
    uint32_t nr = 0, nvc = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      nr += (uint32_t)__popcll(H[j]);
      nvc += (uint32_t)__popcll(V[j]);
    }
    n_valid += nvc;
    if (n_staged + nr > kStageRuns) flush_runs();
    if (c_staged == kStageChunks) flush_chunks();
    // per row (wave-uniform): heads and valid records before it, and the
    // valid records before the first head of the rows after it (all of the
    // chunk's if none)
    uint32_t hbase[kPer], vbase[kPer], vnext[kPer];
    {
      uint32_t hb = 0, vb = 0;
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        hbase[j] = hb;
        vbase[j] = vb;
        hb += (uint32_t)__popcll(H[j]);
        vb += (uint32_t)__popcll(V[j]);
      }
      uint32_t vn = vb;
#pragma unroll
      for (int j = kPer - 1; j >= 0; --j) {
        vnext[j] = vn;
        if (H[j]) {
          const uint32_t b = (uint32_t)__ffsll((unsigned long long)H[j]) - 1u;
          vn = vbase[j] + (uint32_t)__popcll(V[j] & ((1ull << b) - 1ull));
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      if (!((H[j] >> lane) & 1ull)) continue;
      const uint32_t li = hbase[j] + __builtin_amdgcn_mbcnt_hi((uint32_t)(H[j] >> 32),
                                                                __builtin_amdgcn_mbcnt_lo((uint32_t)H[j], 0u));
      const uint32_t vp = vbase[j] + __builtin_amdgcn_mbcnt_hi((uint32_t)(V[j] >> 32),
                                                                __builtin_amdgcn_mbcnt_lo((uint32_t)V[j], 0u));
      // the next head in this row (two shifts: lane + 1 may be 64)
      const uint64_t later = H[j] & ((~0ull << lane) << 1);
      uint32_t vq = vnext[j];
      if (later) {
        const uint32_t b = (uint32_t)__ffsll((unsigned long long)later) - 1u;
        vq = vbase[j] + (uint32_t)__popcll(V[j] & ((1ull << b) - 1ull));
      }
      const uint32_t cnt = vq - vp;
      s_stage[wv][n_staged + li] = (uint64_t)cx[j] | ((uint64_t)cnt << 32);
      if (cnt) {
        // the context range, and the context digit histograms, per run
        ctx_min = cx[j] < ctx_min ? cx[j] : ctx_min;
        ctx_max = cx[j] > ctx_max ? cx[j] : ctx_max;
#pragma unroll
        for (int d = 0; d < 4; ++d) atomicAdd(&s_hist[d][(cx[j] >> (8 * d)) & 0xFFu], cnt);
      }
    }
    if (lane == 0) s_ctab[wv][c_staged] = nr | ((n_out + n_staged) << kChunkCountBits);
    ++c_staged;
    n_staged += nr;
    wave_runs += nr;
  }
  if (n_staged) flush_runs();
  if (c_staged) flush_chunks();
  ts_min = wave_min(ts_min);
  ts_max = wave_max(ts_max);
  const uint64_t cmin = wave_min(ctx_min);
  const uint64_t cmax = wave_max(ctx_max);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0 && wave_runs) atomicAdd(&s_runs, (unsigned long long)wave_runs);
  if ((threadIdx.x & 63) == 0) {
    s_red[w][0] = n_valid;
    s_red[w][1] = n_badk;
    s_red[w][2] = n_badr;
    s_red[w][3] = n_begin;
    s_red[w][4] = ts_min;
    s_red[w][5] = ts_max;
    s_red[w][6] = cmin;
    s_red[w][7] = cmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t v[8];
    for (int k = 0; k < 8; ++k) v[k] = s_red[0][k];
    for (int q = 1; q < 4; ++q) {
      for (int k = 0; k < 4; ++k) v[k] += s_red[q][k];
      v[4] = s_red[q][4] < v[4] ? s_red[q][4] : v[4];
      v[5] = s_red[q][5] > v[5] ? s_red[q][5] : v[5];
      v[6] = s_red[q][6] < v[6] ? s_red[q][6] : v[6];
      v[7] = s_red[q][7] > v[7] ? s_red[q][7] : v[7];
    }
    unsigned long long* c = (unsigned long long*)a.counters;
    if (v[0]) atomicAdd(&c[ARGUS_C_N_VALID], v[0]);
    if (v[1]) atomicAdd(&c[ARGUS_C_N_BAD_KIND], v[1]);
    if (v[2]) atomicAdd(&c[ARGUS_C_N_BAD_REGION], v[2]);
    if (v[3]) atomicAdd(&c[ARGUS_C_N_BEGIN], v[3]);
    if (v[0] - v[3]) atomicAdd(&c[ARGUS_C_N_END], v[0] - v[3]);
    if (s_runs) atomicAdd((unsigned long long*)&a.plan->n_runs, s_runs);
    if (v[0]) {
      atomicMin(&c[ARGUS_C_TS_MIN], v[4]);
      atomicMax(&c[ARGUS_C_TS_MAX], v[5]);
      atomicMin(&c[ARGUS_C_CTX_MIN], v[6]);
      atomicMax(&c[ARGUS_C_CTX_MAX], v[7]);
    }
  }
  for (int i = threadIdx.x; i < 4 * kRadixBins; i += 256) {
    const uint32_t h = (&s_hist[0][0])[i];
    if (h) atomicAdd(&a.hist[i], h);
  }
}

hipError_t launch_ingest(const RunArgs& a, hipStream_t s) {
  IngestArgs ia{(const uint4*)a.rec, a.n, a.R, a.out.d_counters, a.w.rec_hist, a.w.plan,
                a.w.key[1], a.w.chunk_runs};
  // up to 1024 blocks: four waves per SIMD, each streaming many chunks
  // (measured faster than more or fewer on the 2^28-record trace)
  hipLaunchKernelGGL(k_ingest, dim3(ingest_blocks(a.n)), dim3(256), 0, s, ia);
  return hipGetLastError();
}

// ------------------------------------------------------------------ plan

struct PlanArgs {
  DevPlan* plan;
  const uint64_t* counters;
  const uint32_t* hist;  // rec_hist
  uint32_t* off;         // rec_off
  uint32_t phase;        // 1: context passes; 2: full sort (if needed)
  uint32_t force_radix;  // ARGUS_FORCE_RECORD_RADIX
  uint64_t run_cap;      // runs the run path accepts
};

__device__ __forceinline__ uint64_t mask_bits(uint32_t bits) {
  return bits >= 64 ? kU64Max : ((1ull << bits) - 1);
}

// Plans the passes of one sort phase on the device (no host round trip).
// A digit position is active if more than one bin of its histogram is used;
// active passes ping-pong between the two buffers and the two look-back
// status arrays; the first pass of the record sort reads the raw records.
__global__ __launch_bounds__(256) void k_plan(PlanArgs a) {
  __shared__ uint32_t s_scr[4];
  __shared__ uint32_t s_active[kDigitPositions];
  DevPlan* p = a.plan;
  const int t = threadIdx.x;
  if (a.phase == 2 && !p->unsorted) return;
  const uint64_t n_valid = a.counters[ARGUS_C_N_VALID];
  if (a.phase == 1 && t == 0) {
    p->n_valid = n_valid;
    p->n_begin = a.counters[ARGUS_C_N_BEGIN];
    KeySpace k{};
    if (n_valid) {
      const uint64_t ts_min = a.counters[ARGUS_C_TS_MIN], ts_max = a.counters[ARGUS_C_TS_MAX];
      const uint64_t c_min = a.counters[ARGUS_C_CTX_MIN], c_max = a.counters[ARGUS_C_CTX_MAX];
      k.ts_min = ts_min;
      k.ts_bits = bit_width64(ts_max - ts_min);
      k.ctx_min = c_min;
      k.ctx_bits = bit_width64(c_max - c_min);
    }
    k.ts_mask = mask_bits(k.ts_bits);
    k.wide = (k.ts_bits + k.ctx_bits > 64) ? 1u : 0u;
    p->rec = k;
    p->match_tiles = ceil_div(n_valid, kMatchTile);
    // Long runs of one context in the input (per-warp buffers written in
    // chunks): sort the runs, then place the records, instead of radix
    // passes over every record.
    p->runs = (!a.force_radix && !k.wide && n_valid > 0 && p->n_runs <= a.run_cap) ? 1u : 0u;
  }
  // Histogram triviality and exclusive offsets for the positions of this phase.
  const int pos_lo = 0, pos_hi = a.phase == 1 ? 4 : kDigitPositions;
  for (int pos = pos_lo; pos < pos_hi; ++pos) {
    const uint32_t h = a.hist[pos * kRadixBins + t];
    const int used = __syncthreads_count(h != 0);
    uint32_t total;
    const uint32_t ex = block_excl_scan256(h, s_scr, &total);
    a.off[pos * kRadixBins + t] = ex;
    if (t == 0) s_active[pos] = used > 1 ? 1u : 0u;
  }
  __syncthreads();
  if (t != 0) return;
  if (a.phase == 1 && p->runs) {
    // the runs are sorted instead (k_runs_plan plans those passes)
    for (int sl = 0; sl < 4; ++sl) p->rs[sl].active = 0;
    p->rec_final = 0;
    p->rec_active = 0;
  } else if (a.phase == 1) {
    // Context digits only: when every context is already in time order in the
    // input, a stable sort on the context alone gives (ctx, ts, input) order.
    uint32_t nact = 0;
    for (int pos = 0; pos < 4; ++pos) nact += s_active[pos];
    uint32_t j = 0;
    for (int sl = 0; sl < 4; ++sl) {
      SlotPlan& sp = p->rs[sl];
      const uint32_t act = s_active[sl] || (nact == 0 && sl == 0);
      sp.active = act;
      sp.pos = (uint32_t)sl;
      if (!act) continue;
      sp.src = j == 0 ? 2u : ((j - 1) & 1u);
      sp.dst = j & 1u;
      sp.lb = j & 1u;
      sp.n_elems = j == 0 ? p->n_records : n_valid;
      sp.n_out = (uint32_t)n_valid;
      sp.tiles = ceil_div(sp.n_elems, kSortTile);
      p->rec_final = sp.dst;
      ++j;
    }
    p->rec_active = j;
  } else {
    // Full sort: every varying timestamp digit, then every varying context
    // digit, continuing the ping-pong from the context-sorted buffer.
    uint32_t j = p->rec_active;
    uint32_t cur = p->rec_final;
    for (int sl = kPhase2Slot; sl < kSlots; ++sl) {
      const uint32_t pos = sl < 12 ? (uint32_t)sl : (uint32_t)(sl - 12);
      SlotPlan& sp = p->rs[sl];
      const uint32_t act = s_active[pos] ? 1u : 0u;
      sp.active = act;
      sp.pos = pos;
      if (!act) continue;
      sp.src = cur;
      sp.dst = cur ^ 1u;
      sp.lb = j & 1u;
      sp.n_elems = n_valid;
      sp.n_out = (uint32_t)n_valid;
      sp.tiles = ceil_div(n_valid, kSortTile);
      cur ^= 1u;
      ++j;
    }
    p->rec_final = cur;
    p->rec_active = j;
  }
}

hipError_t launch_plan(const RunArgs& a, hipStream_t s) {
  PlanArgs pa{a.w.plan, a.out.d_counters, a.w.rec_hist, a.w.rec_off, 1,
              (a.flags & ARGUS_FORCE_RECORD_RADIX) ? 1u : 0u, a.w.run_cap};
  hipLaunchKernelGGL(k_plan, dim3(1), dim3(256), 0, s, pa);
  return hipGetLastError();
}

hipError_t launch_plan2(const RunArgs& a, hipStream_t s) {
  PlanArgs pa{a.w.plan, a.out.d_counters, a.w.rec_hist, a.w.rec_off, 2, 0u, 0ull};
  hipLaunchKernelGGL(k_plan, dim3(1), dim3(256), 0, s, pa);
  return hipGetLastError();
}

// ------------------------------------------------- context sort over runs
//
// When the input holds long runs of one context (trace buffers written per
// warp, interleaved in chunks), a stable sort of the records by context is:
// the runs sorted stably by context (a radix sort over runs, not records),
// each run's first position an exclusive scan of the run lengths in that
// order, and every record written to its run's position plus its rank among
// the run's valid records.  Within a context, runs and the records of a run
// keep input order, so the result equals the record radix sort's.

// Two-level exclusive scan of run counts: which 0 scans the runs of each
// chunk (-> index of each chunk's first run), which 1 the valid records of
// each run in sorted run order (-> each run's first position).
struct RunScanArgs {
  DevPlan* plan;
  uint32_t which;
  const uint32_t* chunk_runs;
  uint32_t* run_base;
  const uint32_t* run_cnt;
  uint32_t* run_pos;
  const uint32_t* pay[2];  // sorted run ids
  uint64_t* bsum;          // [grid]
  // which 1: which runs start their context (for the tile sums; bit 31 of
  // run_pos)
  const uint64_t* key[2];  // sorted run keys (context offset << ts_bits)
  ChunkWaves cw;  // which 0: where each chunk's word is
};

// which 0: the run count of chunk i (from the ingest's chunk table)
__device__ __forceinline__ uint32_t rscan_chunk_runs(const RunScanArgs& a, uint64_t i) {
  return a.chunk_runs[chunk_slot(a.cw, i)] & ((1u << kChunkCountBits) - 1u);
}

__device__ __forceinline__ uint64_t rscan_len(const RunScanArgs& a) {
  return a.which == 0 ? ceil_div(a.plan->n_records, kChunk) : a.plan->n_runs;
}

__global__ __launch_bounds__(256) void k_rscan_part(RunScanArgs a) {
  const DevPlan* p = a.plan;
  if (!p->runs) return;
  __shared__ uint64_t s_w[4];
  const uint64_t m = rscan_len(a);
  const uint64_t per = ceil_div(m, gridDim.x);
  const uint64_t i0 = (uint64_t)blockIdx.x * per, i1 = i0 + per < m ? i0 + per : m;
  const uint32_t* ids = a.pay[p->rec_final];
  uint64_t sum = 0;
  for (uint64_t i = i0 + threadIdx.x; i < i1; i += 256)
    sum += a.which == 0 ? rscan_chunk_runs(a, i) : a.run_cnt[ids[i]];
  sum = wave_sum(sum);
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = sum;
  __syncthreads();
  if (threadIdx.x == 0) a.bsum[blockIdx.x] = s_w[0] + s_w[1] + s_w[2] + s_w[3];
}

// Exclusive scan of the block sums in place (one block).
__global__ __launch_bounds__(1024) void k_rscan_top(RunScanArgs a, uint32_t nblk) {
  if (!a.plan->runs) return;
  __shared__ uint64_t s_w[16];
  const uint32_t t = threadIdx.x, lane = t & 63, w = t >> 6;
  const uint32_t per = (nblk + 1023) / 1024;
  const uint32_t k0 = t * per, k1 = k0 + per < nblk ? k0 + per : nblk;
  uint64_t sum = 0;
  for (uint32_t k = k0; k < k1; ++k) sum += a.bsum[k];
  uint64_t x = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o);
    if ((int)lane >= o) x += y;
  }
  if (lane == 63) s_w[w] = x;
  __syncthreads();
  uint64_t pre = x - sum;
  for (uint32_t q = 0; q < w; ++q) pre += s_w[q];
  for (uint32_t k = k0; k < k1; ++k) {
    const uint64_t v = a.bsum[k];
    a.bsum[k] = pre;
    pre += v;
  }
}

__global__ __launch_bounds__(256) void k_rscan_apply(RunScanArgs a) {
  const DevPlan* p = a.plan;
  if (!p->runs) return;
  __shared__ uint32_t s_w[4];
  const uint64_t m = rscan_len(a);
  const uint64_t per = ceil_div(m, gridDim.x);
  const uint64_t i0 = (uint64_t)blockIdx.x * per, i1 = i0 + per < m ? i0 + per : m;
  const uint32_t* ids = a.pay[p->rec_final];
  const uint32_t t = threadIdx.x, lane = t & 63, w = t >> 6;
  uint64_t carry = a.bsum[blockIdx.x];
  for (uint64_t c0 = i0; c0 < i1; c0 += 1024) {
    uint32_t v[4], sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint64_t i = c0 + 4 * t + q;
      v[q] = i < i1 ? (a.which == 0 ? rscan_chunk_runs(a, i) : a.run_cnt[ids[i]]) : 0u;
      sum += v[q];
    }
    const uint32_t x = (uint32_t)wave_incl_scan32((int32_t)sum);
    if (lane == 63) s_w[w] = x;
    __syncthreads();
    uint64_t pre = carry + x - sum;
    uint64_t all = carry;
    for (uint32_t q = 0; q < 4; ++q) {
      if (q < w) pre += s_w[q];
      all += s_w[q];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint64_t i = c0 + 4 * t + q;
      if (i < i1) {
        if (a.which == 0) {
          a.run_base[i] = (uint32_t)pre;
        } else {
          const uint32_t id = ids[i];
          // A run starts its context if it has valid records and the
          // previous run has another context; runs without valid records
          // sort as context offset 0, so the runs of offset 0 start it only
          // at position 0.
          const uint32_t tb = p->rec.ts_bits;
          const uint64_t* keys = a.key[p->rec_final];
          const uint32_t ctx = tb >= 64 ? 0u : (uint32_t)(keys[i] >> tb);
          const uint32_t prev = i > 0 ? (tb >= 64 ? 0u : (uint32_t)(keys[i - 1] >> tb)) : 0xFFFFFFFFu;
          const uint32_t head = v[q] > 0 && (ctx == 0 ? pre == 0 : prev != ctx) ? 1u : 0u;
          a.run_pos[id] = (uint32_t)pre | (head << 31);
        }
      }
      pre += v[q];
    }
    carry = all;
    __syncthreads();
  }
}

static uint32_t rscan_blocks(uint64_t cap) {
  uint64_t b = ceil_div(cap ? cap : 1, 4096);
  if (b > kMaxScanBlocks) b = kMaxScanBlocks;
  return b < 1 ? 1u : (uint32_t)b;
}

static hipError_t launch_rscan(const RunArgs& a, uint32_t which, uint64_t cap, hipStream_t s) {
  RunScanArgs r{};
  r.plan = a.w.plan;
  r.which = which;
  r.chunk_runs = a.w.chunk_runs;
  r.run_base = a.w.run_base;
  r.run_cnt = a.w.run_cnt;
  r.run_pos = a.w.run_pos;
  for (int b = 0; b < 2; ++b) {
    r.pay[b] = a.w.pay[b];
    r.key[b] = a.w.key[b];
  }
  r.bsum = a.w.scan_bsum;
  r.cw = chunk_waves(a.w.chunks, ingest_blocks(a.n) * 4);
  const uint32_t nblk = rscan_blocks(cap);
  hipLaunchKernelGGL(k_rscan_part, dim3(nblk), dim3(256), 0, s, r);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rscan_top, dim3(1), dim3(1024), 0, s, r, nblk);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rscan_apply, dim3(nblk), dim3(256), 0, s, r);
  return hipGetLastError();
}

hipError_t launch_runs_base(const RunArgs& a, hipStream_t s) { return launch_rscan(a, 0, a.w.chunks, s); }
hipError_t launch_runs_pos(const RunArgs& a, hipStream_t s) { return launch_rscan(a, 1, a.w.run_cap, s); }

struct RunCompactArgs {
  DevPlan* plan;
  const uint64_t* runs_raw;
  const uint32_t* chunk_runs;
  const uint32_t* run_base;
  uint64_t* key;      // key[0]: context offset << ts_bits
  uint32_t* pay;      // pay[0]: run id
  uint32_t* run_cnt;
  uint32_t* run_hist; // [4][256]
  ChunkWaves cw;      // where each chunk's run list is
};

// The runs of every chunk, in input order, as sort elements (key: context
// offset, payload: run id), their lengths, and the context-digit histograms
// over runs.  A run without valid records sorts as the lowest context.
__global__ __launch_bounds__(256) void k_runs_compact(RunCompactArgs a) {
  DevPlan* p = a.plan;
  if (!p->runs) return;
  __shared__ uint32_t s_hist[4][kRadixBins];
  for (int i = threadIdx.x; i < 4 * kRadixBins; i += 256) (&s_hist[0][0])[i] = 0;
  __syncthreads();
  const KeySpace ks = p->rec;
  const uint64_t chunks = ceil_div(p->n_records, kChunk);
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  for (uint64_t c = (uint64_t)blockIdx.x * 256 + threadIdx.x; c < chunks; c += stride) {
    const uint32_t cword = a.chunk_runs[chunk_slot(a.cw, c)];
    const uint32_t nr = cword & ((1u << kChunkCountBits) - 1u);
    const uint64_t* list = a.runs_raw + wave_slot0(a.cw, c % a.cw.W) * kChunk + (cword >> kChunkCountBits);
    const uint32_t rb = a.run_base[c];
    for (uint32_t j = 0; j < nr && j < (uint32_t)kChunk; ++j) {
      const uint64_t v = list[j];
      const uint32_t cnt = (uint32_t)(v >> 32);
      const uint64_t rel = cnt ? (uint64_t)((uint32_t)v - (uint32_t)ks.ctx_min) : 0ull;
      const uint32_t rid = rb + j;
      a.key[rid] = ks.ts_bits >= 64 ? 0ull : (rel << ks.ts_bits);
      a.pay[rid] = rid;
      a.run_cnt[rid] = cnt;
      const uint32_t ctx = (uint32_t)(ks.ctx_min + rel);
#pragma unroll
      for (int d = 0; d < 4; ++d) atomicAdd(&s_hist[d][(ctx >> (8 * d)) & 0xFFu], 1u);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 4 * kRadixBins; i += 256) {
    const uint32_t h = (&s_hist[0][0])[i];
    if (h) atomicAdd(&a.run_hist[i], h);
  }
}

hipError_t launch_runs_compact(const RunArgs& a, hipStream_t s) {
  RunCompactArgs r{a.w.plan, a.w.key[1], a.w.chunk_runs, a.w.run_base, a.w.key[0], a.w.pay[0],
                   a.w.run_cnt, a.w.run_hist, chunk_waves(a.w.chunks, ingest_blocks(a.n) * 4)};
  uint64_t blocks = ceil_div(a.w.chunks ? a.w.chunks : 1, 256);
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(k_runs_compact, dim3((uint32_t)blocks), dim3(256), 0, s, r);
  return hipGetLastError();
}

// Plans the context passes over the runs (packed elements in buffer 0).
__global__ __launch_bounds__(256) void k_runs_plan(DevPlan* p, const uint32_t* hist, uint32_t* off) {
  __shared__ uint32_t s_scr[4];
  __shared__ uint32_t s_active[4];
  if (!p->runs) return;
  const int t = threadIdx.x;
  for (int pos = 0; pos < 4; ++pos) {
    const uint32_t h = hist[pos * kRadixBins + t];
    const int used = __syncthreads_count(h != 0);
    uint32_t total;
    off[pos * kRadixBins + t] = block_excl_scan256(h, s_scr, &total);
    if (t == 0) s_active[pos] = used > 1 ? 1u : 0u;
  }
  __syncthreads();
  if (t != 0) return;
  const uint64_t n_runs = p->n_runs;
  uint32_t j = 0;
  for (int sl = 0; sl < 4; ++sl) {
    SlotPlan& sp = p->rs[sl];
    sp.active = s_active[sl];
    sp.pos = (uint32_t)sl;
    if (!sp.active) continue;
    sp.src = j & 1u;
    sp.dst = (j & 1u) ^ 1u;
    sp.lb = j & 1u;
    sp.n_elems = n_runs;
    sp.n_out = (uint32_t)n_runs;
    sp.tiles = ceil_div(n_runs, kSortTile);
    ++j;
  }
  p->rec_final = j & 1u;
  p->rec_active = j;
}

hipError_t launch_runs_plan(const RunArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_runs_plan, dim3(1), dim3(256), 0, s, a.w.plan, a.w.run_hist, a.w.rec_off);
  return hipGetLastError();
}

struct RunScatterArgs {
  DevPlan* plan;
  const uint4* rec;
  uint64_t n;
  uint32_t R;
  const uint32_t* run_base;
  const uint32_t* run_pos;
  uint64_t* key;  // key[0]
  uint32_t* pay;  // pay[0]
  uint64_t* counters;
  const uint8_t* region_class;
  uint32_t K, G, shift;
  // for the tile sums: which runs start their context
  const uint32_t* run_cnt;
};

// Every valid record to its run's position plus its rank among the run's
// valid records, packed as in the radix path (key (ctx - ctx_min) << ts_bits
// | (ts - ts_min), payload region | (kind - 1) << 16 | class << 24).  One
// wave per chunk, as in the ingest.  For the tile sums it also marks the
// first record of each context in its payload (kPayStart) and checks that
// the valid records of a context in the chunk are in time order
// (k_runs_check checks where runs meet).
__global__ __launch_bounds__(256) void k_runs_scatter(RunScatterArgs a) {
  DevPlan* p = a.plan;
  if (!p->runs) return;
  __shared__ uint8_t s_cls[kClsLds];
  // per wave and run of the chunk: first position minus its head's rank,
  // first position, valid records | starts its context << 31
  __shared__ uint32_t s_roff[4][kChunk], s_rpos[4][kChunk], s_rcnt[4][kChunk];
  // per wave and chunk position: timestamp and context
  __shared__ uint64_t s_ts[4][kChunk];
  __shared__ uint32_t s_cx[4][kChunk];
  const uint32_t wv = threadIdx.x >> 6;
  bool bad = false;
  const bool cls_lds = a.K && a.R <= kClsLds;
  if (cls_lds)
    for (uint32_t r = threadIdx.x; r < a.R; r += 256) s_cls[r] = a.region_class[r];
  __syncthreads();
  const KeySpace ks = p->rec;
  const uint64_t nv = p->n_valid;
  constexpr int kPer = 4;
  const uint64_t stride = (uint64_t)gridDim.x * 256 * kPer;
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t first = ((uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * (64 * kPer);
  // the next chunk's records and run base are loaded while this one is written
  uint4 nr_[kPer];
  uint32_t nrb = 0;
  auto issue = [&](uint64_t b) {
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint64_t i = b + (uint64_t)j * 64 + lane;
      nr_[j] = a.rec[i < a.n ? i : a.n - 1];
    }
    nrb = a.run_base[b / kChunk];
  };
  if (first < a.n) issue(first);
  for (uint64_t base = first; base < a.n; base += stride) {
    uint4 r[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) r[j] = nr_[j];
    const uint32_t rb = nrb;
    if (base + stride < a.n) issue(base + stride);
    uint32_t cx[kPer];
    bool inr[kPer], vl[kPer];
    const uint32_t rem = a.n - base < (uint64_t)kChunk ? (uint32_t)(a.n - base) : (uint32_t)kChunk;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint32_t kind = (r[j].w >> 16) & 0xFFu;
      cx[j] = r[j].z;
      inr[j] = 64u * j + lane < rem;
      vl[j] = inr[j] && (kind == 1 || kind == 2) && (r[j].w & 0xFFFFu) < a.R;
    }
    // the positions, context-start flags and sizes of the chunk's first 64
    // runs, one per lane, in flight while the masks are built
    const uint64_t n_runs = p->n_runs;
    const uint32_t prid = rb + lane;
    const bool pin = prid < n_runs;
    const uint32_t pre_word = pin ? a.run_pos[prid] : 0u;
    const uint32_t pre_pos = pre_word & kRunPosMask, pre_head = pre_word >> 31;
    const uint32_t pre_cnt = pin ? a.run_cnt[prid] : 0u;
    uint64_t H[4], V[4];
    chunk_masks(cx, inr, vl, H, V);
    // Run of each record (heads before it, inclusive) and its rank among the
    // chunk's valid records; each run head publishes its run's first
    // position minus its own rank in the wave's LDS slots.  A chunk whose
    // in-range records are all valid (the usual case) needs no more LDS:
    // its order check and run bounds come from neighbouring lanes.
    uint64_t IR[kPer];
    bool all_valid = true;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      IR[j] = __ballot(inr[j]);
      all_valid = all_valid && V[j] == IR[j];
    }
    uint32_t li[kPer], vr[kPer], hflag[kPer];
    int32_t lastv[kPer];  // last valid chunk position in earlier rows (-1: none)
    uint32_t hb = 0, vb = 0;
    int32_t lv = -1;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint32_t hr = hb + (uint32_t)__builtin_amdgcn_mbcnt_hi(
                                   (uint32_t)(H[j] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)H[j], 0u));
      vr[j] = vb + (uint32_t)__builtin_amdgcn_mbcnt_hi(
                       (uint32_t)(V[j] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)V[j], 0u));
      const bool head = (H[j] >> lane) & 1ull;
      const uint32_t sp = (uint32_t)__shfl((int)pre_pos, (int)(hr & 63u));
      const uint32_t sh = (uint32_t)__shfl((int)pre_head, (int)(hr & 63u));
      const uint32_t sc = (uint32_t)__shfl((int)pre_cnt, (int)(hr & 63u));
      hflag[j] = 0;
      if (head) {
        const uint32_t rid = rb + hr;
        const bool near = hr < 64u;
        const uint32_t far_word = near ? 0u : a.run_pos[rid];
        const uint32_t rp = near ? sp : (far_word & kRunPosMask);
        s_roff[wv][hr] = rp - vr[j];
        hflag[j] = near ? sh : far_word >> 31;
        if (!all_valid) {
          s_rpos[wv][hr] = rp;
          s_rcnt[wv][hr] = (near ? sc : a.run_cnt[rid]) | (hflag[j] << 31);
        }
      }
      li[j] = hr + (head ? 1u : 0u) - 1u;
      if (!all_valid) {
        s_ts[wv][64 * j + lane] = (uint64_t)r[j].x | ((uint64_t)r[j].y << 32);
        s_cx[wv][64 * j + lane] = cx[j];
        lastv[j] = lv;
        if (V[j]) lv = 64 * j + 63 - (int32_t)__clzll((long long)V[j]);
      }
      hb += (uint32_t)__popcll(H[j]);
      vb += (uint32_t)__popcll(V[j]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint64_t ts = (uint64_t)r[j].x | ((uint64_t)r[j].y << 32);
      bool first_v = false, starts = false;
      if (all_valid) {
        // previous record: the previous lane, or the last lane of the row before
        // (lane 0 of the first row starts a run: its value is not used)
        const int jp = j > 0 ? j - 1 : 0;
        const uint32_t fx = (uint32_t)__builtin_amdgcn_readlane((int)r[jp].x, 63);
        const uint32_t fy = (uint32_t)__builtin_amdgcn_readlane((int)r[jp].y, 63);
        const uint64_t tp = ((uint64_t)lane_prev(r[j].y, fy) << 32) | lane_prev(r[j].x, fx);
        const bool h = (H[j] >> lane) & 1ull;
        if (vl[j] && !h && tp > ts) bad = true;
        first_v = h;
        starts = h && hflag[j];
      }
      if (!vl[j]) continue;
      const uint32_t run = li[j];
      const uint64_t out = (uint64_t)(uint32_t)(s_roff[wv][run] + vr[j]);
      if (out >= nv) {
        flag_internal_error(a.counters, 1024);
        continue;
      }
      if (!all_valid) {
        // the previous valid record of the chunk, if it has the same context
        const uint64_t below = V[j] & ((1ull << lane) - 1ull);
        const int32_t pv = below ? 64 * j + 63 - (int32_t)__clzll((long long)below) : lastv[j];
        if (pv >= 0 && s_cx[wv][pv] == cx[j] && s_ts[wv][pv] > ts) bad = true;
        const uint32_t rpos = s_rpos[wv][run], rc = s_rcnt[wv][run];
        first_v = (uint32_t)out == rpos;
        starts = first_v && (rc >> 31);
      }
      const uint64_t rel = (uint64_t)(cx[j] - (uint32_t)ks.ctx_min);
      a.key[out] = (ks.ts_bits >= 64 ? 0ull : (rel << ks.ts_bits)) | (ts - ks.ts_min);
      const uint32_t region = r[j].w & 0xFFFFu;
      uint32_t cls = 0xFFu;
      if (swept_ctx(cx[j], a.K, a.G, a.shift)) cls = cls_lds ? s_cls[region] : a.region_class[region];
      a.pay[out] = pack_payload(region, (r[j].w >> 16) & 0xFFu, cls) | (starts ? kPayStart : 0u);
    }
  }
  if (__syncthreads_or(bad) && threadIdx.x == 0) p->unsorted = 1;
  if (blockIdx.x == 0 && threadIdx.x == 0) p->rec_final = 0;
}

hipError_t launch_runs_scatter(const RunArgs& a, hipStream_t s) {
  RunScatterArgs r{a.w.plan, (const uint4*)a.rec, a.n, a.R, a.w.run_base, a.w.run_pos,
                   a.w.key[0], a.w.pay[0], a.out.d_counters, a.region_class, a.K, a.G, a.shift,
                   a.w.run_cnt};
  // 1280 blocks, five per compute unit (as many as the LDS holds), measured
  // fastest: more loads in flight than with 1024 or fewer
  uint64_t blocks = ceil_div(a.n, 256 * 4 * 4);
  if (blocks > 1280) blocks = 1280;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_runs_scatter, dim3((uint32_t)blocks), dim3(256), 0, s, r);
  return hipGetLastError();
}

// After the run path the full sort (if needed) starts on a look-back status
// array that only the shorter run passes have cleared: clear it whole.
__global__ __launch_bounds__(256) void k_lb_clear(DevPlan* p, uint64_t* lb0, uint64_t* lb1) {
  if (!p->runs || !p->unsorted) return;
  uint64_t* lb = (p->rec_active & 1u) ? lb1 : lb0;
  const uint64_t words = ceil_div(p->n_valid, kSortTile) * kRadixBins;
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < words; i += stride) lb[i] = 0;
}

hipError_t launch_lb_clear(const RunArgs& a, hipStream_t s) {
  uint64_t blocks = ceil_div(ceil_div(a.n ? a.n : 1, kSortTile) * kRadixBins, 256 * 8);
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_lb_clear, dim3((uint32_t)blocks), dim3(256), 0, s, a.w.plan, a.w.lb[0], a.w.lb[1]);
  return hipGetLastError();
}

// ----------------------------------------------------------- sortedness

// Grid of k_tsum (and of the tile scan, which follows its runs of tiles).
static uint32_t tsum_blocks(const RunArgs& a);

struct TsumArgs {
  DevPlan* plan;
  const uint64_t* key[2];
  const uint32_t* pay[2];
  const uint32_t* ctxw[2];
  uint64_t* tsum;     // [match tiles]
  BlockSum* bsum;     // [grid]: each block's run of tiles composed
  uint32_t mode;      // 0: after the context passes (check the order too); 1: after the full sort
};

// Per matching tile (2048 consecutive sorted records): the map from the depth
// before the tile to the depth after it, its BEGINs and its context starts
// (k_mscan turns these into each tile's entering values, so that k_match
// needs no look-back).  In mode 0 it also checks that the context-only sort
// left (ctx, ts) non-decreasing; if not (some context was out of time order
// in the input) the full sort runs and mode 1 redoes the sums.  Block b takes
// the b-th contiguous run of tiles and also stores the run composed.
__global__ __launch_bounds__(256) void k_tsum(TsumArgs a) {
  DevPlan* p = a.plan;
  if (a.mode == 0 && p->runs) return;  // k_runs_check and k_tsum_codes instead
  if (a.mode == 0 && p->force_full) {
    if (blockIdx.x == 0 && threadIdx.x == 0) p->unsorted = 1;
    return;
  }
  if (a.mode == 1 && !p->unsorted) return;
  __shared__ Fn s_wfn[4];
  __shared__ uint32_t s_wnb[4];
  const uint64_t nv = p->n_valid;
  const uint64_t tiles = ceil_div(nv, kMatchTile);
  const uint32_t b = p->rec_final;
  const uint64_t* key = a.key[b];
  const uint32_t* pay = a.pay[b];
  const uint32_t* cw = a.ctxw[b];
  const KeySpace ks = p->rec;
  const bool wide = ks.wide != 0;
  const uint32_t tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t p0 = tid * kMatchItems;
  auto ctx_of = [&](uint64_t i, uint64_t k) -> uint32_t {
    return wide ? cw[i] : (ks.ts_bits >= 64 ? 0u : (uint32_t)(k >> ks.ts_bits));
  };
  bool bad = false;
  const uint64_t per = ceil_div(tiles, gridDim.x);
  const uint64_t t0 = (uint64_t)blockIdx.x * per, t1 = t0 + per < tiles ? t0 + per : tiles;
  Fn run = fn_id();
  uint32_t run_nb = 0, run_nh = 0;
  for (uint64_t tile = t0; tile < t1; ++tile) {
    const uint64_t base = tile * kMatchTile;
    const uint32_t cnt = nv - base < (uint64_t)kMatchTile ? (uint32_t)(nv - base) : (uint32_t)kMatchTile;
    uint64_t k[kMatchItems];
    uint32_t c[kMatchItems], kind = 0, fv = 0;
    if (p0 + kMatchItems <= cnt) {
      const uint4* k4 = (const uint4*)(key + base + p0);
#pragma unroll
      for (int q = 0; q < kMatchItems / 2; ++q) {
        const uint4 v = k4[q];
        k[2 * q] = (uint64_t)v.x | ((uint64_t)v.y << 32);
        k[2 * q + 1] = (uint64_t)v.z | ((uint64_t)v.w << 32);
      }
      const uint4* p4 = (const uint4*)(pay + base + p0);
#pragma unroll
      for (int q = 0; q < kMatchItems / 4; ++q) {
        const uint4 v = p4[q];
        kind |= ((v.x >> 16) & 1u) << (4 * q) | ((v.y >> 16) & 1u) << (4 * q + 1) |
                ((v.z >> 16) & 1u) << (4 * q + 2) | ((v.w >> 16) & 1u) << (4 * q + 3);
      }
      fv = 0xFFu;
    } else {
#pragma unroll
      for (int i = 0; i < kMatchItems; ++i) {
        const uint32_t q = p0 + i;
        k[i] = q < cnt ? key[base + q] : 0ull;
        if (q < cnt) {
          kind |= ((pay[base + q] >> 16) & 1u) << i;
          fv |= 1u << i;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kMatchItems; ++i) c[i] = ctx_of(base + p0 + i < nv ? base + p0 + i : 0, k[i]);
    // the record before this thread's first one
    uint32_t c_prev = (uint32_t)__shfl_up((int)c[kMatchItems - 1], 1);
    uint64_t k_prev = __shfl_up(k[kMatchItems - 1], 1);
    bool has_prev = true;
    if (lane == 0) {
      const uint64_t pp = base + p0;
      has_prev = pp > 0 && pp <= nv;
      if (has_prev) {
        k_prev = key[pp - 1];
        c_prev = ctx_of(pp - 1, k_prev);
      }
    }
    Fn f = fn_id();
    uint32_t nb = 0, nh = 0;
#pragma unroll
    for (int i = 0; i < kMatchItems; ++i) {
      if (!((fv >> i) & 1u)) continue;
      const bool hp = i > 0 || has_prev;
      const uint32_t cp = i > 0 ? c[i - 1] : c_prev;
      const uint64_t kp = i > 0 ? k[i - 1] : k_prev;
      const bool head = !hp || cp != c[i];
      if (a.mode == 0 && hp) bad |= wide ? (cp > c[i] || (cp == c[i] && kp > k[i])) : kp > k[i];
      const bool isb = ((kind >> i) & 1u) == 0;
      const Fn e = head ? Fn{1u, 0, isb ? 1 : 0} : Fn{0u, isb ? 1 : -1, 0};
      f = compose(f, e);
      nb += isb;
      nh += head;
    }
    // tile sums: wave scans, then the four waves in order
    const Fn x = wave_scan_fn(f);
    const uint32_t nbx = (uint32_t)wave_incl_scan32((int32_t)(nb | (nh << 16)));
    if (lane == 63) {
      s_wfn[w] = x;
      s_wnb[w] = nbx;
    }
    __syncthreads();
    if (tid == 0) {
      Fn all = fn_id();
      uint32_t nball = 0;
      for (int q = 0; q < 4; ++q) {
        all = compose(all, s_wfn[q]);
        nball += s_wnb[q];
      }
      a.tsum[tile] = pack_tile_sum(all, nball);
      run = compose(run, all);
      run_nb += nball & 0xFFFFu;
      run_nh += nball >> 16;
    }
    __syncthreads();
  }
  if (tid == 0) a.bsum[blockIdx.x] = BlockSum{run, run_nb, run_nh};
  if (a.mode == 0 && __syncthreads_or(bad) && threadIdx.x == 0) p->unsorted = 1;
}

static uint32_t tsum_blocks(const RunArgs& a) {
  uint64_t blocks = a.w.match_tiles;
  if (blocks > kMaxScanBlocks) blocks = kMaxScanBlocks;
  return blocks < 1 ? 1u : (uint32_t)blocks;
}

hipError_t launch_tsum(const RunArgs& a, int mode, hipStream_t s) {
  TsumArgs ta{};
  ta.plan = a.w.plan;
  for (int b = 0; b < 2; ++b) {
    ta.key[b] = a.w.key[b];
    ta.pay[b] = a.w.pay[b];
    ta.ctxw[b] = a.w.ctxw[b];
  }
  ta.tsum = a.w.tsum;
  ta.bsum = a.w.bsum;
  ta.mode = (uint32_t)mode;
  hipLaunchKernelGGL(k_tsum, dim3(tsum_blocks(a)), dim3(256), 0, s, ta);
  return hipGetLastError();
}

// ------------------------------------------- tile sums after the run scatter

struct RunCheckArgs {
  DevPlan* plan;
  const uint32_t* run_cnt;
  const uint32_t* run_pos;
  const uint64_t* key;  // sorted keys (key[0])
};

// The order check where runs meet: the first record of each run against
// the record before it in sorted order, when both belong to one context.
// (Inside a chunk the run scatter checks.)
__global__ __launch_bounds__(256) void k_runs_check(RunCheckArgs a) {
  DevPlan* p = a.plan;
  if (!p->runs) return;
  if (p->force_full) {
    if (blockIdx.x == 0 && threadIdx.x == 0) p->unsorted = 1;
    return;
  }
  const uint64_t n_runs = p->n_runs;
  const uint32_t tb = p->rec.ts_bits;
  bool bad = false;
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  for (uint64_t r = (uint64_t)blockIdx.x * 256 + threadIdx.x; r < n_runs; r += stride) {
    const uint32_t pos = a.run_pos[r] & kRunPosMask;
    if (a.run_cnt[r] == 0 || pos == 0) continue;
    const uint64_t k0 = a.key[pos - 1], k1 = a.key[pos];
    // same context (key bits above ts_bits) and time going back
    if ((tb >= 64 || (k0 >> tb) == (k1 >> tb)) && k0 > k1) bad = true;
  }
  if (__syncthreads_or(bad) && threadIdx.x == 0) p->unsorted = 1;
}

hipError_t launch_runs_check(const RunArgs& a, hipStream_t s) {
  RunCheckArgs r{a.w.plan, a.w.run_cnt, a.w.run_pos, a.w.key[0]};
  uint64_t blocks = ceil_div(a.w.run_cap, 256);
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_runs_check, dim3((uint32_t)blocks), dim3(256), 0, s, r);
  return hipGetLastError();
}

struct TsumCodeArgs {
  const DevPlan* plan;
  const uint32_t* pay;  // payloads of the sorted records (pay[0])
  uint64_t* tsum;
  BlockSum* bsum;
};

// The tile sums of k_tsum (same tiles per block, same outputs) from the
// payloads the run scatter wrote (kind and context-start bits), without the
// keys.  One wave per tile, the block's four waves on four consecutive
// tiles: the wave loads the tile's payloads contiguously, keeps two bits
// per record in LDS, and each lane then composes 32 consecutive records.
__global__ __launch_bounds__(256, 8) void k_tsum_codes(TsumCodeArgs a) {
  const DevPlan* p = a.plan;
  if (!p->runs) return;
  __shared__ Fn s_wfn[4];
  __shared__ uint32_t s_wnb[4];
  __shared__ __align__(8) uint8_t s_code[4][kMatchTile / 4];  // per wave: 4 records per byte
  constexpr uint32_t kPerLane = kMatchTile / 64;  // 32
  const uint64_t nv = p->n_valid;
  const uint64_t tiles = ceil_div(nv, kMatchTile);
  const uint32_t tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t p0 = lane * kPerLane;
  const uint64_t per = ceil_div(tiles, gridDim.x);
  const uint64_t t0 = (uint64_t)blockIdx.x * per, t1 = t0 + per < tiles ? t0 + per : tiles;
  Fn run = fn_id();
  uint32_t run_nb = 0, run_nh = 0;
  auto code_of = [](uint32_t v) -> uint32_t {
    return (((v >> 16) & 1u) ^ 1u) | ((v & kPayStart) ? 2u : 0u);  // BEGIN | start << 1
  };
  for (uint64_t tq = t0; tq < t1; tq += 4) {
    const uint64_t tile = tq + w;
    Fn f = fn_id();
    uint32_t nb = 0, nh = 0;
    if (tile < t1) {
      const uint64_t base = tile * kMatchTile;
      const uint32_t cnt = nv - base < (uint64_t)kMatchTile ? (uint32_t)(nv - base) : (uint32_t)kMatchTile;
      // a full tile (all but the last) loads its payloads in one batch; a
      // choice per load would make each wait for the one before
      uint4 u[kPerLane / 4];
      if (cnt == kMatchTile) {
#pragma unroll
        for (int q = 0; q < (int)kPerLane / 4; ++q)
          u[q] = *(const uint4*)(a.pay + base + (uint32_t)q * 256u + 4u * lane);
      } else {
#pragma unroll
        for (int q = 0; q < (int)kPerLane / 4; ++q) {
          const uint32_t r0 = (uint32_t)q * 256u + 4u * lane;
          u[q].x = r0 < cnt ? a.pay[base + r0] : 0u;
          u[q].y = r0 + 1 < cnt ? a.pay[base + r0 + 1] : 0u;
          u[q].z = r0 + 2 < cnt ? a.pay[base + r0 + 2] : 0u;
          u[q].w = r0 + 3 < cnt ? a.pay[base + r0 + 3] : 0u;
        }
      }
#pragma unroll
      for (int q = 0; q < (int)kPerLane / 4; ++q) {
        const uint32_t r0 = (uint32_t)q * 256u + 4u * lane;
        s_code[w][r0 >> 2] = (uint8_t)(code_of(u[q].x) | code_of(u[q].y) << 2 |
                                       code_of(u[q].z) << 4 | code_of(u[q].w) << 6);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const uint64_t c = *(const uint64_t*)&s_code[w][p0 >> 2];
#pragma unroll
      for (int i = 0; i < (int)kPerLane; ++i) {
        if (p0 + (uint32_t)i >= cnt) break;
        const uint32_t ci = (uint32_t)(c >> (2 * i)) & 3u;
        const bool isb = ci & 1u, head = (ci >> 1) & 1u;
        const Fn e = head ? Fn{1u, 0, isb ? 1 : 0} : Fn{0u, isb ? 1 : -1, 0};
        f = compose(f, e);
        nb += isb;
        nh += head;
      }
    }
    const Fn x = wave_scan_fn(f);
    const uint32_t nbx = (uint32_t)wave_incl_scan32((int32_t)(nb | (nh << 16)));
    if (lane == 63) {
      if (tile < t1) a.tsum[tile] = pack_tile_sum(x, nbx);
      s_wfn[w] = x;
      s_wnb[w] = nbx;
    }
    __syncthreads();
    if (tid == 0) {
      for (int q = 0; q < 4; ++q) {
        run = compose(run, s_wfn[q]);  // identity for tiles past the run
        run_nb += s_wnb[q] & 0xFFFFu;
        run_nh += s_wnb[q] >> 16;
      }
    }
    __syncthreads();
  }
  if (tid == 0) a.bsum[blockIdx.x] = BlockSum{run, run_nb, run_nh};
}

hipError_t launch_tsum_codes(const RunArgs& a, hipStream_t s) {
  TsumCodeArgs t{a.w.plan, a.w.pay[0], a.w.tsum, a.w.bsum};
  hipLaunchKernelGGL(k_tsum_codes, dim3(tsum_blocks(a)), dim3(256), 0, s, t);
  return hipGetLastError();
}

struct MscanArgs {
  const DevPlan* plan;
  const uint64_t* tsum;
  BlockSum* bsum;  // in: each k_tsum block's run; out (k_mscan_top): what comes before it
  TileCarry* carry;
  uint32_t nblk;   // k_tsum blocks
};

// Exclusive scan of the k_tsum block sums (one block; each thread composes
// a contiguous run of them).  Overwrites each block sum with the composition
// of everything before that block.
__global__ __launch_bounds__(1024) void k_mscan_top(MscanArgs a) {
  __shared__ Fn s_wfn[16];
  __shared__ uint32_t s_wnb[16], s_wnh[16];
  const uint32_t t = threadIdx.x, lane = t & 63, w = t >> 6;
  const uint32_t per = (a.nblk + 1023) / 1024;
  const uint32_t k0 = t * per, k1 = k0 + per < a.nblk ? k0 + per : a.nblk;
  Fn f = fn_id();
  uint32_t nb = 0, nh = 0;
  for (uint32_t k = k0; k < k1; ++k) {
    const BlockSum b = a.bsum[k];
    f = compose(f, b.f);
    nb += b.nb;
    nh += b.nh;
  }
  const Fn x = wave_scan_fn(f);
  const uint32_t xb = (uint32_t)wave_incl_scan32((int32_t)nb);
  const uint32_t xh = (uint32_t)wave_incl_scan32((int32_t)nh);
  if (lane == 63) {
    s_wfn[w] = x;
    s_wnb[w] = xb;
    s_wnh[w] = xh;
  }
  Fn ex = Fn{(uint32_t)__shfl_up((int)x.reset, 1), __shfl_up(x.a, 1), __shfl_up(x.c, 1)};
  if (lane == 0) ex = fn_id();
  __syncthreads();
  Fn pre = fn_id();
  uint32_t pb = xb - nb, ph = xh - nh;
  for (uint32_t q = 0; q < w; ++q) {
    pre = compose(pre, s_wfn[q]);
    pb += s_wnb[q];
    ph += s_wnh[q];
  }
  f = compose(pre, ex);
  for (uint32_t k = k0; k < k1; ++k) {
    const BlockSum b = a.bsum[k];
    a.bsum[k] = BlockSum{f, pb, ph};
    f = compose(f, b.f);
    pb += b.nb;
    ph += b.nh;
  }
}

// Entering values of every matching tile: block b of k_tsum's grid scans its
// run of tile sums (256 at a time) after what comes before the run.
__global__ __launch_bounds__(256) void k_mscan_tiles(MscanArgs a) {
  __shared__ Fn s_wfn[4];
  __shared__ uint32_t s_wnb[4], s_wnh[4];
  const uint64_t tiles = a.plan->match_tiles;
  const uint64_t per = ceil_div(tiles, gridDim.x);
  const uint64_t t0 = (uint64_t)blockIdx.x * per, t1 = t0 + per < tiles ? t0 + per : tiles;
  const uint32_t t = threadIdx.x, lane = t & 63, w = t >> 6;
  const BlockSum b0 = a.bsum[blockIdx.x];
  Fn run = b0.f;
  uint64_t run_nb = b0.nb, run_nh = b0.nh;
  for (uint64_t c0 = t0; c0 < t1; c0 += 256) {
    const uint64_t k = c0 + t;
    Fn g = fn_id();
    uint32_t nbh = 0;
    if (k < t1) unpack_tile_sum(a.tsum[k], &g, &nbh);
    const uint32_t nb = nbh & 0xFFFFu, nh = nbh >> 16;
    const Fn x = wave_scan_fn(g);
    const uint32_t xb = (uint32_t)wave_incl_scan32((int32_t)nb);
    const uint32_t xh = (uint32_t)wave_incl_scan32((int32_t)nh);
    if (lane == 63) {
      s_wfn[w] = x;
      s_wnb[w] = xb;
      s_wnh[w] = xh;
    }
    Fn ex = Fn{(uint32_t)__shfl_up((int)x.reset, 1), __shfl_up(x.a, 1), __shfl_up(x.c, 1)};
    if (lane == 0) ex = fn_id();
    __syncthreads();
    Fn pre = run, all = run;
    uint64_t pb = run_nb, ph = run_nh, ab = run_nb, ah = run_nh;
    for (uint32_t q = 0; q < 4; ++q) {
      if (q < w) {
        pre = compose(pre, s_wfn[q]);
        pb += s_wnb[q];
        ph += s_wnh[q];
      }
      all = compose(all, s_wfn[q]);
      ab += s_wnb[q];
      ah += s_wnh[q];
    }
    pre = compose(pre, ex);
    pb += xb - nb;
    ph += xh - nh;
    if (k < t1) {
      TileCarry c;
      c.s_in = (uint32_t)apply(pre, 0);
      c.hpre = (uint32_t)ph;
      c.nbpre = pb;
      a.carry[k] = c;
    }
    run = all;
    run_nb = ab;
    run_nh = ah;
    __syncthreads();
  }
}

hipError_t launch_mscan(const RunArgs& a, hipStream_t s) {
  MscanArgs m{a.w.plan, a.w.tsum, a.w.bsum, a.w.carry, tsum_blocks(a)};
  hipLaunchKernelGGL(k_mscan_top, dim3(1), dim3(1024), 0, s, m);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_mscan_tiles, dim3(m.nblk), dim3(256), 0, s, m);
  return hipGetLastError();
}

// -------------------------------------------------- timestamp histograms

struct TsHistArgs {
  DevPlan* plan;
  const uint64_t* key[2];
  uint32_t* hist;  // rec_hist positions 4..11
};

// Only when the full sort is needed: histograms of the eight raw timestamp
// digits of the (packed) records.
__global__ __launch_bounds__(256) void k_ts_hist(TsHistArgs a) {
  const DevPlan* p = a.plan;
  if (!p->unsorted) return;
  __shared__ uint32_t s_hist[8][kRadixBins];
  for (int i = threadIdx.x; i < 8 * kRadixBins; i += 256) (&s_hist[0][0])[i] = 0;
  __syncthreads();
  const uint64_t n = p->n_valid;
  const KeySpace ks = p->rec;
  const uint64_t* key = a.key[p->rec_final];
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  const uint64_t first = (uint64_t)blockIdx.x * 256 + (threadIdx.x & ~63u);
  for (uint64_t base = first; base < n; base += stride) {
    const uint64_t i = base + (threadIdx.x & 63);
    const bool valid = i < n;
    uint64_t ts = 0;
    if (valid) {
      const uint64_t k = key[i];
      ts = ks.ts_min + (ks.wide ? k : (k & ks.ts_mask));
    }
#pragma unroll
    for (int d = 0; d < 8; ++d) wave_hist_add(s_hist[d], (uint32_t)(ts >> (8 * d)) & 0xFFu, valid);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 8 * kRadixBins; i += 256) {
    const uint32_t h = (&s_hist[0][0])[i];
    if (h) atomicAdd(&a.hist[4 * kRadixBins + i], h);
  }
}

hipError_t launch_ts_hist(const RunArgs& a, hipStream_t s) {
  TsHistArgs ta{a.w.plan, {a.w.key[0], a.w.key[1]}, a.w.rec_hist};
  uint64_t blocks = ceil_div(a.n, 256 * 4 * 4);
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_ts_hist, dim3((uint32_t)blocks), dim3(256), 0, s, ta);
  return hipGetLastError();
}

}  // namespace argus
