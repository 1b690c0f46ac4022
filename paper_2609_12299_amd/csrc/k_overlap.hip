// k_overlap.hip -- compute/communication overlap between region classes.
//
// The paper's Section 4.3 tunes compute/communication overlap from region
// timings; the quantity here is, per group of contexts (an SM subset, the
// paper's Section 3.2 scope), and for every pair of classes (A, B):
//   U[A][B] = time during which some class-A and some class-B instance are
//             active (for A == B: time during which class A is active);
//   Q[A][B] = sum over pairs of distinct instances, one of class A and one
//             of class B (unordered pairs when A == B), of their intersection.
// Events (t_begin, +1, class) and (t_end, -1, class) of matched, classified
// instances are put in (group, time) order beforehand, either by merging the
// per-context runs of the sorted records (k_merge.hip, whose last round also
// sweeps) or, when merging does not apply, by a radix sort of (group, time)
// keys with a class payload (k_radix).  This kernel sweeps the radix-sorted
// events: it scans the per-class active counts c (segmented by group,
// decoupled look-back across tiles) and, for each gap between consecutive
// events of a group, adds gap * [c_A > 0 and c_B > 0] to U and gap * c_A *
// c_B (or gap * c_A (c_A - 1) / 2 for A == B) to Q.  Equal times give zero
// gaps, so the order among ties does not matter.
#include "sweep_common.h"

namespace argus {

template <int KM>
struct Counts {
  int32_t c[KM];
};

struct SweepArgs {
  const DevPlan* plan;
  const uint64_t* key[2];
  const uint32_t* pay[2];
  const uint32_t* ctxw[2];
  uint64_t* slb;
  uint64_t* ov_u;  // [G][36]
  uint64_t* ov_q;  // [G][36]
  uint32_t K;
  uint32_t G;
  uint32_t* tile_ctr;
  uint64_t* counters;
};

template <int KM>
__global__ __launch_bounds__(kSweepThreads) void k_sweep(SweepArgs a) {
  constexpr int NP = KM * (KM + 1) / 2;
  constexpr int IT = kSweepItems;
  const DevPlan* P = a.plan;
  if (P->ev_merge) return;  // merged events are swept by k_merge_sweep
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  __shared__ uint32_t s_tile;
  __shared__ uint64_t s_u[kSweepSlots][NP];
  __shared__ uint64_t s_q[kSweepSlots][NP];
  __shared__ int32_t s_wd[4][KM];
  __shared__ uint32_t s_wr[4];
  __shared__ int32_t s_cin[KM];
  __shared__ uint32_t s_g0;

  const uint64_t n = P->n_ev;
  const uint64_t tiles = ceil_div(n, kSweepTile);
  const KeySpace ks = P->ev;
  const bool wide = ks.wide != 0;
  const uint32_t buf = P->ev_final;
  const uint64_t* gk = a.key[buf];
  const uint32_t* gp = a.pay[buf];
  const uint32_t* gc = a.ctxw[buf];
  constexpr uint32_t kNoGroup = 0xFFFFFFFFu;
  // (group, time, class | is_end << 8) of event i; class 0xFF changes no count
  auto decode = [&](uint64_t k, uint32_t pay, uint32_t cw, uint32_t* g, uint64_t* t,
                    uint32_t* py) {
    *g = wide ? cw : (ks.ts_bits >= 64 ? 0u : (uint32_t)(k >> ks.ts_bits));
    *t = wide ? k : (k & ks.ts_mask);
    *py = pay;
  };
  auto load_one = [&](uint64_t i, uint32_t* g, uint64_t* t, uint32_t* py) {
    decode(gk[i], gp[i], wide ? gc[i] : 0u, g, t, py);
  };

  for (;;) {
  if (tid == 0) s_tile = atomicAdd(&a.tile_ctr[kCtrSweep], 1u);
  for (int i = tid; i < kSweepSlots * NP; i += kSweepThreads) {
    (&s_u[0][0])[i] = 0;
    (&s_q[0][0])[i] = 0;
  }
  __syncthreads();
  const uint64_t tile = s_tile;
  if (tile >= tiles) break;
  const uint64_t base = tile * kSweepTile;
  const uint32_t cnt = n - base < (uint64_t)kSweepTile ? (uint32_t)(n - base) : (uint32_t)kSweepTile;
  const uint32_t p0 = (uint32_t)tid * IT;

  // ---- this thread's 8 consecutive events, the one before and the one after
  uint32_t g[IT], py[IT];
  uint64_t t[IT];
  if (p0 + IT <= cnt && !wide) {
    const uint4* k4 = (const uint4*)(gk + base + p0);
    const uint4* q4 = (const uint4*)(gp + base + p0);
    uint32_t pw[IT];
#pragma unroll
    for (int q = 0; q < IT / 4; ++q) {
      const uint4 v = q4[q];
      pw[4 * q] = v.x;
      pw[4 * q + 1] = v.y;
      pw[4 * q + 2] = v.z;
      pw[4 * q + 3] = v.w;
    }
#pragma unroll
    for (int q = 0; q < IT / 2; ++q) {
      const uint4 v = k4[q];
      decode((uint64_t)v.x | ((uint64_t)v.y << 32), pw[2 * q], 0u, &g[2 * q], &t[2 * q], &py[2 * q]);
      decode((uint64_t)v.z | ((uint64_t)v.w << 32), pw[2 * q + 1], 0u, &g[2 * q + 1],
             &t[2 * q + 1], &py[2 * q + 1]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      g[i] = kNoGroup;
      t[i] = 0;
      py[i] = 0xFFu;
      if (p0 + i < cnt) load_one(base + p0 + i, &g[i], &t[i], &py[i]);
    }
  }
  uint32_t g_prev = kNoGroup, g_next = kNoGroup, pdummy;
  uint64_t t_next = 0, tdummy;
  if (p0 < cnt && base + p0 > 0) load_one(base + p0 - 1, &g_prev, &tdummy, &pdummy);
  if (base + p0 + IT < n && p0 + IT <= cnt) load_one(base + p0 + IT, &g_next, &t_next, &pdummy);
  if (tid == 0) s_g0 = g[0];

  // ---- per-thread aggregate: reset flag and count deltas since the last start
  uint32_t reset = 0;
  int32_t d[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) d[k] = 0;
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    if (g[i] == kNoGroup) continue;
    const uint32_t gb = i > 0 ? g[i - 1] : g_prev;
    if (gb != g[i]) {
      reset = 1;
#pragma unroll
      for (int k = 0; k < KM; ++k) d[k] = 0;
    }
    const int32_t delta = ((py[i] >> 8) & 1u) ? -1 : 1;
#pragma unroll
    for (int k = 0; k < KM; ++k) d[k] += ((py[i] & 0xFFu) == (uint32_t)k) ? delta : 0;
  }
  // wave inclusive scan (g after f: g.reset ? g : f + g)
  uint32_t xr = reset;
  int32_t xd[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) xd[k] = d[k];
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t yr = __shfl_up(xr, o);
    int32_t yd[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) yd[k] = __shfl_up(xd[k], o);
    if (lane >= o && !xr) {
      xr = yr;
#pragma unroll
      for (int k = 0; k < KM; ++k) xd[k] += yd[k];
    }
  }
  uint32_t er = __shfl_up(xr, 1);
  int32_t ed[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) ed[k] = __shfl_up(xd[k], 1);
  if (lane == 0) {
    er = 0;
#pragma unroll
    for (int k = 0; k < KM; ++k) ed[k] = 0;
  }
  if (lane == 63) {
    s_wr[w] = xr;
#pragma unroll
    for (int k = 0; k < KM; ++k) s_wd[w][k] = xd[k];
  }
  __syncthreads();
  // prefix of the earlier waves, then this thread's exclusive map
  uint32_t pr = 0;
  int32_t pd[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) pd[k] = 0;
  for (int q = 0; q < w; ++q) {
    if (s_wr[q]) {
      pr = 1;
#pragma unroll
      for (int k = 0; k < KM; ++k) pd[k] = s_wd[q][k];
    } else {
#pragma unroll
      for (int k = 0; k < KM; ++k) pd[k] += s_wd[q][k];
    }
  }
  if (er) {
    pr = 1;
#pragma unroll
    for (int k = 0; k < KM; ++k) pd[k] = ed[k];
  } else {
#pragma unroll
    for (int k = 0; k < KM; ++k) pd[k] += ed[k];
  }

  // ---- look-back for the counts entering the tile.  Wave 0 inspects 64
  // predecessor tiles per round trip (lane j: the j-th nearest not yet
  // folded in).  A tile's aggregate is (reset, deltas): reset when a group
  // starts inside it, deltas since that start; folding keeps the nearer
  // aggregate whole when it resets.
  if (w == 0) {
    uint32_t tr = 0;
    int32_t td[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) td[k] = 0;
    for (int qq = 0; qq < 4; ++qq) {
      if (s_wr[qq]) {
        tr = 1;
#pragma unroll
        for (int k = 0; k < KM; ++k) td[k] = s_wd[qq][k];
      } else {
#pragma unroll
        for (int k = 0; k < KM; ++k) td[k] += s_wd[qq][k];
      }
    }
    int64_t cin[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) cin[k] = 0;
    uint64_t* lb = a.slb + tile * 8;
    if (tile > 0) {
      if (lane == 0) {
        uint64_t w0 = kFlagAgg | ((uint64_t)tr << 61), w1 = kFlagAgg;
        for (int k = 0; k < 4 && k < KM; ++k) w0 |= (uint64_t)(td[k] + 2048) << (13 * k);
        for (int k = 4; k < KM; ++k) w1 |= (uint64_t)(td[k] + 2048) << (13 * (k - 4));
        st_agent(&lb[0], w0);
        st_agent(&lb[1], w1);
      }
      uint32_t acc_r = 0;  // fold of the tiles between the found one and this tile
      int64_t acc[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) acc[k] = 0;
      int64_t top = (int64_t)tile - 1;
      uint32_t spins = 0;
      for (;;) {
        const int64_t tt = top - lane;
        uint64_t aw0 = 0, aw1 = 0, iw[4] = {0, 0, 0, 0};
        if (tt >= 0) {
          const uint64_t* l = a.slb + (uint64_t)tt * 8;
#pragma unroll
          for (int qq = 0; qq < 4; ++qq) iw[qq] = ld_agent(&l[2 + qq]);
          aw0 = ld_agent(&l[0]);
          aw1 = ld_agent(&l[1]);
        }
        bool incl = true;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) incl &= (iw[qq] & ~kValMask) == kFlagIncl;
        const bool agg = (aw0 & ~kValMask) == kFlagAgg && (aw1 & ~kValMask) == kFlagAgg;
        const uint64_t mi = __ballot(incl), mn = __ballot(!incl && !agg);
        const int ji = mi ? __ffsll((unsigned long long)mi) - 1 : 64;
        const int jn = mn ? __ffsll((unsigned long long)mn) - 1 : 64;
        const bool done = ji < jn;
        const int kk = done ? ji : jn;  // lanes [0, kk) hold aggregates to fold in
        uint32_t xr = 0;
        int32_t xd[KM];
#pragma unroll
        for (int k = 0; k < KM; ++k) xd[k] = 0;
        if (lane < kk) {
          xr = (uint32_t)(aw0 >> 61) & 1u;
#pragma unroll
          for (int k = 0; k < KM; ++k)
            xd[k] = (int32_t)(((k < 4 ? aw0 >> (13 * k) : aw1 >> (13 * (k - 4)))) & 0x1FFFull) - 2048;
        }
        // reduce towards lane 0 (a higher lane is an earlier tile)
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t yr = __shfl_down(xr, o);
          int32_t yd[KM];
#pragma unroll
          for (int k = 0; k < KM; ++k) yd[k] = __shfl_down(xd[k], o);
          if (lane + o < 64 && !xr) {
            xr = yr;
#pragma unroll
            for (int k = 0; k < KM; ++k) xd[k] += yd[k];
          }
        }
        // acc = fold(lanes [0, kk)) then acc
        const uint32_t fr = (uint32_t)__shfl(xr, 0);
        if (!acc_r) {
          acc_r = fr;
#pragma unroll
          for (int k = 0; k < KM; ++k) acc[k] += __shfl(xd[k], 0);
        }
        if (acc_r) {
#pragma unroll
          for (int k = 0; k < KM; ++k) cin[k] = acc[k];
          break;
        }
        if (done) {
#pragma unroll
          for (int k = 0; k < KM; ++k) {
            const uint64_t v = (__shfl(iw[k >> 1], ji) >> (31 * (k & 1))) & 0x7FFFFFFFull;
            cin[k] = (int64_t)v + acc[k];
          }
          break;
        }
        top -= kk;
        if (kk == 0) {
          if (++spins > kMaxSpins) {
            if (lane == 0) flag_internal_error(a.counters, 128);
            break;
          }
          backoff();
        }
      }
    }
    if (lane == 0) {
      int64_t cout[8];
      for (int k = 0; k < 8; ++k) cout[k] = (k < KM) ? (tr ? td[k] : cin[k] + td[k]) : 0;
      for (int qq = 0; qq < 4; ++qq)
        st_agent(&lb[2 + qq], kFlagIncl | (uint64_t)cout[2 * qq] | ((uint64_t)cout[2 * qq + 1] << 31));
#pragma unroll
      for (int k = 0; k < KM; ++k) s_cin[k] = (int32_t)cin[k];
    }
  }
  __syncthreads();

  // ---- sweep this thread's events
  int32_t c[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) c[k] = pr ? pd[k] : s_cin[k] + pd[k];
  const uint32_t g0 = s_g0;
  uint64_t u[NP], q[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    u[k] = 0;
    q[k] = 0;
  }
  uint32_t qg = g[0] != kNoGroup ? g[0] : g0;
  const uint32_t K = a.K;
  auto flush = [&](uint32_t gg) {
    const uint32_t slot = gg - g0;
    if (gg >= a.G) return;
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      if (u[k]) {
        if (slot < kSweepSlots) atomicAdd((unsigned long long*)&s_u[slot][k], (unsigned long long)u[k]);
        else atomicAdd((unsigned long long*)&a.ov_u[(uint64_t)gg * kSweepQWords + k], (unsigned long long)u[k]);
      }
      if (q[k]) {
        if (slot < kSweepSlots) atomicAdd((unsigned long long*)&s_q[slot][k], (unsigned long long)q[k]);
        else atomicAdd((unsigned long long*)&a.ov_q[(uint64_t)gg * kSweepQWords + k], (unsigned long long)q[k]);
      }
      u[k] = 0;
      q[k] = 0;
    }
  };
  bool flushed_early = false;
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    if (g[i] == kNoGroup) break;
    const uint32_t gb = i > 0 ? g[i - 1] : g_prev;
    if (gb != g[i]) {
#pragma unroll
      for (int k = 0; k < KM; ++k) c[k] = 0;
    }
    if (g[i] != qg) {
      flush(qg);
      flushed_early = true;
      qg = g[i];
    }
    const int32_t delta = ((py[i] >> 8) & 1u) ? -1 : 1;
#pragma unroll
    for (int k = 0; k < KM; ++k) c[k] += ((py[i] & 0xFFu) == (uint32_t)k) ? delta : 0;
    const uint32_t gn = i + 1 < IT ? g[i + 1] : g_next;
    const uint64_t tn = i + 1 < IT ? t[i + 1] : t_next;
    if (gn != g[i]) continue;  // last event of its group (or of the data)
    const uint64_t gap = tn - t[i];
    if (gap == 0) continue;
    sweep_gap<KM>(u, q, c, gap, K);
  }
  // Whole waves in one group reduce in registers; everything else goes
  // through LDS atomics.
  const uint32_t g_first = __shfl(qg, 0);
  const bool uniform = __ballot(qg != g_first || flushed_early) == 0ull && (qg - g0) < kSweepSlots;
  if (uniform) {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      uint64_t uv = u[k], qv = q[k];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        uv += __shfl_xor(uv, o);
        qv += __shfl_xor(qv, o);
      }
      u[k] = lane == 0 ? uv : 0;
      q[k] = lane == 0 ? qv : 0;
    }
  }
  flush(qg);
  __syncthreads();
  // ---- tile flush of the LDS slots (slot j: group g0 + j)
  for (uint32_t i = tid; i < (uint32_t)(kSweepSlots * NP); i += kSweepThreads) {
    const uint32_t slot = i / NP, k = i % NP;
    const uint64_t gg = (uint64_t)g0 + slot;
    if (gg >= a.G) continue;
    if (s_u[slot][k]) atomicAdd((unsigned long long*)&a.ov_u[gg * kSweepQWords + k], (unsigned long long)s_u[slot][k]);
    if (s_q[slot][k]) atomicAdd((unsigned long long*)&a.ov_q[gg * kSweepQWords + k], (unsigned long long)s_q[slot][k]);
  }
  __syncthreads();
  }  // tiles
}

hipError_t launch_sweep(const RunArgs& a, hipStream_t s) {
  SweepArgs sa{};
  sa.plan = a.w.plan;
  for (int b = 0; b < 2; ++b) {
    sa.key[b] = a.w.key[b];
    sa.pay[b] = a.w.pay[b];
    sa.ctxw[b] = a.w.ctxw[b];
  }
  sa.slb = a.w.slb;
  sa.ov_u = a.w.ov_mask;
  sa.ov_q = a.w.ov_q;
  sa.K = a.K;
  sa.G = a.G;
  sa.tile_ctr = a.w.tile_ctr;
  sa.counters = a.out.d_counters;
  uint64_t blocks = ceil_div(a.n ? a.n : 1, kSweepTile);
  const void* kern = a.K <= 2 ? (const void*)k_sweep<2> : a.K <= 4 ? (const void*)k_sweep<4> : (const void*)k_sweep<8>;
  const uint64_t resident = persistent_blocks(kern, kSweepThreads);
  if (blocks > resident) blocks = resident;
  if (a.K <= 2)
    hipLaunchKernelGGL(k_sweep<2>, dim3((uint32_t)blocks), dim3(kSweepThreads), 0, s, sa);
  else if (a.K <= 4)
    hipLaunchKernelGGL(k_sweep<4>, dim3((uint32_t)blocks), dim3(kSweepThreads), 0, s, sa);
  else
    hipLaunchKernelGGL(k_sweep<8>, dim3((uint32_t)blocks), dim3(kSweepThreads), 0, s, sa);
  return hipGetLastError();
}

// ------------------------------------------------------------- finalise

struct OvFinalArgs {
  const uint64_t* ov_u;
  const uint64_t* ov_q;
  uint64_t* og;   // [G][2][K][K]
  uint64_t* ogl;  // [2][K][K]
  uint32_t K, G, KM;
};

// The global sums are gathered per block in LDS and added once per block:
// thousands of groups adding straight into the same few words would
// serialise on them.
__global__ __launch_bounds__(256) void k_ov_final(OvFinalArgs a) {
  __shared__ unsigned long long s_g[2 * 64];
  const uint64_t KK = (uint64_t)a.K * a.K;
  const uint64_t total = (uint64_t)a.G * KK;
  for (uint32_t i = threadIdx.x; i < 2 * KK; i += 256) s_g[i] = 0;
  __syncthreads();
  for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (uint64_t)gridDim.x * 256) {
    const uint64_t g = i / KK;
    const uint32_t ab = (uint32_t)(i % KK), x = ab / a.K, y = ab % a.K;
    const uint32_t lo = x < y ? x : y, hi = x < y ? y : x;
    const uint32_t pi = lo * a.KM - lo * (lo - 1) / 2 + (hi - lo);
    const uint64_t u = a.ov_u[g * kSweepQWords + pi], q = a.ov_q[g * kSweepQWords + pi];
    a.og[g * 2 * KK + ab] = u;
    a.og[g * 2 * KK + KK + ab] = q;
    if (u) atomicAdd(&s_g[ab], (unsigned long long)u);
    if (q) atomicAdd(&s_g[KK + ab], (unsigned long long)q);
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < 2 * KK; i += 256)
    if (s_g[i]) atomicAdd((unsigned long long*)&a.ogl[i], s_g[i]);
}

hipError_t launch_ov_final(const RunArgs& a, hipStream_t s) {
  const uint32_t KM = a.K <= 2 ? 2 : (a.K <= 4 ? 4 : 8);
  OvFinalArgs f{a.w.ov_mask, a.w.ov_q, a.out.d_overlap_group, a.out.d_overlap_global, a.K, a.G, KM};
  uint64_t blocks = ceil_div((uint64_t)a.G * a.K * a.K, 256);
  if (blocks > 256) blocks = 256;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_ov_final, dim3((uint32_t)blocks), dim3(256), 0, s, f);
  return hipGetLastError();
}

}  // namespace argus
