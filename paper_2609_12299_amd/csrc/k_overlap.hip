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
// per-context runs of the sorted records (k_merge: one word per record,
// group | time | code) or by a radix sort of (group, time) keys with a class
// payload (k_radix).  This kernel
// scans the per-class active counts c (segmented by group, decoupled
// look-back across tiles) and, for each gap between consecutive events of a
// group, adds gap * [c_A > 0 and c_B > 0] to U and gap * c_A * c_B (or
// gap * c_A (c_A - 1) / 2 for A == B) to Q.  Equal times give zero gaps, so
// the order among ties does not matter.
#include "internal.h"

namespace argus {

constexpr int kSweepQWords = 36;  // stride of the per-group U and Q rows

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
__host__ __device__ constexpr int pair_index(int a, int b) {
  return a * KM - a * (a - 1) / 2 + (b - a);
}

template <int KM>
__global__ __launch_bounds__(kSweepThreads) void k_sweep(SweepArgs a) {
  constexpr int NP = KM * (KM + 1) / 2;
  const DevPlan* P = a.plan;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  __shared__ uint32_t s_tile;
  __shared__ uint64_t s_t[kSweepTile];
  __shared__ uint32_t s_g[kSweepTile];
  __shared__ uint32_t s_pay[kSweepTile];
  __shared__ uint64_t s_u[kSweepSlots][NP];
  __shared__ uint64_t s_q[kSweepSlots][NP];
  __shared__ int32_t s_wd[4][KM];
  __shared__ uint32_t s_wr[4];
  __shared__ int32_t s_cin[KM];
  __shared__ uint32_t s_prev_g, s_has_prev, s_next_g, s_has_next;
  __shared__ uint64_t s_next_t;

  const uint64_t n = P->n_ev;
  const uint64_t tiles = ceil_div(n, kSweepTile);
  for (;;) {
  if (tid == 0) s_tile = atomicAdd(&a.tile_ctr[kCtrSweep], 1u);
  __syncthreads();
  const uint64_t tile = s_tile;
  if (tile >= tiles) break;
  const KeySpace ks = P->ev;
  const bool wide = ks.wide != 0;
  const uint32_t buf = P->ev_final;
  const uint64_t* gk = a.key[buf];
  const uint32_t* gp = a.pay[buf];
  const uint32_t* gc = a.ctxw[buf];
  const uint64_t base = tile * kSweepTile;
  const uint32_t cnt = n - base < (uint64_t)kSweepTile ? (uint32_t)(n - base) : (uint32_t)kSweepTile;
  auto grp = [&](uint64_t k, uint32_t cw) -> uint32_t {
    return wide ? cw : (ks.ts_bits >= 64 ? 0u : (uint32_t)(k >> ks.ts_bits));
  };
  auto tof = [&](uint64_t k) -> uint64_t { return wide ? k : (k & ks.ts_mask); };
  // Merged event words: key = word >> 5; code 0 (no event) gets a class
  // that matches no counter.
  const bool mfmt = P->ev_merge != 0;
  auto key_at = [&](uint64_t i) -> uint64_t { return mfmt ? gk[i] >> kEvCodeBits : gk[i]; };
  auto pay_at = [&](uint64_t i) -> uint32_t {
    if (!mfmt) return gp[i];
    const uint32_t c = (uint32_t)(gk[i] & ((1u << kEvCodeBits) - 1u));
    return c ? ((c - 1u) >> 1) | (((c - 1u) & 1u) << 8) : 0xFFu;
  };

  for (int j = 0; j < kSweepItems; ++j) {
    const uint32_t i = (uint32_t)j * kSweepThreads + tid;
    if (i < cnt) {
      const uint64_t k = key_at(base + i);
      s_t[i] = tof(k);
      s_g[i] = grp(k, wide ? gc[base + i] : 0u);
      s_pay[i] = pay_at(base + i);
    }
  }
  for (int i = tid; i < kSweepSlots * NP; i += kSweepThreads) {
    (&s_u[0][0])[i] = 0;
    (&s_q[0][0])[i] = 0;
  }
  if (tid == 0) {
    s_has_prev = base > 0;
    s_prev_g = base > 0 ? grp(key_at(base - 1), wide ? gc[base - 1] : 0u) : 0u;
    s_has_next = base + cnt < n;
    if (base + cnt < n) {
      const uint64_t k = key_at(base + cnt);
      s_next_g = grp(k, wide ? gc[base + cnt] : 0u);
      s_next_t = tof(k);
    }
  }
  __syncthreads();

  // ---- per-thread aggregate: reset flag and count deltas since the last start
  const uint32_t p0 = (uint32_t)tid * kSweepItems;
  uint32_t reset = 0;
  int32_t d[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) d[k] = 0;
#pragma unroll
  for (int i = 0; i < kSweepItems; ++i) {
    const uint32_t p = p0 + i;
    if (p >= cnt) break;
    const uint32_t g = s_g[p];
    const bool head = p == 0 ? (!s_has_prev || s_prev_g != g) : s_g[p - 1] != g;
    if (head) {
      reset = 1;
#pragma unroll
      for (int k = 0; k < KM; ++k) d[k] = 0;
    }
    const uint32_t py = s_pay[p];
    const int32_t delta = ((py >> 8) & 1u) ? -1 : 1;
#pragma unroll
    for (int k = 0; k < KM; ++k) d[k] += ((py & 0xFFu) == (uint32_t)k) ? delta : 0;
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

  // ---- look-back for the counts entering the tile
  if (tid == 0) {
    uint32_t tr = 0;
    int32_t td[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) td[k] = 0;
    for (int q = 0; q < 4; ++q) {
      if (s_wr[q]) {
        tr = 1;
#pragma unroll
        for (int k = 0; k < KM; ++k) td[k] = s_wd[q][k];
      } else {
#pragma unroll
        for (int k = 0; k < KM; ++k) td[k] += s_wd[q][k];
      }
    }
    int64_t cin[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    uint64_t* lb = a.slb + tile * 8;
    if (tile > 0) {
      uint64_t w0 = kFlagAgg | ((uint64_t)tr << 61), w1 = kFlagAgg;
      for (int k = 0; k < 4 && k < KM; ++k) w0 |= (uint64_t)(td[k] + 2048) << (13 * k);
      for (int k = 4; k < KM; ++k) w1 |= (uint64_t)(td[k] + 2048) << (13 * (k - 4));
      st_agent(&lb[0], w0);
      st_agent(&lb[1], w1);
      int64_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      int64_t tt = (int64_t)tile - 1;
      uint32_t spins = 0;
      while (tt >= 0) {
        const uint64_t* l = a.slb + (uint64_t)tt * 8;
        uint64_t iw[4];
        bool incl = true;
        for (int q = 0; q < 4; ++q) {
          iw[q] = ld_agent(&l[2 + q]);
          incl &= (iw[q] & ~kValMask) == kFlagIncl;
        }
        if (incl) {
          for (int k = 0; k < 8; ++k) {
            const uint64_t v = (iw[k >> 1] >> (31 * (k & 1))) & 0x7FFFFFFFull;
            cin[k] = (int64_t)v + acc[k];
          }
          break;
        }
        const uint64_t a0 = ld_agent(&l[0]), a1 = ld_agent(&l[1]);
        if ((a0 & ~kValMask) == kFlagAgg && (a1 & ~kValMask) == kFlagAgg) {
          for (int k = 0; k < 4; ++k) acc[k] += (int64_t)((a0 >> (13 * k)) & 0x1FFFull) - 2048;
          for (int k = 4; k < 8; ++k) acc[k] += (int64_t)((a1 >> (13 * (k - 4))) & 0x1FFFull) - 2048;
          if ((a0 >> 61) & 1ull) {
            for (int k = 0; k < 8; ++k) cin[k] = acc[k];
            break;
          }
          --tt;
          continue;
        }
        if (++spins > kMaxSpins) {
          flag_internal_error(a.counters, 128);
          break;
        }
        backoff();
      }
    }
    int64_t cout[8];
    for (int k = 0; k < 8; ++k) cout[k] = (k < KM) ? (tr ? td[k] : cin[k] + td[k]) : 0;
    for (int q = 0; q < 4; ++q)
      st_agent(&lb[2 + q], kFlagIncl | (uint64_t)cout[2 * q] | ((uint64_t)cout[2 * q + 1] << 31));
#pragma unroll
    for (int k = 0; k < KM; ++k) s_cin[k] = (int32_t)cin[k];
  }
  __syncthreads();

  // ---- sweep this thread's events
  int32_t c[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) c[k] = pr ? pd[k] : s_cin[k] + pd[k];
  const uint32_t g0 = s_g[0];
  uint64_t u[NP], q[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    u[k] = 0;
    q[k] = 0;
  }
  uint32_t qg = p0 < cnt ? s_g[p0] : g0;
  const uint32_t K = a.K;
  auto flush = [&](uint32_t g) {
    const uint32_t slot = g - g0;
    if (g >= a.G) return;
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      if (u[k]) {
        if (slot < kSweepSlots) atomicAdd((unsigned long long*)&s_u[slot][k], (unsigned long long)u[k]);
        else atomicAdd((unsigned long long*)&a.ov_u[(uint64_t)g * kSweepQWords + k], (unsigned long long)u[k]);
      }
      if (q[k]) {
        if (slot < kSweepSlots) atomicAdd((unsigned long long*)&s_q[slot][k], (unsigned long long)q[k]);
        else atomicAdd((unsigned long long*)&a.ov_q[(uint64_t)g * kSweepQWords + k], (unsigned long long)q[k]);
      }
      u[k] = 0;
      q[k] = 0;
    }
  };
  bool flushed_early = false;
#pragma unroll
  for (int i = 0; i < kSweepItems; ++i) {
    const uint32_t p = p0 + i;
    if (p >= cnt) break;
    const uint32_t g = s_g[p];
    const bool head = p == 0 ? (!s_has_prev || s_prev_g != g) : s_g[p - 1] != g;
    if (head) {
#pragma unroll
      for (int k = 0; k < KM; ++k) c[k] = 0;
    }
    if (g != qg) {
      flush(qg);
      flushed_early = true;
      qg = g;
    }
    const uint32_t py = s_pay[p];
    const int32_t delta = ((py >> 8) & 1u) ? -1 : 1;
#pragma unroll
    for (int k = 0; k < KM; ++k) c[k] += ((py & 0xFFu) == (uint32_t)k) ? delta : 0;
    uint64_t gap = 0;
    if (p + 1 < cnt) {
      if (s_g[p + 1] == g) gap = s_t[p + 1] - s_t[p];
    } else if (s_has_next && s_next_g == g) {
      gap = s_next_t - s_t[p];
    }
    if (gap == 0) continue;
#pragma unroll
    for (int x = 0; x < KM; ++x) {
#pragma unroll
      for (int y = x; y < KM; ++y) {
        if ((uint32_t)y >= K) continue;
        const int pi = pair_index<KM>(x, y);
        const uint64_t cx = (uint64_t)(c[x] > 0 ? c[x] : 0), cy = (uint64_t)(c[y] > 0 ? c[y] : 0);
        if (cx > 0 && cy > 0) u[pi] += gap;
        if (x != y) q[pi] += gap * cx * cy;
        else if (cx > 1) q[pi] += gap * (cx * (cx - 1) / 2);
      }
    }
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
  // ---- tile flush of the LDS slots
  const uint32_t last_g = s_g[cnt - 1];
  const uint32_t nslots = (last_g - g0 + 1) < (uint32_t)kSweepSlots ? last_g - g0 + 1 : (uint32_t)kSweepSlots;
  for (uint32_t i = tid; i < nslots * NP; i += kSweepThreads) {
    const uint32_t slot = i / NP, k = i % NP;
    const uint64_t gg = (uint64_t)(g0 + slot);
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

__global__ __launch_bounds__(256) void k_ov_final(OvFinalArgs a) {
  const uint64_t KK = (uint64_t)a.K * a.K;
  const uint64_t total = (uint64_t)a.G * KK;
  for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (uint64_t)gridDim.x * 256) {
    const uint64_t g = i / KK;
    const uint32_t ab = (uint32_t)(i % KK), x = ab / a.K, y = ab % a.K;
    const uint32_t lo = x < y ? x : y, hi = x < y ? y : x;
    const uint32_t pi = lo * a.KM - lo * (lo - 1) / 2 + (hi - lo);
    const uint64_t u = a.ov_u[g * kSweepQWords + pi], q = a.ov_q[g * kSweepQWords + pi];
    a.og[g * 2 * KK + ab] = u;
    a.og[g * 2 * KK + KK + ab] = q;
    if (u) atomicAdd((unsigned long long*)&a.ogl[ab], (unsigned long long)u);
    if (q) atomicAdd((unsigned long long*)&a.ogl[KK + ab], (unsigned long long)q);
  }
}

hipError_t launch_ov_final(const RunArgs& a, hipStream_t s) {
  const uint32_t KM = a.K <= 2 ? 2 : (a.K <= 4 ? 4 : 8);
  OvFinalArgs f{a.w.ov_mask, a.w.ov_q, a.out.d_overlap_group, a.out.d_overlap_global, a.K, a.G, KM};
  uint64_t blocks = ceil_div((uint64_t)a.G * a.K * a.K, 256);
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_ov_final, dim3((uint32_t)blocks), dim3(256), 0, s, f);
  return hipGetLastError();
}

}  // namespace argus
