// k_samples.hip -- PC samples attributed to region instances, and PC-keyed
// metrics lifted into regions.
//
// The paper's Section 3.2 maps PC-keyed evidence to regions with a separate
// mapping run: each warp's region transitions are replayed as a stack of
// open regions, and an execution of the instruction at PC p counts for the
// region that is innermost at that moment.  Section 3.5 turns the counts
// n(r, p) into weights alpha(r, p) = n(r, p) / sum_r' n(r', p), lifts an
// additive metric as m_hat(r) = sum_p alpha(r, p) m(p) and reports the
// association entropy H(p) = -sum_r alpha log alpha.
//
// Here the stacks are already resolved: argus_attr_run wrote every instance
// with its interval, level and parent, in (context, begin time) order.  So
// the instances active at time t in a context are exactly the ancestors (or
// self) of the last instance of that context that began at or before t
// which have not ended by t: one binary search and a short walk up the
// parent links give a sample's owner, the innermost matched active
// instance.  The counts go to a dense [P][R] table with 64-bit atomics
// (integer, so the order of the adds does not matter).  Per PC one wave
// forms T(p), alpha, the owner count and H(p); per region one block adds
// the separately rounded products alpha * m(p) in a fixed order (512
// strands by p mod 512, combined by halving), so m_hat is reproducible bit
// for bit.
#include <string.h>

#include <mutex>

#include "internal.h"

// Every product is rounded before it is added: hipcc would otherwise fuse
// a * b + c into one fused multiply-add, which rounds once (the file is
// also built with -ffp-contract=off).
#pragma clang fp contract(off)

namespace argus {

struct SampArgs {
  const argus_instance* inst;
  const uint64_t* n_inst;
  uint64_t max_inst;
  const uint4* smp;
  uint64_t ns;
  const uint32_t* w;
  const double* metrics;
  uint32_t R, P, M;
  uint64_t* counters;
  uint64_t* n;
  double* alpha;
  uint64_t* pc_total;
  uint32_t* owners;
  double* entropy;
  uint64_t* region_total;
  double* mhat;
};

constexpr int kSampThreads = 256;

// Zero the count table and the counters (a fill kernel: no memset node when
// the caller captures the launch in a graph).
__global__ __launch_bounds__(kSampThreads) void k_s_clear(SampArgs a) {
  const uint64_t total = (uint64_t)a.P * a.R;
  const uint64_t stride = (uint64_t)gridDim.x * kSampThreads;
  for (uint64_t i = (uint64_t)blockIdx.x * kSampThreads + threadIdx.x; i < total; i += stride)
    a.n[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x < ARGUS_S_NUM_COUNTERS) a.counters[threadIdx.x] = 0;
}

// Sum of a per-thread u64 over the block, added to *dst by one thread.
__device__ __forceinline__ void block_add(uint64_t v, uint64_t* dst, uint64_t* s_part) {
  v = row_sum64(v);
  v = rows_sum64(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) s_part[w] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t t = 0;
    for (int k = 0; k < kSampThreads / 64; ++k) t += s_part[k];
    if (t) atomicAdd((unsigned long long*)dst, (unsigned long long)t);
  }
  __syncthreads();
}

__global__ __launch_bounds__(kSampThreads) void k_s_join(SampArgs a) {
  __shared__ uint64_t s_part[kSampThreads / 64];
  const uint64_t avail = *a.n_inst;
  const uint64_t ni = avail < a.max_inst ? avail : a.max_inst;
  const uint4* inst = reinterpret_cast<const uint4*>(a.inst);  // two uint4 per instance
  uint64_t bad = 0, wt = 0, watt = 0, wun = 0, winner = 0, wbadi = 0;
  const uint64_t stride = (uint64_t)gridDim.x * kSampThreads;
  // blocks go to the 8 XCDs round-robin: give each XCD a contiguous eighth
  // of the block indices (when the grid divides by 8), so that neighbouring
  // samples, whose searches end in the same lines, share one L2
  const uint32_t G = gridDim.x;
  const uint32_t bid = G % 8 == 0 ? (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8 : blockIdx.x;
  // The owner of one sample from its search result: walk up from the last
  // instance that began at or before ts; the active ones are its ancestors
  // (or itself) that have not ended by ts, and the first matched one among
  // them is the owner.
  auto finish = [&](uint64_t lo, uint64_t ts, uint32_t ctx, uint32_t pc, uint64_t w) {
    int64_t owner_region = -1;
    bool inner = false;
    uint64_t x = lo;  // one past the candidate
    while (x > 0) {
      const uint64_t y = x - 1;
      const uint4 h0 = inst[2 * y];
      const uint4 h1 = inst[2 * y + 1];
      // every word the step uses loaded before the first test (the compiler
      // would otherwise load each after the test before it)
      asm volatile("" ::"v"(h0.z), "v"(h0.w), "v"(h1.x), "v"(h1.y), "v"(h1.w));
      if (h1.x != ctx) break;
      const uint64_t t_end = (uint64_t)h0.z | ((uint64_t)h0.w << 32);
      const uint32_t reg = h1.w & 0xFFFFu, ereg = h1.w >> 16;
      const bool closed = ereg != kNoEnd;
      if (!closed || ts < t_end) {
        if (closed && ereg == reg) {
          owner_region = reg < a.R ? (int64_t)reg : -2;  // -2: not an instance of this R
          break;
        }
        inner = true;
      }
      // parents precede their children; anything else ends the walk
      if (h1.y >= y) break;
      x = (uint64_t)h1.y + 1;
    }
    if (owner_region < 0) {
      if (owner_region == -2) wbadi += w;
      else wun += w;
      return;
    }
    watt += w;
    if (inner) winner += w;
    atomicAdd((unsigned long long*)&a.n[(uint64_t)pc * a.R + (uint64_t)owner_region],
              (unsigned long long)w);
  };
  // Two samples per thread (i and i + stride), their searches in lockstep:
  // each search is a chain of dependent loads, and two chains per lane keep
  // twice the requests in flight.  The search finds the first instance whose
  // (context, begin time) exceeds the sample's; the key is compared with
  // bitwise operators, so that a level's two loads go out together.
  for (uint64_t i = (uint64_t)bid * kSampThreads + threadIdx.x; i < a.ns; i += 2 * stride) {
    const uint64_t i1 = i + stride;
    const bool has1 = i1 < a.ns;
    const uint4 s0 = a.smp[i], s1 = a.smp[has1 ? i1 : i];
    const uint64_t ts0 = (uint64_t)s0.x | ((uint64_t)s0.y << 32);
    const uint64_t ts1 = (uint64_t)s1.x | ((uint64_t)s1.y << 32);
    const uint32_t ctx0 = s0.z, pc0 = s0.w, ctx1 = s1.z, pc1 = s1.w;
    const uint64_t w0 = a.w ? (uint64_t)a.w[i] : 1ull;
    const uint64_t w1 = a.w ? (uint64_t)a.w[has1 ? i1 : i] : 1ull;
    const bool ok0 = pc0 < a.P, ok1 = has1 && pc1 < a.P;
    if (ok0) wt += w0;
    else bad += 1;
    if (has1) {
      if (ok1) wt += w1;
      else bad += 1;
    }
    uint64_t lo0 = 0, hi0 = ok0 ? ni : 0, lo1 = 0, hi1 = ok1 ? ni : 0;
    while ((lo0 < hi0) | (lo1 < hi1)) {
      const bool a0 = lo0 < hi0, a1 = lo1 < hi1;
      const uint64_t m0 = (lo0 + hi0) >> 1, m1 = (lo1 + hi1) >> 1;
      const uint64_t q0 = a0 ? m0 : 0, q1 = a1 ? m1 : 0;  // a finished chain reads instance 0
      const uint4 g0 = inst[2 * q0], g1 = inst[2 * q1];
      const uint32_t c0 = inst[2 * q0 + 1].x, c1 = inst[2 * q1 + 1].x;
      const uint64_t tb0 = (uint64_t)g0.x | ((uint64_t)g0.y << 32);
      const uint64_t tb1 = (uint64_t)g1.x | ((uint64_t)g1.y << 32);
      const bool gt0 = (c0 > ctx0) | ((c0 == ctx0) & (tb0 > ts0));
      const bool gt1 = (c1 > ctx1) | ((c1 == ctx1) & (tb1 > ts1));
      if (a0) {
        if (gt0) hi0 = m0;
        else lo0 = m0 + 1;
      }
      if (a1) {
        if (gt1) hi1 = m1;
        else lo1 = m1 + 1;
      }
    }
    if (ok0) finish(lo0, ts0, ctx0, pc0, w0);
    if (ok1) finish(lo1, ts1, ctx1, pc1, w1);
  }
  block_add(bad, &a.counters[ARGUS_S_N_BAD_PC], s_part);
  block_add(wt, &a.counters[ARGUS_S_W_TOTAL], s_part);
  block_add(watt, &a.counters[ARGUS_S_W_ATTRIBUTED], s_part);
  block_add(wun, &a.counters[ARGUS_S_W_UNATTRIBUTED], s_part);
  block_add(winner, &a.counters[ARGUS_S_W_INNER_UNMATCHED], s_part);
  block_add(wbadi, &a.counters[ARGUS_S_W_BAD_INSTANCE], s_part);
  if (blockIdx.x == 0 && threadIdx.x == 0) a.counters[ARGUS_S_N_SAMPLES] = a.ns;
}

// One wave per PC: T(p), the owners, alpha (one rounded division each) and
// H(p) (per-lane sums, then a fixed butterfly over the wave).
constexpr int kPcRegs = 4;  // rows of up to 256 regions held in registers
__global__ __launch_bounds__(kSampThreads) void k_s_pc(SampArgs a) {
  const uint64_t wave = ((uint64_t)blockIdx.x * kSampThreads + threadIdx.x) >> 6;
  const uint64_t nwaves = (uint64_t)gridDim.x * (kSampThreads / 64);
  const uint32_t lane = threadIdx.x & 63;
  uint64_t pairs = 0;
  for (uint64_t p = wave; p < a.P; p += nwaves) {
    const uint64_t* row = a.n + p * a.R;
    double* arow = a.alpha + p * a.R;
    uint64_t t = 0;
    uint32_t own = 0;
    double h = 0.0;
    if (a.R <= 64 * kPcRegs) {
      // the row in registers, its loads issued together (indices clamped to
      // the row), read once for the total, alpha and H
      uint64_t v[kPcRegs];
#pragma unroll
      for (int k = 0; k < kPcRegs; ++k) {
        const uint32_t r = lane + 64u * k;
        v[k] = row[r < a.R ? r : a.R - 1];
      }
#pragma unroll
      for (int k = 0; k < kPcRegs; ++k) {
        if (lane + 64u * k >= a.R) v[k] = 0;
        t += v[k];
        own += v[k] != 0;
      }
      t = rows_sum64(row_sum64(t));
      own = rows_sum32(row_sum32(own));
      const double td = (double)t;
#pragma unroll
      for (int k = 0; k < kPcRegs; ++k) {
        const uint32_t r = lane + 64u * k;
        double al = 0.0;
        if (v[k]) {
          al = (double)v[k] / td;
          const double t_h = al * log(al);
          h = h - t_h;
        }
        if (r < a.R) arow[r] = al;
      }
    } else {
      for (uint32_t r = lane; r < a.R; r += 64) {
        const uint64_t v = row[r];
        t += v;
        own += v != 0;
      }
      t = rows_sum64(row_sum64(t));
      own = rows_sum32(row_sum32(own));
      const double td = (double)t;
      for (uint32_t r = lane; r < a.R; r += 64) {
        const uint64_t v = row[r];
        double al = 0.0;
        if (v) {
          al = (double)v / td;
          const double t_h = al * log(al);
          h = h - t_h;
        }
        arow[r] = al;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) h = h + __shfl_xor(h, off);
    if (lane == 0) {
      a.pc_total[p] = t;
      a.owners[p] = own;
      a.entropy[p] = h;
    }
    pairs += own;
  }
  if (lane == 0 && pairs)
    atomicAdd((unsigned long long*)&a.counters[ARGUS_S_N_PAIRS], (unsigned long long)pairs);
}

// Per region r: its total count (an integer sum, in any order), and each
// lifted metric as the products alpha(r, p) * m(p), each rounded, summed in
// a fixed order (the paper fixes none): 512 strands, strand j adding from +0
// and in increasing p the products with p mod 512 = j, then the strands
// combined by halving, strand j += strand j + h for j < h, h = 256, ..., 1;
// m_hat(r) is strand 0.  One block of 512 threads per region and pair of
// metrics: thread j is strand j, with the loads of kLiftRounds values of p
// issued together; the halving runs through LDS down to 64 strands, then
// within one wave.
//
// alpha(r, p) is zero exactly where the count is (a non-zero count over a
// total below 2^64 is at least 2^-64), and a sum that starts at +0 never
// becomes -0 under round-to-nearest, so a p without a count adds +0 and
// leaves the strand unchanged bit for bit: strands need no selection of
// their terms across lanes.
constexpr uint32_t kLiftMetrics = 2;
constexpr uint32_t kLiftStrands = 512;
constexpr int kLiftRounds = 8;  // values of p per strand and load batch

__global__ __launch_bounds__(kLiftStrands) void k_s_region(SampArgs a) {
  __shared__ double s_acc[kLiftMetrics][kLiftStrands];
  __shared__ uint64_t s_tot[kLiftStrands / 64];
  // Blocks go to the 8 XCDs round-robin; the regions of one XCD are made
  // consecutive, so that the column lines they share (8 regions per 64-byte
  // line of n and alpha) come through that XCD's L2 once.
  const uint32_t per = (a.R + 7) / 8;
  const uint64_t r = (uint64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
  if (r >= a.R) return;  // the whole block, before any barrier
  const uint32_t j = threadIdx.x, lane = j & 63, w = j >> 6;
  const bool totals = blockIdx.y == 0;
  const uint32_t k0 = blockIdx.y * kLiftMetrics;
  const uint32_t mk = a.M > k0 ? (a.M - k0 < kLiftMetrics ? a.M - k0 : kLiftMetrics) : 0u;
  const double* m0 = mk > 0 ? a.metrics + (uint64_t)k0 * a.P : nullptr;
  const double* m1 = mk > 1 ? a.metrics + (uint64_t)(k0 + 1) * a.P : nullptr;
  uint64_t tot = 0;
  double acc0 = 0.0, acc1 = 0.0;
  for (uint64_t p0 = 0; p0 < a.P; p0 += (uint64_t)kLiftStrands * kLiftRounds) {
    uint64_t nv[kLiftRounds];
    double al[kLiftRounds], x0[kLiftRounds], x1[kLiftRounds];
    // indices clamped to P - 1 (the values of p >= P are dropped below),
    // each array's loads in one block so that they go out together
    if (totals) {
#pragma unroll
      for (int u = 0; u < kLiftRounds; ++u) {
        const uint64_t p = p0 + (uint64_t)kLiftStrands * u + j;
        nv[u] = a.n[(p < a.P ? p : a.P - 1) * a.R + r];
      }
    }
    if (m0) {
#pragma unroll
      for (int u = 0; u < kLiftRounds; ++u) {
        const uint64_t p = p0 + (uint64_t)kLiftStrands * u + j;
        const uint64_t pc = p < a.P ? p : a.P - 1;
        al[u] = a.alpha[pc * a.R + r];
        x0[u] = m0[pc];
      }
    }
    if (m1) {
#pragma unroll
      for (int u = 0; u < kLiftRounds; ++u) {
        const uint64_t p = p0 + (uint64_t)kLiftStrands * u + j;
        x1[u] = m1[p < a.P ? p : a.P - 1];
      }
    }
#pragma unroll
    for (int u = 0; u < kLiftRounds; ++u) {
      const uint64_t p = p0 + (uint64_t)kLiftStrands * u + j;
      const bool in = p < a.P;
      if (totals) tot += in ? nv[u] : 0ull;
      if (m0) {
        const bool has = in && al[u] != 0.0;
        acc0 = acc0 + (has ? al[u] * x0[u] : 0.0);
        if (m1) acc1 = acc1 + (has ? al[u] * x1[u] : 0.0);
      }
    }
  }
  if (mk > 0) {
    s_acc[0][j] = acc0;
    s_acc[1][j] = acc1;
  }
  if (totals) {
    const uint64_t t = rows_sum64(row_sum64(tot));
    if (lane == 0) s_tot[w] = t;
  }
  __syncthreads();
  if (mk > 0) {
    for (uint32_t h = kLiftStrands / 2; h >= 64; h >>= 1) {
      if (j < h) {
        s_acc[0][j] = s_acc[0][j] + s_acc[0][j + h];
        s_acc[1][j] = s_acc[1][j] + s_acc[1][j + h];
      }
      __syncthreads();
    }
    if (w == 0) {
      double v0 = s_acc[0][lane], v1 = s_acc[1][lane];
#pragma unroll
      for (int h = 32; h >= 1; h >>= 1) {
        v0 = v0 + __shfl_down(v0, h);
        v1 = v1 + __shfl_down(v1, h);
      }
      if (lane == 0) {
        a.mhat[(uint64_t)k0 * a.R + r] = v0;
        if (mk > 1) a.mhat[(uint64_t)(k0 + 1) * a.R + r] = v1;
      }
    }
  }
  if (totals && j == 0) {
    uint64_t t = 0;
    for (uint32_t q = 0; q < kLiftStrands / 64; ++q) t += s_tot[q];
    a.region_total[r] = t;
  }
}

}  // namespace argus

using namespace argus;

namespace {

std::mutex g_dev_mu;
int g_dev_ok[64] = {};  // 1: device checked to be gfx950

int check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ARGUS_E_HIP;
  if (dev < 0 || dev >= 64) return ARGUS_E_DEVICE;
  std::lock_guard<std::mutex> lock(g_dev_mu);
  if (!g_dev_ok[dev]) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return ARGUS_E_HIP;
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return ARGUS_E_DEVICE;
    g_dev_ok[dev] = 1;
  }
  return ARGUS_OK;
}

bool aligned(const void* p, uintptr_t to) { return ((uintptr_t)p & (to - 1)) == 0; }

uint32_t grid_for(uint64_t items, uint64_t per_block, uint32_t cap) {
  uint64_t g = (items + per_block - 1) / per_block;
  if (g > cap) g = cap;
  return g < 1 ? 1u : (uint32_t)g;
}

}  // namespace

extern "C" int argus_attr_samples(const argus_samples_config* cfg, const argus_samples_io* io,
                                  void* stream_v) {
  if (!cfg || !io) return ARGUS_E_INVAL;
  if (cfg->abi_version != ARGUS_ATTR_ABI_VERSION) return ARGUS_E_ABI;
  const uint64_t R = cfg->num_regions, P = cfg->num_pcs, M = cfg->num_metrics;
  if (R < 1 || R > 65535 || P < 1 || P > (1u << 24) || M > 64) return ARGUS_E_INVAL;
  if (P * R > (1ull << 31)) return ARGUS_E_CAPACITY;
  if (!io->d_n_instances || (io->max_instances > 0 && !io->d_instances)) return ARGUS_E_INVAL;
  if (io->n_samples > 0 && !io->d_samples) return ARGUS_E_INVAL;
  if (!io->d_counters || !io->d_n || !io->d_alpha || !io->d_pc_total || !io->d_pc_owners ||
      !io->d_entropy || !io->d_region_total)
    return ARGUS_E_INVAL;
  if (M > 0 && (!io->d_metrics || !io->d_mhat)) return ARGUS_E_INVAL;
  if (!aligned(io->d_instances, 16) || !aligned(io->d_samples, 16) ||
      !aligned(io->d_n_instances, 8) || !aligned(io->d_weights, 4) ||
      !aligned(io->d_metrics, 8) || !aligned(io->d_counters, 8) || !aligned(io->d_n, 8) ||
      !aligned(io->d_alpha, 8) || !aligned(io->d_pc_total, 8) || !aligned(io->d_pc_owners, 4) ||
      !aligned(io->d_entropy, 8) || !aligned(io->d_region_total, 8) || !aligned(io->d_mhat, 8))
    return ARGUS_E_ALIGN;
  const int dc = check_device();
  if (dc != ARGUS_OK) return dc;

  SampArgs a{};
  a.inst = io->d_instances;
  a.n_inst = io->d_n_instances;
  a.max_inst = io->max_instances;
  a.smp = reinterpret_cast<const uint4*>(io->d_samples);
  a.ns = io->n_samples;
  a.w = io->d_weights;
  a.metrics = io->d_metrics;
  a.R = (uint32_t)R;
  a.P = (uint32_t)P;
  a.M = (uint32_t)M;
  a.counters = io->d_counters;
  a.n = io->d_n;
  a.alpha = io->d_alpha;
  a.pc_total = io->d_pc_total;
  a.owners = io->d_pc_owners;
  a.entropy = io->d_entropy;
  a.region_total = io->d_region_total;
  a.mhat = io->d_mhat;
  hipStream_t s = (hipStream_t)stream_v;
  hipLaunchKernelGGL(k_s_clear, dim3(grid_for(P * R, kSampThreads, 4096)), dim3(kSampThreads), 0,
                     s, a);
  hipLaunchKernelGGL(k_s_join, dim3(grid_for(a.ns, kSampThreads, 4096)), dim3(kSampThreads), 0, s,
                     a);
  hipLaunchKernelGGL(k_s_pc, dim3(grid_for(P, kSampThreads / 64, 4096)), dim3(kSampThreads), 0,
                     s, a);
  const uint32_t lift_y = M > 0 ? (uint32_t)((M + kLiftMetrics - 1) / kLiftMetrics) : 1u;
  hipLaunchKernelGGL(k_s_region, dim3(8 * (uint32_t)((R + 7) / 8), lift_y), dim3(kLiftStrands), 0, s,
                     a);
  return hipGetLastError() == hipSuccess ? ARGUS_OK : ARGUS_E_HIP;
}
