// sweep_common.h -- the per-gap accumulation of the class-overlap sweep of
// radix-sorted events, and the layout of the per-group U and Q rows shared
// with the last merge round (which sweeps the events it has just merged).
//
// For each gap between consecutive events of a group, with per-class
// active counts c (after the earlier event):
//   U[A][B] += gap  if c_A > 0 and c_B > 0,
//   Q[A][B] += gap * c_A * c_B  (A != B),  gap * c_A (c_A - 1) / 2  (A == B),
// over class pairs A <= B; all arithmetic mod 2^64.
#pragma once

#include <type_traits>

#include "internal.h"

namespace argus {

constexpr int kSweepQWords = 36;  // stride of the per-group U and Q rows

template <int KM>
__host__ __device__ constexpr int pair_index(int a, int b) {
  return a * KM - a * (a - 1) / 2 + (b - a);
}

// a * b mod 2^64 for a 32-bit b
__device__ __forceinline__ uint64_t mul64x32(uint64_t a, uint32_t b) {
  return (uint64_t)(uint32_t)a * b + ((uint64_t)((uint32_t)(a >> 32) * b) << 32);
}

// Adds one gap (gap > 0) to the U and Q accumulators of NP = KM (KM + 1) / 2
// pairs.  K <= KM classes are live.
template <int KM>
__device__ __forceinline__ void sweep_gap(uint64_t* u, uint64_t* q, const int32_t* c, uint64_t gap,
                                          uint32_t K) {
  uint32_t cc[KM];
  bool small = (gap >> 32) == 0;
#pragma unroll
  for (int x = 0; x < KM; ++x) {
    cc[x] = c[x] > 0 ? (uint32_t)c[x] : 0u;
    small = small && cc[x] < 65536u;
  }
  if (small) {
    // gap < 2^32 and counts < 2^16: each term is one 32 x 32 -> 64-bit
    // multiply-add (pair products and pair counts fit 32 bits)
    const uint32_t g32 = (uint32_t)gap;
#pragma unroll
    for (int x = 0; x < KM; ++x) {
#pragma unroll
      for (int y = x; y < KM; ++y) {
        if ((uint32_t)y >= K) continue;
        const int pi = pair_index<KM>(x, y);
        u[pi] += (cc[x] && cc[y]) ? (uint64_t)g32 : 0ull;
        const uint32_t w = x != y ? __umul24(cc[x], cc[y])
                                  : __umul24(cc[x], cc[x] - (cc[x] > 0)) >> 1;
        q[pi] += (uint64_t)g32 * w;
      }
    }
  } else {
    uint64_t gx[KM];
#pragma unroll
    for (int x = 0; x < KM; ++x) gx[x] = mul64x32(gap, cc[x]);
#pragma unroll
    for (int x = 0; x < KM; ++x) {
#pragma unroll
      for (int y = x; y < KM; ++y) {
        if ((uint32_t)y >= K) continue;
        const int pi = pair_index<KM>(x, y);
        if (cc[x] && cc[y]) u[pi] += gap;
        if (x != y) {
          q[pi] += mul64x32(gx[x], cc[y]);
        } else if (cc[x] > 1) {
          const uint64_t pairs = (uint64_t)cc[x] * (cc[x] - 1) / 2;
          q[pi] += gap * pairs;
        }
      }
    }
  }
}

}  // namespace argus
