// k_resolve.hip -- stack pairs that cross tile boundaries.
//
// After k_match, each tile t has summarised what it could not resolve:
//   * pops: ENDs that close levels [lo_head, s_in) open when t started;
//   * pushes: BEGINs at levels [lo_tail, s_out) still open when t ends;
//   * references to enclosing instances at levels [op_lo, s_in) (parents of
//     BEGINs opened in t, and what their children closed in t take off their
//     exclusive time).
// With key(t) = -1 if t holds a context start, else the lowest depth seen in
// t, the END closing a push at level L of tile t is the pop at level L of the
// first later tile with key <= L (if that tile continues the context and
// pops L; otherwise the BEGIN is unclosed), and the instance open at level L
// when tile t starts is the push at level L of the last earlier tile with
// key <= L.  Both searches run on a min-tree over the tile keys.
#include "internal.h"

namespace argus {

constexpr int64_t kInf = 0x7FFFFFFFFFFFFFFFll;

// ------------------------------------------------------------ tile tree

struct TreeArgs {
  const DevPlan* plan;
  const TileDesc* tiles;
  int64_t* tree;
  uint64_t leaves;
};

// Leaves and the bottom levels (subtrees of up to 1024 leaves per block).
__global__ __launch_bounds__(256) void k_tree_lo(TreeArgs a) {
  __shared__ int64_t s[2048];
  const uint64_t ntiles = a.plan->match_tiles;
  const uint64_t sub = a.leaves < 1024 ? a.leaves : 1024;
  const uint64_t first = (uint64_t)blockIdx.x * sub;
  for (uint64_t i = threadIdx.x; i < sub; i += 256) {
    const uint64_t t = first + i;
    const int64_t v = t < ntiles ? a.tiles[t].key : kInf;
    s[sub + i] = v;
    a.tree[a.leaves + t] = v;
  }
  __syncthreads();
  // A heap over this block's `sub` leaves in LDS (node j has children 2j and
  // 2j + 1; leaves at sub..2sub-1).  Its level of `width` nodes is part of the
  // global level of width * gridDim.x nodes, at this block's offset.
  for (uint64_t width = sub / 2; width >= 1; width >>= 1) {
    for (uint64_t k = threadIdx.x; k < width; k += 256) {
      const uint64_t node = width + k;
      const int64_t l = s[2 * node], r = s[2 * node + 1];
      const int64_t m = l < r ? l : r;
      s[node] = m;
      const uint64_t gwidth = width * gridDim.x;
      a.tree[gwidth + (uint64_t)blockIdx.x * width + k] = m;
    }
    __syncthreads();
    if (width == 1) break;
  }
}

// Upper levels above the per-block subtrees (one block).
__global__ __launch_bounds__(1024) void k_tree_hi(TreeArgs a, uint64_t roots) {
  for (uint64_t width = roots / 2; width >= 1; width >>= 1) {
    for (uint64_t k = threadIdx.x; k < width; k += 1024) {
      const uint64_t node = width + k;
      const int64_t l = a.tree[2 * node], r = a.tree[2 * node + 1];
      a.tree[node] = l < r ? l : r;
    }
    __syncthreads();
    if (width == 1) break;
  }
}

hipError_t launch_tree(const RunArgs& a, hipStream_t s) {
  TreeArgs ta{a.w.plan, a.w.tiles, a.w.tree, a.w.tree_leaves};
  const uint64_t sub = a.w.tree_leaves < 1024 ? a.w.tree_leaves : 1024;
  const uint64_t blocks = a.w.tree_leaves / sub;
  hipLaunchKernelGGL(k_tree_lo, dim3((uint32_t)blocks), dim3(256), 0, s, ta);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || blocks == 1) return e;
  hipLaunchKernelGGL(k_tree_hi, dim3(1), dim3(1024), 0, s, ta, blocks);
  return hipGetLastError();
}

// ------------------------------------------------------------- searches

// First tile index > t with key <= v, or -1.
__device__ __forceinline__ int64_t first_le(const int64_t* tree, uint64_t leaves, uint64_t t,
                                            int64_t v) {
  uint64_t node = t + leaves;
  while (node > 1) {
    if (!(node & 1) && tree[node + 1] <= v) {
      node = node + 1;
      while (node < leaves) node = (tree[2 * node] <= v) ? 2 * node : 2 * node + 1;
      return (int64_t)(node - leaves);
    }
    node >>= 1;
  }
  return -1;
}

// Last tile index < t with key <= v, or -1.
__device__ __forceinline__ int64_t last_le(const int64_t* tree, uint64_t leaves, uint64_t t,
                                           int64_t v) {
  uint64_t node = t + leaves;
  while (node > 1) {
    if ((node & 1) && tree[node - 1] <= v) {
      node = node - 1;
      while (node < leaves) node = (tree[2 * node + 1] <= v) ? 2 * node + 1 : 2 * node;
      return (int64_t)(node - leaves);
    }
    node >>= 1;
  }
  return -1;
}

struct ResolveArgs {
  const DevPlan* plan;
  const TileDesc* tiles;
  const int64_t* tree;
  uint64_t leaves;
  const uint64_t* pop_ts;
  const uint32_t* pop_reg;
  const uint32_t* pushes;
  uint32_t* op_parent;
  const uint64_t* op_sum;
  argus_instance* inst;
  uint64_t* excl;  // exclusive time of each instance, accumulated in place
  uint64_t* counters;
  // overlap events of pairs matched across tiles (merge path)
  uint64_t* ev[2];
  const uint32_t* push_pos;
  const uint32_t* pop_pos;
  const uint8_t* region_class;
  uint32_t K, G, shift;
};

// Instance open at level L when tile t starts.  (Such a tile always exists
// for the levels k_match refers to; the checks only keep every access in
// bounds.)
__device__ __forceinline__ uint32_t enclosing(const ResolveArgs& a, uint64_t t, uint32_t L) {
  const int64_t tp = last_le(a.tree, a.leaves, t, (int64_t)L);
  if (tp < 0) return kNoParent;
  const TileDesc d = a.tiles[tp];
  if (L < d.lo_tail || L - d.lo_tail >= d.n_push) return kNoParent;
  return a.pushes[(uint64_t)tp * kMatchTile + (L - d.lo_tail)];
}

// Eight lanes per tile (a tile has a few open levels at either end), so
// that a wave keeps eight tiles' dependent loads in flight.
constexpr uint32_t kResolveLanes = 8;
__global__ __launch_bounds__(256) void k_resolve(ResolveArgs a) {
  const uint64_t t = (uint64_t)blockIdx.x * (256 / kResolveLanes) + (threadIdx.x / kResolveLanes);
  const uint32_t lane = threadIdx.x % kResolveLanes;
  if (t >= a.plan->match_tiles) return;
  const TileDesc d = a.tiles[t];
  const uint64_t pool = t * kMatchTile;
  const uint64_t nb = a.plan->n_begin;
  const uint64_t nv = a.plan->n_valid;
  const KeySpace ks = a.plan->rec;
  const uint32_t g_bits = a.G > 1 ? bit_width64(a.G - 1) : 0u;
  const bool ev_on = a.K > 0 && ks.ts_bits + g_bits + kEvCodeBits <= 64;
  const uint32_t es = ks.ts_bits + kEvCodeBits;
  uint64_t* evo = a.ev[a.plan->rec_final ^ 1u];
  // BEGINs still open at the end of tile t.
  for (uint32_t i = lane; i < d.n_push; i += kResolveLanes) {
    const uint32_t L = d.lo_tail + i;
    const uint32_t id = a.pushes[pool + i];
    if (id >= nb) {
      flag_internal_error(a.counters, 64);
      continue;
    }
    // the instance's own fields, in flight during the tree walk
    argus_instance* x = a.inst + id;
    const uint64_t t_begin = x->t_begin;
    const uint32_t xreg = x->region_id, xctx = x->ctx_key, xpar = x->parent;
    const int64_t t2 = first_le(a.tree, a.leaves, t, (int64_t)L);
    if (t2 < 0) continue;  // context ends with the data: unclosed
    const TileDesc d2 = a.tiles[t2];
    // bitwise: both bounds loaded together
    if ((L < d2.lo_head) | (L - d2.lo_head >= d2.n_pop)) continue;  // context ended: unclosed
    const uint64_t q = (uint64_t)t2 * kMatchTile + (L - d2.lo_head);
    const uint64_t t_end = a.pop_ts[q];
    const uint32_t ereg = a.pop_reg[q];
    x->t_end = t_end;
    x->end_region_id = (uint16_t)ereg;
    const uint64_t incl = t_end - t_begin;
    if (ev_on && ereg == xreg) {
      // both events of a classified instance of a group < G
      const uint32_t cls = a.region_class[ereg];
      const uint64_t g = a.shift >= 32 ? 0u : (xctx >> a.shift);
      const uint32_t pb = a.push_pos[pool + i], pe = a.pop_pos[q];
      if (cls < a.K && g < a.G) {
        if (pb < nv && pe < nv) {
          const uint64_t hi = es < 64 ? (g << es) : 0ull;
          evo[pb] = hi | ((t_begin - ks.ts_min) << kEvCodeBits) | (1u + 2u * cls);
          evo[pe] = hi | ((t_end - ks.ts_min) << kEvCodeBits) | (2u + 2u * cls);
        } else {
          flag_internal_error(a.counters, 64);
        }
      }
    }
    // exclusive times in place: its duration in, and out of its parent's
    atomicAdd((unsigned long long*)&a.excl[id], (unsigned long long)incl);
    uint32_t pf = xpar;
    if (pf == kNoParent) continue;
    if (pf & kParentPending) pf = L >= 1 ? enclosing(a, t, L - 1) : kNoParent;
    if (pf == kNoParent || pf >= nb) continue;
    atomicAdd((unsigned long long*)&a.excl[pf], (unsigned long long)(0ull - incl));
  }
  // Instances open when tile t starts that tile t refers to.
  for (uint32_t i = lane; i < d.n_op; i += kResolveLanes) {
    const uint32_t L = d.op_lo + i;
    const uint32_t pid = enclosing(a, t, L);
    a.op_parent[pool + i] = pid;
    const uint64_t sum = a.op_sum[pool + i];
    if (sum && pid < nb) atomicAdd((unsigned long long*)&a.excl[pid], (unsigned long long)sum);
  }
}

hipError_t launch_resolve(const RunArgs& a, hipStream_t s) {
  ResolveArgs r{a.w.plan, a.w.tiles, a.w.tree, a.w.tree_leaves, a.w.pop_ts, a.w.pop_reg,
                a.w.pushes, a.w.op_parent, a.w.op_sum, a.w.inst, a.w.excl,
                a.out.d_counters};
  for (int b = 0; b < 2; ++b) r.ev[b] = a.w.key[b];
  r.push_pos = a.w.push_pos;
  r.pop_pos = a.w.pop_pos;
  r.region_class = a.region_class;
  r.K = a.K;
  r.G = a.G;
  r.shift = a.shift;
  const uint64_t blocks = ceil_div(a.w.match_tiles, 256 / kResolveLanes);
  hipLaunchKernelGGL(k_resolve, dim3((uint32_t)blocks), dim3(256), 0, s, r);
  return hipGetLastError();
}

}  // namespace argus
