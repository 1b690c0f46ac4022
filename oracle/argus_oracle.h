/*
 * argus_oracle.h -- CPU reference ("oracle") for region attribution over
 * begin/end marker traces.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that tests, the smoke
 * check and the benchmark's CPU-baseline leg can check the GPU library
 * against a plain, slow, single-threaded implementation of the same
 * definitions.  The product path never links, loads or calls it, and it
 * shares no header, helper, table or kernel with the GPU library.
 *
 * What it computes follows the paper's Section 3.2 (BEGIN and END markers
 * bound a region; pairing them per context gives intervals labelled with
 * their region; the open regions of a context form a stack whose top is the
 * innermost one), Section 3.3 (durations come from a traced reference
 * region), Section 3.5 (the fields a report holds, and how it shows that an
 * attribution is ambiguous) and Section 4.3 (compute/communication overlap).  Where the
 * paper is silent the readings are the ones listed with each function in
 * argus_oracle.cpp.
 *
 * Byte layouts (little-endian):
 *   record   (16 B): u64 ts @0, u32 ctx_key @8, u16 region_id @12,
 *                    u8 kind @14 (1 = BEGIN, 2 = END), u8 pad @15.
 *   instance (32 B): u64 t_begin @0, u64 t_end @8, u32 ctx_key @16,
 *                    u32 parent @20, u32 level @24, u16 region_id @28,
 *                    u16 end_region_id @30.
 */
#ifndef ARGUS_ORACLE_H
#define ARGUS_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Indices into the counters array. */
enum {
  ORC_N_RECORDS = 0,
  ORC_N_VALID = 1,
  ORC_N_BAD_KIND = 2,
  ORC_N_BAD_REGION = 3,
  ORC_N_BEGIN = 4,
  ORC_N_END = 5,
  ORC_TS_MIN = 6,
  ORC_TS_MAX = 7,
  ORC_N_CTX = 8,
  ORC_N_MATCHED = 9,
  ORC_N_MISMATCHED = 10,
  ORC_N_UNCLOSED = 11,
  ORC_N_ORPHAN_END = 12,
  ORC_N_SELF_NESTED = 13,
  ORC_MAX_LEVEL = 14,
  ORC_N_OVERLAP_SKIPPED = 15,
  ORC_CTX_MIN = 16,
  ORC_CTX_MAX = 17,
  ORC_NUM_COUNTERS = 32 /* 18..31 are always zero */
};

/* Columns of one row of the per-region statistics ([num_regions][142]). */
enum {
  ORC_RS_COUNT = 0,
  ORC_RS_INCL_SUM = 1,
  ORC_RS_EXCL_SUM = 2,
  ORC_RS_INCL_MIN = 3,
  ORC_RS_INCL_MAX = 4,
  ORC_RS_EXCL_MIN = 5,
  ORC_RS_EXCL_MAX = 6,
  ORC_RS_UNCLOSED = 7,
  ORC_RS_ORPHAN_END = 8,
  ORC_RS_MISM_AS_BEGIN = 9,
  ORC_RS_MISM_AS_END = 10,
  ORC_RS_SELF_NESTED = 11,
  ORC_RS_HIST_INCL = 12, /* 65 bins */
  ORC_RS_HIST_EXCL = 77, /* 65 bins */
  ORC_RS_WIDTH = 142
};

/*
 * Runs the whole definition on host memory.
 *   records        n records (16 B each).
 *   num_regions    R, 1..65535; region_id >= R makes a record invalid.
 *   num_classes    K, 0..8; 0 disables overlap.
 *   region_class   [R] class of each region (>= K means unclassified);
 *                  may be NULL when K == 0.
 *   group_shift    group = ctx_key >> group_shift (0..32; 32 puts every
 *                  context in group 0).
 *   num_groups     G; contexts whose group is >= G are left out of overlap.
 *   counters       [ORC_NUM_COUNTERS]
 *   region_stats   [R * ORC_RS_WIDTH]
 *   overlap_group  [G * 2 * K * K] (U matrix then Q matrix per group) or NULL
 *   overlap_global [2 * K * K] or NULL
 *   instances      [inst_cap] 32-byte instances or NULL
 *   instance_excl  [inst_cap] or NULL
 * Returns 0, -1 for bad arguments, -2 if n_begin exceeds inst_cap while an
 * instance output was requested.
 */
int argus_oracle_run(const void* records, uint64_t n, uint32_t num_regions,
                     uint32_t num_classes, const uint8_t* region_class,
                     uint32_t group_shift, uint32_t num_groups,
                     uint64_t* counters, uint64_t* region_stats,
                     uint64_t* overlap_group, uint64_t* overlap_global,
                     void* instances, uint64_t* instance_excl,
                     uint64_t inst_cap);

/* ------------------------------------------------------------------------
 * PC-sample attribution (Section 3.2: the innermost active region of the
 * executing warp receives each execution count; Section 3.5: count-weighted
 * lifting of PC-keyed metrics into regions, with association entropy as
 * ambiguity metadata).
 *
 *   sample (16 B): u64 ts @0, u32 ctx_key @8, u32 pc @12.
 *
 *   instances      n_inst instances in canonical order (as argus_oracle_run
 *                  writes them).
 *   samples        n_samples samples; weights [n_samples] executions per
 *                  sample, or NULL for 1 each.
 *   num_regions    R; num_pcs P (a sample with pc >= P is counted as bad and
 *                  takes no further part); num_metrics M; metrics [M * P]
 *                  (metric k of pc p at k * P + p), may be NULL iff M == 0.
 * Outputs (all required except alpha and mhat when M == 0):
 *   counters       [ORC_S_NUM_COUNTERS]
 *   n_rp           [P * R]  n(r, p) at p * R + r
 *   alpha          [P * R]  alpha(r, p) = n(r, p) / T(p), 0 where n == 0; or NULL
 *   pc_total       [P]      T(p) = sum over r of n(r, p)
 *   pc_owners      [P]      regions r with n(r, p) > 0
 *   entropy        [P]      H(p) = -sum over r with n > 0 of alpha log alpha
 *                           (natural log; 0 when T(p) == 0)
 *   region_total   [R]      sum over p of n(r, p)
 *   mhat           [M * R]  sum over p with n(r, p) > 0 of alpha(r, p) m(p),
 *                           in 512 strands (p mod 512, each in increasing
 *                           p) combined by halving; or NULL when M == 0
 * Returns 0, or -1 for bad arguments. */
enum {
  ORC_S_N_SAMPLES = 0,       /* sample records */
  ORC_S_N_BAD_PC = 1,        /* samples with pc >= P */
  ORC_S_W_TOTAL = 2,         /* weight of the samples with a valid pc */
  ORC_S_W_ATTRIBUTED = 3,    /* weight given to a matched instance */
  ORC_S_W_UNATTRIBUTED = 4,  /* weight with no matched active instance */
  ORC_S_W_INNER_UNMATCHED = 5, /* attributed weight whose innermost active
                                  instance was mismatched or unclosed */
  ORC_S_N_PAIRS = 6,         /* (r, p) with n(r, p) > 0 */
  ORC_S_NUM_COUNTERS = 8
};

int argus_oracle_samples(const void* instances, uint64_t n_inst,
                         const void* samples, uint64_t n_samples,
                         const uint32_t* weights, uint32_t num_regions,
                         uint32_t num_pcs, uint32_t num_metrics,
                         const double* metrics, uint64_t* counters,
                         uint64_t* n_rp, double* alpha, uint64_t* pc_total,
                         uint32_t* pc_owners, double* entropy,
                         uint64_t* region_total, double* mhat);

/* ------------------------------------------------------------------------
 * Scopes and iteration ordinals (Section 3.2: a scope selects dynamic
 * executions of a region -- by warp role, iteration window or SM subset;
 * Section 3.3: probes are specialised per iteration).
 *
 * ordinal[x] = number of instances y < x (canonical order) of the same
 * context whose BEGIN region equals x's: the 0-based iteration of region
 * x in its context.  Instance x is in scope when
 *   (ctx & role_mask) in [role_lo, role_hi],
 *   (ctx >> group_shift, 0 if group_shift >= 32) in [group_lo, group_hi],
 *   ordinal[x] in [iter_lo, iter_hi], and
 *   region_mask == NULL or region_mask[region] != 0.
 * stats [R * ORC_RS_WIDTH]: the per-region statistics of argus_oracle_run
 * over the in-scope instances only (orphan_end stays 0: orphans are no
 * instances; mism_as_end is counted by the END region of an in-scope
 * mismatched instance; self_nested when the parent, in scope or not, has
 * the same region).
 * counters [ORC_SC_NUM_COUNTERS].  excl [n_inst] exclusive durations. */
typedef struct {
  uint32_t role_mask, role_lo, role_hi;
  uint32_t group_shift, group_lo, group_hi;
  uint32_t iter_lo, iter_hi;
} orc_scope;

enum {
  ORC_SC_N_INSTANCES = 0,
  ORC_SC_N_IN_SCOPE = 1,
  ORC_SC_N_MATCHED = 2,
  ORC_SC_N_MISMATCHED = 3,
  ORC_SC_N_UNCLOSED = 4,
  ORC_SC_N_SELF_NESTED = 5,
  ORC_SC_N_ITERATIONS = 6, /* 1 + the largest ordinal (0 without instances) */
  ORC_SC_NUM_COUNTERS = 8
};

int argus_oracle_scope(const void* instances, const uint64_t* excl, uint64_t n_inst,
                       uint32_t num_regions, const orc_scope* scope,
                       const uint8_t* region_mask, uint32_t* ordinal,
                       uint64_t* stats, uint64_t* counters);

/* ------------------------------------------------------------------------
 * Probe <-> reference join (Section 3.3: a forced-completion probe measures
 * the exposed latency of one asynchronous operation at one iteration; the
 * interval is joined to the same operation in the same iteration of the
 * reference trace through stable identity and scope, never by timestamp;
 * Section 3.5: exact joins by scope coordinates; Appendix B: mean and the
 * 0/20/40/60/80th percentiles of the exposed latency).
 *
 *   probe (32 B): u64 t_start @0, u64 t_end @8, u32 ctx_key @16,
 *                 u32 iteration @20, u16 op_region @24, u16 pad, u32 pad.
 *
 * A probe is bad when t_end < t_start or op_region >= R.  Otherwise it joins
 * the reference instance of its context with BEGIN region op_region whose
 * iteration ordinal (see argus_oracle_scope) equals its iteration; no such
 * instance: unjoined.  Latency = t_end - t_start.
 * Per probe: ref [n_probes] (instance index or 0xFFFFFFFF) and completion
 * [n_probes] = t_begin of the reference instance + latency (UINT64_MAX if
 * not joined).
 * Groups: one per reference instance with joined probes, in increasing
 * instance index; group columns [ORC_PG_WIDTH] u64 each: instance, count,
 * latency sum, t_issue (the instance's t_begin), p0 (min), p20, p40, p60,
 * p80, p100 (max), where p_q is the k-th smallest latency with
 * k = max(1, ceil(q * count / 100)); mean [groups] = (double)sum /
 * (double)count.
 * counters [ORC_PR_NUM_COUNTERS].  Returns 0, -1 bad arguments, -2 if the
 * groups exceed group_cap. */
enum {
  ORC_PG_INSTANCE = 0, ORC_PG_COUNT = 1, ORC_PG_SUM = 2, ORC_PG_ISSUE = 3, ORC_PG_P0 = 4,
  ORC_PG_P20 = 5, ORC_PG_P40 = 6, ORC_PG_P60 = 7, ORC_PG_P80 = 8, ORC_PG_P100 = 9,
  ORC_PG_WIDTH = 10
};
enum {
  ORC_PR_N_PROBES = 0, ORC_PR_N_BAD = 1, ORC_PR_N_JOINED = 2, ORC_PR_N_UNJOINED = 3,
  ORC_PR_N_GROUPS = 4, ORC_PR_NUM_COUNTERS = 8
};

int argus_oracle_probes(const void* instances, uint64_t n_inst, uint32_t num_regions,
                        const void* probes, uint64_t n_probes, uint32_t* ref,
                        uint64_t* completion, uint64_t* groups, double* mean,
                        uint64_t group_cap, uint64_t* counters);

/* ------------------------------------------------------------------------
 * Phase handoffs (Section 4.2: in a persistent kernel the time spent in the
 * intervals between successive cooperative phases is a measured quantity
 * of its own; Section 2 names a phase handoff as a region a developer can
 * change).
 *
 * At level L, two instances x and y of one context are successive phases
 * when y is the next instance after x with the same parent and level L
 * (for L = 0: the next top-level instance of the context).  For closed x:
 * gap = t_begin(y) - t_end(x) (an unclosed x has no successor: everything
 * after it in its context is nested inside it).
 *   pairs [R * R * 4]: for (region(x), region(y)) count, gap sum (mod 2^64),
 *                      min (UINT64_MAX if none), max
 *   hist [65]: gaps by bit width
 *   parent_gap [n_inst] or NULL: per parent instance, the sum of the gaps
 *                      between its successive level-L children (L >= 1)
 *   counters [ORC_PH_NUM_COUNTERS] */
enum {
  ORC_PH_N_AT_LEVEL = 0, ORC_PH_N_GAPS = 1, ORC_PH_GAP_SUM = 2, ORC_PH_NUM_COUNTERS = 8
};

int argus_oracle_handoffs(const void* instances, uint64_t n_inst, uint32_t num_regions,
                          uint32_t level, uint64_t* pairs, uint64_t* hist, uint64_t* parent_gap,
                          uint64_t* counters);

#ifdef __cplusplus
}
#endif

#endif
