/*
 * argus_attr.h -- region attribution over begin/end marker traces on one
 * MI355X (gfx950) GPU.  C ABI, version 1, little-endian.
 *
 * What the library computes.  It follows the paper's Section 3.2 (regions
 * are named by their begin and end markers; a time-ordered trace of those
 * markers yields the intervals of each region; one stack of open regions per
 * warp decides which region is innermost at any moment), Section 3.3 (a
 * region's duration comes from its marker trace), Section 3.5 (directly
 * observed fields, with ambiguity reported rather than hidden) and Section
 * 4.3 (overlap of compute and communication regions):
 *
 *   1. Validate each record: kind must be BEGIN (1) or END (2) (else
 *      "bad kind"), then region_id must be < num_regions (else "bad region").
 *      Invalid records take no further part.
 *   2. Order the valid records by (ctx_key, ts, input index).
 *   3. Per execution context, replay a nested stack: a BEGIN opens an
 *      instance (numbered by its position in that order, level = stack
 *      depth, parent = the instance on top of the stack); an END closes the
 *      instance on top of the stack whatever its region (MATCHED when the
 *      regions agree, MISMATCHED otherwise); an END on an empty stack is an
 *      orphan; instances still open when the context ends are UNCLOSED.
 *   4. Exclusive duration of a closed instance = its inclusive duration
 *      (t_end - t_begin) minus the inclusive durations of its closed direct
 *      children.  Unclosed instances have exclusive duration 0.
 *   5. Per region, over MATCHED instances: count, sums, min/max of inclusive
 *      and exclusive duration, and 65-bin log2 histograms (bin = bit width of
 *      the duration: 0 for 0, floor(log2 d) + 1 otherwise); plus ambiguity
 *      counts: unclosed, orphan END, mismatched (by begin and by end region)
 *      and self-nested (matched instance whose parent has the same region).
 *   6. If num_classes > 0: per group (ctx_key >> group_shift, groups below
 *      num_groups), over MATCHED instances whose region has a class below
 *      num_classes, with half-open intervals [t_begin, t_end):
 *      U[A][B] = time during which some class-A and some class-B instance
 *      are active; Q[A][B] = sum over pairs of distinct instances (one of
 *      class A, one of class B; unordered pairs for A == B) of their
 *      intersection length.  The global matrices are sums over groups.
 *
 * All results are exact integers; sums wrap modulo 2^64.
 */
#ifndef ARGUS_ATTR_H
#define ARGUS_ATTR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ARGUS_ATTR_ABI_VERSION 1u

/* ---------------------------------------------------------------- records */
enum { ARGUS_KIND_BEGIN = 1, ARGUS_KIND_END = 2 };

/* One marker record, 16 bytes, 16-byte aligned in device memory.  `pad` is
 * ignored. */
typedef struct argus_record {
  uint64_t ts;        /* timestamp in cycles of the context's clock */
  uint32_t ctx_key;   /* execution context (e.g. block * warps + warp) */
  uint16_t region_id; /* stable region id, < num_regions */
  uint8_t kind;       /* ARGUS_KIND_BEGIN or ARGUS_KIND_END */
  uint8_t pad;
} argus_record;

/* One region instance, 32 bytes.  Instances are numbered by the position of
 * their BEGIN in (ctx_key, ts, input index) order. */
typedef struct argus_instance {
  uint64_t t_begin;
  uint64_t t_end;         /* UINT64_MAX if UNCLOSED */
  uint32_t ctx_key;
  uint32_t parent;        /* instance index of the parent, ARGUS_NO_PARENT */
  uint32_t level;         /* stack depth at the BEGIN; 0 = top level */
  uint16_t region_id;     /* region of the BEGIN */
  uint16_t end_region_id; /* region of the closing END; ARGUS_UNCLOSED if none.
                             MISMATCHED iff != region_id (and not UNCLOSED) */
} argus_instance;

#define ARGUS_NO_PARENT 0xFFFFFFFFu
#define ARGUS_UNCLOSED 0xFFFFu

/* ------------------------------------------------------ counters (u64 each) */
enum {
  ARGUS_C_N_RECORDS = 0,
  ARGUS_C_N_VALID = 1,
  ARGUS_C_N_BAD_KIND = 2,
  ARGUS_C_N_BAD_REGION = 3,
  ARGUS_C_N_BEGIN = 4,
  ARGUS_C_N_END = 5,
  ARGUS_C_TS_MIN = 6,          /* over valid records; UINT64_MAX if none */
  ARGUS_C_TS_MAX = 7,          /* 0 if none */
  ARGUS_C_N_CTX = 8,           /* distinct ctx_key among valid records */
  ARGUS_C_N_MATCHED = 9,
  ARGUS_C_N_MISMATCHED = 10,
  ARGUS_C_N_UNCLOSED = 11,
  ARGUS_C_N_ORPHAN_END = 12,
  ARGUS_C_N_SELF_NESTED = 13,
  ARGUS_C_MAX_LEVEL = 14,      /* max level over BEGINs; 0 if none */
  ARGUS_C_N_OVERLAP_SKIPPED = 15, /* matched classified, group >= num_groups */
  ARGUS_C_CTX_MIN = 16,        /* UINT64_MAX if none */
  ARGUS_C_CTX_MAX = 17,
  ARGUS_C_INTERNAL_ERROR = 31, /* 0; nonzero only if the library detected an
                                  internal inconsistency (a bug) */
  ARGUS_NUM_COUNTERS = 32      /* 18..30 are zero */
};

/* ------------------------------------- per-region statistics, u64 [R][142] */
enum {
  ARGUS_RS_COUNT = 0,      /* matched instances */
  ARGUS_RS_INCL_SUM = 1,
  ARGUS_RS_EXCL_SUM = 2,
  ARGUS_RS_INCL_MIN = 3,   /* UINT64_MAX when count == 0 */
  ARGUS_RS_INCL_MAX = 4,
  ARGUS_RS_EXCL_MIN = 5,   /* UINT64_MAX when count == 0 */
  ARGUS_RS_EXCL_MAX = 6,
  ARGUS_RS_UNCLOSED = 7,
  ARGUS_RS_ORPHAN_END = 8,
  ARGUS_RS_MISM_AS_BEGIN = 9,
  ARGUS_RS_MISM_AS_END = 10,
  ARGUS_RS_SELF_NESTED = 11,
  ARGUS_RS_HIST_INCL = 12, /* 65 bins */
  ARGUS_RS_HIST_EXCL = 77, /* 65 bins */
  ARGUS_RS_WIDTH = 142
};

/* ------------------------------------------------------------------ config */
enum {
  ARGUS_OUT_INSTANCES = 1u,     /* write out->d_instances */
  ARGUS_OUT_INSTANCE_EXCL = 2u, /* write out->d_instance_excl */
  ARGUS_FORCE_FULL_SORT = 4u,   /* always sort on every timestamp digit, even
                                   when each context is already in time order
                                   in the input (results are identical; for
                                   measurement and testing) */
  ARGUS_FORCE_EVENT_SORT = 8u,  /* order the overlap events with a radix sort
                                   of (group, time) even where merging the
                                   per-context runs applies (results are
                                   identical; for measurement and testing) */
  ARGUS_FORCE_RECORD_RADIX = 16u /* sort the records by context with radix
                                   passes over every record even where the
                                   input holds long runs of one context, which
                                   are otherwise sorted as runs (results are
                                   identical; for measurement and testing) */
};

typedef struct argus_attr_config {
  uint32_t abi_version;   /* must equal ARGUS_ATTR_ABI_VERSION */
  uint32_t num_regions;   /* R: 1..65535 */
  uint32_t num_classes;   /* K: 0..8; 0 disables the overlap step */
  uint32_t group_shift;   /* group = ctx_key >> group_shift; 0..32 (32: one group) */
  uint32_t num_groups;    /* G: rows of the per-group overlap output; 1..2^20 if K > 0 */
  uint32_t flags;         /* ARGUS_OUT_* / ARGUS_FORCE_* */
  uint64_t max_records;   /* capacity this handle is planned for, < 2^31 */
  const uint8_t* d_region_class; /* device [R]; class of each region, >= K means
                                    unclassified; caller-owned; may be NULL iff K == 0 */
} argus_attr_config;

/* Output buffers, all device memory, all caller-owned.  `run` initialises
 * every one of them. */
typedef struct argus_attr_outputs {
  uint64_t* d_counters;        /* [ARGUS_NUM_COUNTERS] */
  uint64_t* d_region_stats;    /* [R][ARGUS_RS_WIDTH] */
  uint64_t* d_overlap_group;   /* [G][2][K][K]: U then Q; required iff K > 0 */
  uint64_t* d_overlap_global;  /* [2][K][K]; required iff K > 0 */
  argus_instance* d_instances; /* [n_begin <= n_records]; required iff flag 1 */
  uint64_t* d_instance_excl;   /* [n_begin]; required iff flag 2 */
} argus_attr_outputs;

/* ------------------------------------------------------------ error codes */
enum {
  ARGUS_OK = 0,
  ARGUS_E_INVAL = -1,    /* NULL pointer, bad R/K/G/shift, missing buffer */
  ARGUS_E_ABI = -2,      /* abi_version mismatch */
  ARGUS_E_ALIGN = -3,    /* records not 16-B aligned or workspace not 256-B aligned */
  ARGUS_E_CAPACITY = -4, /* n_records > max_records, or workspace too small */
  ARGUS_E_DEVICE = -5,   /* current device is not gfx950 */
  ARGUS_E_HIP = -6,      /* a HIP call failed; see argus_attr_last_error */
  ARGUS_E_IO = -7        /* a file could not be written (trace export) */
};

typedef struct argus_attr argus_attr; /* opaque host-side handle */

/* Create a handle from a copy of *cfg.  Checks the configuration only (no
 * GPU call).  On success writes *out and returns ARGUS_OK; on failure *out
 * is set to NULL and a negative code is returned. */
int argus_attr_create(const argus_attr_config* cfg, argus_attr** out);

/* Device workspace `run` needs for n_records records (bytes; callers pass a
 * buffer at least this large, 256-byte aligned).  0 if h is NULL or
 * n_records exceeds the handle's capacity. */
size_t argus_attr_workspace_bytes(const argus_attr* h, uint64_t n_records);

/* Enqueue the whole computation on `stream` (a hipStream_t; NULL = the
 * default stream) and return without synchronising.  `d_records` points to
 * n_records device records (16-byte aligned, caller-owned, not modified).
 * The library allocates no memory and makes no host<->device copies; every
 * output is initialised on the stream.  Results are valid once the stream
 * has completed.  Argument errors are reported before any GPU call.  Data
 * anomalies never fail the call: they are counted.  A handle must not run
 * on two streams at once; distinct handles are independent. */
int argus_attr_run(argus_attr* h, const argus_record* d_records, uint64_t n_records,
                   void* d_workspace, size_t workspace_bytes,
                   const argus_attr_outputs* out, void* stream);

/* ------------------------------------------------ allocation-free variant */
/* Size of the library's built-in workspace: one array of this many bytes per
 * GPU the library runs on, held until the process ends. */
#define ARGUS_NOALLOC_SCRATCH_BYTES (64u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * computation as argus_attr_run, with the same arguments except the
 * workspace, which is the library's built-in array on the current device
 * instead.  It calls no allocating routine.  Outputs and records are the
 * caller's, as for argus_attr_run.
 *
 * Limit: returns ARGUS_E_CAPACITY (before any GPU call, with a message in
 * argus_attr_last_error) when argus_attr_workspace_bytes(h, n_records)
 * exceeds ARGUS_NOALLOC_SCRATCH_BYTES -- for example about 2^19 records with
 * num_classes == 0, or 2^16 records with 4 classes over 2048 groups.
 * Every call on one GPU uses that GPU's one array, whatever the handle:
 * calls that overlap in time on one GPU (on different streams, or from
 * different threads) race and give undefined results.  Calls in order on
 * one stream are safe; each call initialises what it reads. */
int argus_attr_run_noalloc(argus_attr* h, const argus_record* d_records, uint64_t n_records,
                           const argus_attr_outputs* out, void* stream);

/* ------------------------------------------------ PC-sample attribution */
/* Lifting of PC-keyed measurements into region space (the paper's Section
 * 3.2: a mapping run replays each warp's stack of open regions, and every
 * execution of the instruction at a PC counts for the region innermost at
 * that moment; Section 3.5: count-weighted attribution with association
 * entropy as ambiguity metadata).  Works on the instance array that
 * argus_attr_run wrote.
 *
 * One sample is one or more executions of the instruction with index `pc`
 * (0 <= pc < num_pcs) at time `ts` in context `ctx_key`.  Its owner is the
 * innermost MATCHED instance of that context active at ts (t_begin <= ts <
 * t_end; an unclosed instance is active from t_begin on and never owns).
 * Then, with n(r, p) the executions of p owned by region r and
 * T(p) = sum over r of n(r, p):
 *   alpha(r, p) = n(r, p) / T(p)              (0 where n(r, p) == 0)
 *   H(p)        = - sum over r with n(r, p) > 0 of alpha log alpha  (natural log)
 *   m_hat(r)    = sum over p with n(r, p) > 0 of alpha(r, p) * m(p)
 * in IEEE double: each alpha is one correctly rounded division; m_hat adds
 * the rounded products one at a time in increasing p (so the result is
 * reproducible bit for bit); H is summed in an unspecified order and
 * carries the error of the device logarithm (a few ulp per term). */
typedef struct argus_sample {
  uint64_t ts;      /* cycles of the context's clock, as in the records */
  uint32_t ctx_key;
  uint32_t pc;      /* instruction index, < num_pcs (else counted as bad) */
} argus_sample;     /* 16 bytes, 16-byte aligned */

enum {
  ARGUS_S_N_SAMPLES = 0,         /* sample records */
  ARGUS_S_N_BAD_PC = 1,          /* samples with pc >= num_pcs (no further part) */
  ARGUS_S_W_TOTAL = 2,           /* executions (weights) of the other samples */
  ARGUS_S_W_ATTRIBUTED = 3,      /* executions given to a matched instance */
  ARGUS_S_W_UNATTRIBUTED = 4,    /* executions with no matched active instance */
  ARGUS_S_W_INNER_UNMATCHED = 5, /* attributed executions whose innermost active
                                    instance was mismatched or unclosed */
  ARGUS_S_N_PAIRS = 6,           /* (r, p) with n(r, p) > 0 */
  ARGUS_S_W_BAD_INSTANCE = 7,    /* executions whose owner has region_id >= num_regions
                                    (instances of another configuration); not counted
                                    anywhere else; 0 for instances of a run with this R */
  ARGUS_S_NUM_COUNTERS = 8
};

typedef struct argus_samples_config {
  uint32_t abi_version; /* ARGUS_ATTR_ABI_VERSION */
  uint32_t num_regions; /* R, 1..65535: the R of the run that wrote the instances */
  uint32_t num_pcs;     /* P, 1..2^24, with P * R <= 2^31 */
  uint32_t num_metrics; /* M, 0..64: PC-keyed additive metrics to lift */
} argus_samples_config;

/* All pointers are device memory, caller-owned, 16-byte aligned where they
 * hold 16-byte elements. */
typedef struct argus_samples_io {
  const argus_instance* d_instances; /* canonical order, as argus_attr_run writes it */
  const uint64_t* d_n_instances;     /* device scalar: instances in the array, e.g.
                                        &d_counters[ARGUS_C_N_BEGIN] of that run (read on
                                        the device, so no host synchronisation) */
  uint64_t max_instances;            /* capacity of d_instances; at most this many are read */
  const argus_sample* d_samples;     /* [n_samples] */
  uint64_t n_samples;
  const uint32_t* d_weights;         /* [n_samples] executions per sample; NULL: 1 each */
  const double* d_metrics;           /* [M][P] m(p); may be NULL iff M == 0 */
  uint64_t* d_counters;              /* out [ARGUS_S_NUM_COUNTERS] */
  uint64_t* d_n;                     /* out [P][R] n(r, p) */
  double* d_alpha;                   /* out [P][R] alpha(r, p) */
  uint64_t* d_pc_total;              /* out [P] T(p) */
  uint32_t* d_pc_owners;             /* out [P] regions with n(r, p) > 0 */
  double* d_entropy;                 /* out [P] H(p); 0 when T(p) == 0 */
  uint64_t* d_region_total;          /* out [R] sum over p of n(r, p) */
  double* d_mhat;                    /* out [M][R] m_hat(r); may be NULL iff M == 0 */
} argus_samples_io;

/* Enqueue the attribution on `stream` and return without synchronising;
 * every output is initialised on the stream and valid once it completes.
 * Allocates nothing.  Argument errors (ARGUS_E_INVAL, ARGUS_E_ABI,
 * ARGUS_E_ALIGN, ARGUS_E_CAPACITY) are returned before any GPU call;
 * ARGUS_E_DEVICE if the current device is not gfx950, ARGUS_E_HIP if a
 * launch fails. */
int argus_attr_samples(const argus_samples_config* cfg, const argus_samples_io* io,
                       void* stream);

/* ------------------------------------------ scopes and iteration ordinals */
/* Section 3.2 of the paper separates a region (the code) from its scope:
 * which dynamic executions are reported -- a warp role, an iteration window
 * or a subset of SMs; Section 3.3 specialises probes to one iteration of a
 * loop region.  Works on the instance array (and exclusive durations) that
 * argus_attr_run wrote.
 *
 * ordinal[x] = the number of instances before x (canonical order) of the
 * same context with the same BEGIN region: the 0-based iteration of that
 * region in its context (every status counts).  Instance x is in scope when
 *   (ctx_key & role_mask) in [role_lo, role_hi]            (warp role)
 *   (ctx_key >> group_shift; 0 if group_shift >= 32) in [group_lo, group_hi]
 *                                                          (SM subset)
 *   ordinal[x] in [iter_lo, iter_hi]                       (iteration window)
 *   d_region_mask == NULL or d_region_mask[region_id] != 0 (region set)
 * Scoped statistics use the ARGUS_RS_* layout over the in-scope instances:
 * matched ones give count, sums, min/max and histograms; unclosed and
 * mismatched (by BEGIN region, and by END region for mism_as_end) ones are
 * counted; self_nested when the parent (in scope or not) has the same region;
 * orphan_end is 0 (orphan ENDs are no instances).  All integers. */
typedef struct argus_scope {
  uint32_t role_mask, role_lo, role_hi;
  uint32_t group_shift, group_lo, group_hi;
  uint32_t iter_lo, iter_hi;
} argus_scope; /* everything: {0, 0, 0, 32, 0, 0, 0, 0xFFFFFFFF} */

enum {
  ARGUS_SC_N_INSTANCES = 0,
  ARGUS_SC_N_IN_SCOPE = 1,
  ARGUS_SC_N_MATCHED = 2,
  ARGUS_SC_N_MISMATCHED = 3,
  ARGUS_SC_N_UNCLOSED = 4,
  ARGUS_SC_N_SELF_NESTED = 5,
  ARGUS_SC_N_ITERATIONS = 6, /* 1 + the largest ordinal; 0 without instances */
  ARGUS_SC_INTERNAL = 7,     /* internal-error bits: 0 unless a consistency check in the
                                library fails (2: an instance's region_id >= num_regions) */
  ARGUS_SC_NUM_COUNTERS = 8
};

typedef struct argus_scope_config {
  uint32_t abi_version; /* ARGUS_ATTR_ABI_VERSION */
  uint32_t num_regions; /* R of the run that wrote the instances */
  argus_scope scope;
} argus_scope_config;

typedef struct argus_scope_io {
  const argus_instance* d_instances; /* canonical order (16-byte aligned) */
  const uint64_t* d_instance_excl;   /* exclusive durations, as argus_attr_run writes them */
  const uint64_t* d_n_instances;     /* device scalar, e.g. &d_counters[ARGUS_C_N_BEGIN] */
  uint64_t max_instances;            /* capacity of the instance arrays, < 2^31 */
  const uint8_t* d_region_mask;      /* [R] or NULL */
  uint32_t* d_ordinal;               /* out [max_instances]; the first n are written */
  uint64_t* d_stats;                 /* out [R][ARGUS_RS_WIDTH] */
  uint64_t* d_counters;              /* out [ARGUS_SC_NUM_COUNTERS] */
} argus_scope_io;

/* Device workspace argus_attr_scope needs for up to max_instances instances
 * (256-byte aligned); 0 if max_instances >= 2^31. */
size_t argus_attr_scope_workspace_bytes(uint64_t max_instances);

/* Enqueue ordinals and scoped statistics on `stream` without synchronising.
 * Allocates nothing; argument errors are returned before any GPU call. */
int argus_attr_scope(const argus_scope_config* cfg, const argus_scope_io* io,
                     void* d_workspace, size_t workspace_bytes, void* stream);

/* ----------------------------------------- probe <-> reference exact join */
/* Section 3.3 of the paper: a forced-completion probe measures the exposed
 * latency of one asynchronous operation at one selected iteration (the
 * interval from its issue to its forced completion); that interval is
 * joined to the same operation's issue in the same iteration of the
 * reference trace through the operation's stable id and the dynamic scope,
 * never by comparing timestamps across runs (Section 3.5).  Appendix B
 * reports the mean and the 0th/20th/40th/60th/80th percentiles per
 * operation and iteration.
 *
 * A probe is bad when t_end < t_start or op_region >= num_regions.
 * Otherwise it joins the reference instance of its context whose BEGIN
 * region is op_region and whose iteration ordinal (as argus_attr_scope
 * defines it) equals `iteration`; with no such instance it is unjoined.
 * Latency = t_end - t_start.  Per probe: d_ref = the joined instance index
 * (0xFFFFFFFF if none) and d_completion = that instance's t_begin + latency
 * (UINT64_MAX if none).  One group per reference instance with joined
 * probes, in increasing instance index: ARGUS_PG_* columns, where p_q is the
 * k-th smallest latency with k = max(1, ceil(q * count / 100)) (nearest
 * rank; p0 = minimum, p100 = maximum), and d_mean = (double)sum /
 * (double)count (one correctly rounded division).  All else is integer. */
typedef struct argus_probe {
  uint64_t t_start, t_end; /* the probe run's clock */
  uint32_t ctx_key;
  uint32_t iteration;      /* iteration ordinal of the operation's region */
  uint16_t op_region;      /* region id of the operation in the reference */
  uint16_t pad0;
  uint32_t pad1;
} argus_probe;             /* 32 bytes, 16-byte aligned */

enum {
  ARGUS_PG_INSTANCE = 0, ARGUS_PG_COUNT = 1, ARGUS_PG_SUM = 2, ARGUS_PG_ISSUE = 3,
  ARGUS_PG_P0 = 4, ARGUS_PG_P20 = 5, ARGUS_PG_P40 = 6, ARGUS_PG_P60 = 7, ARGUS_PG_P80 = 8,
  ARGUS_PG_P100 = 9, ARGUS_PG_WIDTH = 10
};
enum {
  ARGUS_PR_N_PROBES = 0, ARGUS_PR_N_BAD = 1, ARGUS_PR_N_JOINED = 2, ARGUS_PR_N_UNJOINED = 3,
  ARGUS_PR_N_GROUPS = 4, ARGUS_PR_NUM_COUNTERS = 8 /* 5..7 are zero */
};

typedef struct argus_probes_config {
  uint32_t abi_version; /* ARGUS_ATTR_ABI_VERSION */
  uint32_t num_regions; /* R of the run that wrote the reference instances */
} argus_probes_config;

typedef struct argus_probes_io {
  const argus_instance* d_instances; /* reference, canonical order (16-byte aligned) */
  const uint64_t* d_n_instances;     /* device scalar, e.g. &d_counters[ARGUS_C_N_BEGIN] */
  uint64_t max_instances;            /* capacity of d_instances, < 2^31 */
  const argus_probe* d_probes;       /* [n_probes] */
  uint64_t n_probes;                 /* < 2^31 */
  uint32_t* d_ref;                   /* out [n_probes] */
  uint64_t* d_completion;            /* out [n_probes] */
  uint64_t* d_groups;                /* out [n_probes][ARGUS_PG_WIDTH]; the first
                                        counters[ARGUS_PR_N_GROUPS] rows are written */
  double* d_mean;                    /* out [n_probes], as many as the groups */
  uint64_t* d_counters;              /* out [ARGUS_PR_NUM_COUNTERS] */
} argus_probes_io;

/* Device workspace argus_attr_probes needs (256-byte aligned); 0 if either
 * size is >= 2^31. */
size_t argus_attr_probes_workspace_bytes(uint64_t max_instances, uint64_t n_probes);

/* Enqueue the join and the per-group summaries on `stream` without
 * synchronising.  Allocates nothing; argument errors are returned before
 * any GPU call. */
int argus_attr_probes(const argus_probes_config* cfg, const argus_probes_io* io,
                      void* d_workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------- phase handoffs */
/* Section 4.2 of the paper measures, on the reference trace of a persistent
 * kernel, the time spent in the intervals between successive cooperative
 * phases.  Here the phases are the instances of one nesting level L: y
 * follows x when y is the next level-L instance after x with the same parent
 * (for L = 0, the next top-level instance of the same context).  For such a
 * pair (x closed): gap = t_begin(y) - t_end(x).  An unclosed x has no
 * successor (what follows it is nested inside it).  Integers throughout. */
enum {
  ARGUS_HO_N_AT_LEVEL = 0, /* instances at level L */
  ARGUS_HO_N_GAPS = 1,     /* successive pairs measured */
  ARGUS_HO_GAP_SUM = 2,    /* their gaps, summed mod 2^64 */
  ARGUS_HO_INTERNAL = 7,   /* internal-error bits: 0 unless a consistency check in the
                              library fails */
  ARGUS_HO_NUM_COUNTERS = 8
};

typedef struct argus_handoffs_config {
  uint32_t abi_version; /* ARGUS_ATTR_ABI_VERSION */
  uint32_t num_regions; /* R, 1..4096 (the pair table is R x R) */
  uint32_t level;       /* L */
  uint32_t pad;
} argus_handoffs_config;

typedef struct argus_handoffs_io {
  const argus_instance* d_instances; /* canonical order (16-byte aligned) */
  const uint64_t* d_n_instances;     /* device scalar, e.g. &d_counters[ARGUS_C_N_BEGIN] */
  uint64_t max_instances;            /* capacity, < 2^31 */
  uint64_t* d_pairs;                 /* out [R][R][4]: for (region(x), region(y)): count,
                                        gap sum, min (UINT64_MAX if none), max */
  uint64_t* d_hist;                  /* out [65]: gaps by bit width */
  uint64_t* d_parent_gap;            /* out [max_instances] or NULL: per parent instance,
                                        the sum of the gaps between its successive level-L
                                        children (the handoff time of one step) */
  uint64_t* d_counters;              /* out [ARGUS_HO_NUM_COUNTERS] */
} argus_handoffs_io;

/* Device workspace argus_attr_handoffs needs (256-byte aligned); 0 for
 * max_instances >= 2^31 or num_regions outside 1..4096. */
size_t argus_attr_handoffs_workspace_bytes(uint64_t max_instances, uint32_t num_regions);

/* Enqueue the handoff statistics on `stream` without synchronising.
 * Allocates nothing; argument errors are returned before any GPU call. */
int argus_attr_handoffs(const argus_handoffs_config* cfg, const argus_handoffs_io* io,
                        void* d_workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------- Chrome-trace export */
/* Writes the JSON of Chrome Trace Viewer for region instances and probe
 * summaries, with the lane layout of the paper's Appendix B: a process per
 * group of contexts (ctx_key >> group_shift; an SM or a block); per
 * context, one lane per nesting level of its reference instances (levels
 * >= 7 share lane 7), then for each operation region with probe groups in
 * that context a lane with the mean exposed latency (a slice from the
 * operation's issue in the reference trace, as long as the mean) and a lane
 * with the 80th, 60th, 40th, 20th and 0th percentile bands (slices from the
 * issue, each nested in the previous).  Timestamps are cycles divided by
 * cycles_per_us (microseconds, as the format requires).  Host memory; no
 * GPU call.  Returns ARGUS_OK, ARGUS_E_INVAL for bad arguments (a group
 * naming an instance >= n_instances included) or ARGUS_E_IO. */
enum { ARGUS_TRACE_UNMATCHED = 1u }; /* also draw mismatched pairs */

typedef struct argus_trace_options {
  double cycles_per_us;            /* > 0 */
  uint32_t group_shift;            /* 0..32 */
  uint32_t flags;                  /* ARGUS_TRACE_* */
  const char* const* region_names; /* [num_regions] or NULL ("r<id>") */
  uint32_t num_regions;            /* 1..65535 */
  uint32_t pad;
} argus_trace_options;

int argus_attr_chrome_trace(const argus_instance* h_instances, uint64_t n_instances,
                            const uint64_t* h_groups, const double* h_mean, uint64_t n_groups,
                            const argus_trace_options* opt, const char* path);

/* Destroy a handle; NULL is a no-op. */
void argus_attr_destroy(argus_attr* h);

/* Message for the last non-zero return on this handle ("" if none). */
const char* argus_attr_last_error(const argus_attr* h);

/* ---------------------------------------------------------------- timing */
/* Per-kernel timing for measurement.  While enabled, every `run` records a
 * HIP event before its first launch and after each kernel launch, on its
 * stream (no host synchronisation).  argus_attr_kernel_times synchronises on
 * those events, fills up to `cap` entries of names[] (static strings) and
 * ms[] with the elapsed time of each launch of every run since the previous
 * call, in launch order, forgets them, and returns how many launches there
 * were (which may exceed cap), or a negative code. */
int argus_attr_set_timing(argus_attr* h, int enable);
int argus_attr_kernel_times(argus_attr* h, const char** names, float* ms, int cap);

/* Restricts timing to the launches of one step (a name as reported by
 * argus_attr_kernel_times, e.g. "match"): while a name is set, every timed
 * `run` records one event before and one after each launch of that step
 * only, so that the rest of the run is not slowed by events.  NULL or ""
 * clears the filter.  Returns ARGUS_OK, or ARGUS_E_INVAL for a NULL handle. */
int argus_attr_set_timing_filter(argus_attr* h, const char* name);

#ifdef __cplusplus
}
#endif

#endif /* ARGUS_ATTR_H */
