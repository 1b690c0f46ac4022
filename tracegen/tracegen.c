/*
 * tracegen.c -- seeded synthetic marker traces shaped like the paper's
 * persistent-kernel workloads (Section 4: warp-specialised persistent GEMM,
 * TinyLlama decode megakernel, GEMM + all-gather overlap) plus a large
 * skewed stress trace.
 *
 * This module only GENERATES inputs.  It holds none of the attribution
 * arithmetic (no sorting of records, no matching, no aggregation).  For the
 * well-formed configurations it also writes the list of region instances it
 * generated ("ground truth"), in context-major, begin-time order; a parent is
 * the index of the enclosing generated instance.
 *
 * Randomness: xoshiro256** (Blackman & Vigna, "Scrambled linear
 * pseudorandom number generators", 2018) seeded with splitmix64; every
 * context has its own stream, so the output does not depend on the number
 * of threads.
 *
 * Record layout (16 B): u64 ts, u32 ctx_key, u16 region_id, u8 kind
 * (1 = BEGIN, 2 = END), u8 pad (0).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
  uint64_t ts;
  uint32_t ctx;
  uint16_t region;
  uint8_t kind;
  uint8_t pad;
} tg_record;

typedef struct {
  uint64_t t_begin, t_end;
  uint32_t ctx, parent, level;
  uint16_t region, end_region;
} tg_instance;

_Static_assert(sizeof(tg_record) == 16, "record");
_Static_assert(sizeof(tg_instance) == 32, "instance");

/* ------------------------------------------------------------------ RNG */
typedef struct {
  uint64_t s[4];
} rng_t;

static uint64_t splitmix64(uint64_t* x) {
  uint64_t z = (*x += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static void rng_seed(rng_t* r, uint64_t a, uint64_t b, uint64_t c) {
  uint64_t x = a * 0xD1B54A32D192ED03ull ^ b * 0x8CB92BA72F3D8DD7ull ^ c;
  for (int i = 0; i < 4; ++i) r->s[i] = splitmix64(&x);
}
static inline uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }
static inline uint64_t rng_next(rng_t* r) {
  uint64_t* s = r->s;
  const uint64_t result = rotl(s[1] * 5, 7) * 9;
  const uint64_t t = s[1] << 17;
  s[2] ^= s[0];
  s[3] ^= s[1];
  s[1] ^= s[2];
  s[0] ^= s[3];
  s[2] ^= t;
  s[3] = rotl(s[3], 45);
  return result;
}
static inline double rng_unit(rng_t* r) { /* [0, 1) */
  return (double)(rng_next(r) >> 11) * (1.0 / 9007199254740992.0);
}
static inline uint64_t rng_below(rng_t* r, uint64_t n) { /* [0, n) */
  return (uint64_t)(rng_unit(r) * (double)n) % (n ? n : 1);
}
static inline double rng_exp(rng_t* r, double mean) { return -mean * log1p(-rng_unit(r)); }
static inline double rng_normal(rng_t* r) {
  double u1 = rng_unit(r), u2 = rng_unit(r);
  if (u1 < 1e-300) u1 = 1e-300;
  return sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
}
static inline uint64_t rng_lognormal_cycles(rng_t* r, double mu, double sigma) {
  double v = exp(mu + sigma * rng_normal(r));
  uint64_t d = (uint64_t)llround(v);
  return d < 1 ? 1 : d;
}
static inline uint64_t gap_exp(rng_t* r, double mean) {
  return 1 + (uint64_t)floor(rng_exp(r, mean));
}

/* A region id in [lo, lo + n) different from `avoid` (if avoid is in range
 * and n > 1). */
static uint16_t pick_region(rng_t* r, uint32_t lo, uint32_t n, int avoid) {
  if (avoid >= (int)lo && avoid < (int)(lo + n) && n > 1) {
    uint32_t k = (uint32_t)rng_below(r, n - 1);
    uint32_t v = lo + k;
    if ((int)v >= avoid) v += 1;
    return (uint16_t)v;
  }
  return (uint16_t)(lo + rng_below(r, n));
}

/* ----------------------------------------------------------- emitters */
typedef struct {
  tg_record* rec;     /* this context's records (context-major) */
  uint64_t nrec;
  tg_instance* tru;   /* this context's instances, or NULL */
  uint64_t ntru;
  uint64_t tru_base;  /* global index of tru[0] */
  uint32_t ctx;
  /* open-instance stack (indices into tru) for parents */
  uint32_t stk[64];
  int depth;
} emitter;

static void em_begin(emitter* e, uint64_t ts, uint16_t region) {
  tg_record* r = &e->rec[e->nrec++];
  r->ts = ts;
  r->ctx = e->ctx;
  r->region = region;
  r->kind = 1;
  r->pad = 0;
  if (e->tru) {
    tg_instance* x = &e->tru[e->ntru];
    x->t_begin = ts;
    x->t_end = ~0ull;
    x->ctx = e->ctx;
    x->parent = e->depth > 0 ? (uint32_t)(e->tru_base + e->stk[e->depth - 1]) : 0xFFFFFFFFu;
    x->level = (uint32_t)e->depth;
    x->region = region;
    x->end_region = 0xFFFF;
    e->stk[e->depth] = (uint32_t)e->ntru;
    e->ntru++;
  }
  e->depth++;
}
static void em_end(emitter* e, uint64_t ts, uint16_t region) {
  tg_record* r = &e->rec[e->nrec++];
  r->ts = ts;
  r->ctx = e->ctx;
  r->region = region;
  r->kind = 2;
  r->pad = 0;
  e->depth--;
  if (e->tru) {
    tg_instance* x = &e->tru[e->stk[e->depth]];
    x->t_end = ts;
    x->end_region = region;
  }
}

/* ------------------------------------------------------------ configs */
#define SHUF_CHUNK 256


/* C1: random bounded walk, depth <= 3, 8 regions, child region != parent,
 * gaps 1 + Exp(200), per-context base U[0, 1000). */
static void gen_c1(emitter* e, rng_t* r, uint64_t m) {
  uint64_t t = rng_below(r, 1000);
  uint16_t reg[8];
  for (uint64_t i = 0; i < m; ++i) {
    uint64_t rem = m - i;
    int d = e->depth;
    int begin;
    if ((uint64_t)d == rem) begin = 0;
    else if (d == 0) begin = 1;
    else if (d == 3) begin = 0;
    else begin = rng_unit(r) < 0.5;
    if (i > 0) t += gap_exp(r, 200.0);
    if (begin) {
      uint16_t g = pick_region(r, 0, 8, d > 0 ? reg[d - 1] : -1);
      reg[d] = g;
      em_begin(e, t, g);
    } else {
      em_end(e, t, reg[d - 1]);
    }
  }
}

/* C2: persistent GEMM warp.  Producer warps (0, 1): tile id 0 around stages
 * 1..4; consumer warps: tile id 5 around stages 6..11.  Stage durations
 * LogNormal(ln 800, 0.6), gaps 1 + Exp(50). */
static void gen_c2(emitter* e, rng_t* r, uint64_t m, uint32_t warp, uint64_t base) {
  const int producer = warp < 2;
  const uint16_t tile = producer ? 0 : 5;
  const uint16_t first = producer ? 1 : 6;
  const int nst = producer ? 4 : 6;
  const uint64_t full = 2 + 2 * (uint64_t)nst;
  uint64_t t = base;
  uint64_t left = m;
  int first_rec = 1;
  while (left > 0) {
    if (left == 2) { /* a lone stage at top level */
      if (!first_rec) t += gap_exp(r, 50.0);
      em_begin(e, t, first);
      t += rng_lognormal_cycles(r, log(800.0), 0.6);
      em_end(e, t, first);
      left -= 2;
      break;
    }
    int ns = nst;
    if (left < full) ns = (int)((left - 2) / 2);
    if (!first_rec) t += gap_exp(r, 50.0);
    first_rec = 0;
    em_begin(e, t, tile);
    for (int s = 0; s < ns; ++s) {
      t += gap_exp(r, 50.0);
      em_begin(e, t, (uint16_t)(first + s));
      t += rng_lognormal_cycles(r, log(800.0), 0.6);
      em_end(e, t, (uint16_t)(first + s));
    }
    t += gap_exp(r, 50.0);
    em_end(e, t, tile);
    left -= 2 + 2 * (uint64_t)ns;
  }
}

/* C3 helper: one layer's operator instances, a random bracket sequence of
 * `nops` instances nested at most 3 deep, operators of that layer only. */
static void gen_c3_layer(emitter* e, rng_t* r, uint64_t* t, uint32_t layer, int nops) {
  int opened = 0, d = 0;
  uint16_t reg[4];
  int had_child[4] = {0, 0, 0, 0};
  while (opened < nops || d > 0) {
    int begin;
    if (opened == nops) begin = 0;
    else if (d == 0) begin = 1;
    else if (d == 3) begin = 0;
    else begin = rng_unit(r) < 0.35;
    *t += gap_exp(r, 100.0);
    if (begin) {
      uint16_t op = pick_region(r, 8 * layer, 8, d > 0 ? reg[d - 1] : -1);
      if (d > 0) had_child[d - 1] = 1;
      reg[d] = op;
      had_child[d] = 0;
      em_begin(e, *t, op);
      ++opened;
      ++d;
    } else {
      if (!had_child[d - 1]) *t += rng_lognormal_cycles(r, log(3000.0), 0.8);
      em_end(e, *t, reg[d - 1]);
      --d;
    }
  }
}

/* C3: decode megakernel warp: `tokens` tokens, each B(176) ... E(176) around
 * 63 operator instances spread over 22 layers in layer order. */
static void gen_c3(emitter* e, rng_t* r, uint64_t m, uint64_t base) {
  const uint64_t tokens = m / 128;
  uint64_t t = base;
  for (uint64_t k = 0; k < tokens; ++k) {
    if (k > 0) t += gap_exp(r, 100.0);
    em_begin(e, t, 176);
    /* 63 = 22 * 2 + 19: 19 distinct layers get a third instance. */
    int cnt[22];
    int idx[22];
    for (int l = 0; l < 22; ++l) { cnt[l] = 2; idx[l] = l; }
    for (int l = 0; l < 19; ++l) {
      int j = l + (int)rng_below(r, (uint64_t)(22 - l));
      int tmp = idx[l]; idx[l] = idx[j]; idx[j] = tmp;
      cnt[idx[l]] += 1;
    }
    for (uint32_t l = 0; l < 22; ++l) gen_c3_layer(e, r, &t, l, cnt[l]);
    t += gap_exp(r, 100.0);
    em_end(e, t, 176);
  }
}

/* C4: flat compute (warps 0..5, ids 0..5) or comm (warps 6, 7, ids 6..9)
 * regions; lengths LogNormal(ln 5000, 1.0); gaps 1 + Exp(1000) for compute
 * and 1 + Exp(8000) for comm. */
static void gen_c4(emitter* e, rng_t* r, uint64_t m, uint32_t warp, uint64_t base) {
  const int comm = warp >= 6;
  uint64_t t = base;
  for (uint64_t i = 0; i < m / 2; ++i) {
    t += gap_exp(r, comm ? 8000.0 : 1000.0);
    uint16_t g = comm ? (uint16_t)(6 + rng_below(r, 4)) : (uint16_t)rng_below(r, 6);
    em_begin(e, t, g);
    t += rng_lognormal_cycles(r, log(5000.0), 1.0);
    em_end(e, t, g);
  }
}

/* C5: bounded walk, depth <= 8, 1024 regions (child != parent), gaps
 * 1 + Exp(200), base 2^39 + U[0, 2^30); `ins` malformed markers inserted at
 * uniformly chosen positions, each kind by a fair coin: a duplicate BEGIN
 * that repeats the region of the last BEGIN written in this context, or an
 * END of a uniformly random region.  The two kinds are equally frequent, so
 * the excess of the clamped stack depth over the well-formed depth is a
 * reflected random walk and reaches levels near 10^3 in the hot contexts. */
static void gen_c5(emitter* e, rng_t* r, uint64_t m, uint64_t ins) {
  uint64_t t = (1ull << 39) + rng_below(r, 1ull << 30);
  const uint64_t w = m - ins; /* well-formed records */
  uint64_t wdone = 0, ins_left = ins;
  int d = 0;
  uint16_t reg[9];
  uint16_t last_begin = (uint16_t)rng_below(r, 1024);
  for (uint64_t i = 0; i < m; ++i) {
    const uint64_t slots_left = m - i;
    if (i > 0) t += gap_exp(r, 200.0);
    if (ins_left > 0 && rng_unit(r) * (double)slots_left < (double)ins_left) {
      ins_left--;
      tg_record* x = &e->rec[e->nrec++];
      x->ts = t;
      x->ctx = e->ctx;
      x->pad = 0;
      if (rng_unit(r) < 0.5) {
        x->kind = 1;
        x->region = last_begin;
      } else {
        x->kind = 2;
        x->region = (uint16_t)rng_below(r, 1024);
      }
      continue;
    }
    const uint64_t rem = w - wdone;
    int begin;
    if ((uint64_t)d == rem) begin = 0;
    else if (d == 0) begin = 1;
    else if (d == 8) begin = 0;
    else begin = rng_unit(r) < 0.5;
    tg_record* x = &e->rec[e->nrec++];
    x->ts = t;
    x->ctx = e->ctx;
    x->pad = 0;
    if (begin) {
      uint16_t g = pick_region(r, 0, 1024, d > 0 ? reg[d - 1] : -1);
      reg[d++] = g;
      x->kind = 1;
      x->region = g;
      last_begin = g;
    } else {
      --d;
      x->kind = 2;
      x->region = reg[d];
    }
    wdone++;
  }
}

/* ------------------------------------------------------------- driver */
static uint64_t default_blocks(int cfg) {
  switch (cfg) {
    case 1: return 8;
    case 2: return 256;
    case 3: return 256;
    case 4: return 256;
    case 5: return 2048;
  }
  return 0;
}
static uint64_t default_warps(int cfg) {
  switch (cfg) {
    case 1: return 4;
    case 2: return 8;
    case 3: return 16;
    case 4: return 8;
    case 5: return 16;
  }
  return 0;
}
static uint64_t default_size(int cfg) {
  switch (cfg) {
    case 1: return 2048;
    case 2: return 8192;
    case 3: return 16384;
    case 4: return 16384;
    case 5: return 1ull << 28;
  }
  return 0;
}

/* Number of regions and classes of a configuration, and its class table
 * (entries >= K are unclassified).  Returns R, writes K. */
int tg_regions(int cfg, uint8_t* cls_out /* [65536] or NULL */, int* k_out) {
  int R = 0, K = 0;
  switch (cfg) {
    case 1: R = 8; K = 2; break;
    case 2: R = 12; K = 2; break;
    case 3: R = 177; K = 8; break;
    case 4: R = 10; K = 2; break;
    case 5: R = 1024; K = 4; break;
    default: return -1;
  }
  if (cls_out) {
    for (int g = 0; g < R; ++g) {
      uint8_t c = 0xFF;
      switch (cfg) {
        case 1: c = (uint8_t)(g & 1); break;
        case 2: c = g <= 4 ? 0 : 1; break;
        case 3: c = g < 176 ? (uint8_t)(g & 7) : 0xFF; break;
        case 4: c = g <= 5 ? 0 : 1; break;
        case 5: c = (uint8_t)(g & 3); break;
      }
      cls_out[g] = c;
    }
  }
  if (k_out) *k_out = K;
  return R;
}

static const double* g_frac;
static int cmp_frac_desc(const void* a, const void* b) {
  uint64_t i = *(const uint64_t*)a, j = *(const uint64_t*)b;
  if (g_frac[i] > g_frac[j]) return -1;
  if (g_frac[i] < g_frac[j]) return 1;
  return i < j ? -1 : (i > j);
}

/* C5 per-context record counts: Zipf(1.2) over a seeded permutation of the
 * context ranks, scaled to sum to `total` (even), largest-remainder
 * rounding on pairs, at least one pair per context. */
static void c5_counts(uint64_t seed, uint64_t nctx, uint64_t total, uint64_t* m) {
  const uint64_t pairs = total / 2;
  double* w = (double*)malloc(sizeof(double) * nctx);
  uint64_t* perm = (uint64_t*)malloc(sizeof(uint64_t) * nctx);
  double* frac = (double*)malloc(sizeof(double) * nctx);
  rng_t r;
  rng_seed(&r, seed, 5, 0xC5C5);
  for (uint64_t i = 0; i < nctx; ++i) perm[i] = i;
  for (uint64_t i = nctx; i > 1; --i) {
    uint64_t j = rng_below(&r, i);
    uint64_t tmp = perm[i - 1]; perm[i - 1] = perm[j]; perm[j] = tmp;
  }
  double sw = 0;
  for (uint64_t k = 0; k < nctx; ++k) sw += pow((double)(k + 1), -1.2);
  uint64_t given = 0;
  for (uint64_t k = 0; k < nctx; ++k) {
    double ideal = (double)pairs * pow((double)(k + 1), -1.2) / sw;
    uint64_t f = (uint64_t)floor(ideal);
    w[k] = (double)f;
    frac[k] = ideal - (double)f;
    given += f;
  }
  /* largest remainders get the leftover pairs (ties by rank) */
  uint64_t left = pairs - given;
  uint64_t* ord = (uint64_t*)malloc(sizeof(uint64_t) * nctx);
  for (uint64_t k = 0; k < nctx; ++k) ord[k] = k;
  g_frac = frac;
  qsort(ord, nctx, sizeof(uint64_t), cmp_frac_desc);
  for (uint64_t k = 0; k < nctx && left > 0; ++k, --left) w[ord[k]] += 1.0;
  free(ord);
  /* at least one pair each, taken from the largest */
  for (uint64_t k = 0; k < nctx; ++k) {
    if (w[k] < 1.0) { w[k] = 1.0; w[0] -= 1.0; }
  }
  for (uint64_t k = 0; k < nctx; ++k) m[perm[k]] = 2 * (uint64_t)w[k];
  free(w);
  free(perm);
  free(frac);
}

static uint64_t c3_drops(uint64_t n_end) { return (n_end + 500) / 1000; }

/* Exact number of records tg_generate will write. */
int64_t tg_size(int cfg, uint32_t n_blocks, uint32_t warps, uint64_t size) {
  if (cfg < 1 || cfg > 5) return -1;
  uint64_t B = n_blocks ? n_blocks : default_blocks(cfg);
  uint64_t W = warps ? warps : default_warps(cfg);
  uint64_t S = size ? size : default_size(cfg);
  if (cfg == 5) return (int64_t)(S & ~1ull);
  if (cfg == 3) S = (S / 128) * 128;
  S &= ~1ull;
  uint64_t n = B * W * S;
  if (cfg == 3) n -= c3_drops(n / 2);
  return (int64_t)n;
}

/* Number of ground-truth instances (well-formed configs 1, 2, 4), else 0. */
int64_t tg_truth_size(int cfg, uint32_t n_blocks, uint32_t warps, uint64_t size) {
  if (cfg == 1 || cfg == 2 || cfg == 4) return tg_size(cfg, n_blocks, warps, size) / 2;
  return 0;
}

/* Interleave context-major runs into `out`: round robin over the contexts
 * that still have records, `chunk` records at a time. */
static void interleave(const tg_record* src, const uint64_t* off, const uint64_t* cnt,
                       uint64_t nctx, uint64_t chunk, tg_record* out) {
  uint64_t* pos = (uint64_t*)calloc(nctx, sizeof(uint64_t));
  uint64_t* act = (uint64_t*)malloc(sizeof(uint64_t) * nctx);
  uint64_t na = 0;
  for (uint64_t c = 0; c < nctx; ++c)
    if (cnt[c] > 0) act[na++] = c;
  uint64_t o = 0;
  while (na > 0) {
    uint64_t keep = 0;
    for (uint64_t a = 0; a < na; ++a) {
      uint64_t c = act[a];
      uint64_t take = cnt[c] - pos[c];
      if (take > chunk) take = chunk;
      memcpy(out + o, src + off[c] + pos[c], take * sizeof(tg_record));
      o += take;
      pos[c] += take;
      if (pos[c] < cnt[c]) act[keep++] = c;
    }
    na = keep;
  }
  free(pos);
  free(act);
}

/*
 * Generate configuration `cfg` (1..5).  n_blocks, warps and size default to
 * the full configuration when 0; `size` is records per context for 1..4
 * and the total record count for 5.  Writes tg_size() records to `out` and,
 * for configs 1, 2 and 4, tg_truth_size() instances to `truth` (if not
 * NULL).  Returns the number of records, or a negative value on error.
 */
int64_t tg_generate(int cfg, uint64_t seed, uint32_t n_blocks, uint32_t warps,
                    uint64_t size, void* out_v, uint64_t out_cap, void* truth_v,
                    uint64_t truth_cap, int threads) {
  const int64_t total = tg_size(cfg, n_blocks, warps, size);
  if (total < 0) return -1;
  if ((uint64_t)total > out_cap) return -2;
  const uint64_t B = n_blocks ? n_blocks : default_blocks(cfg);
  const uint64_t W = warps ? warps : default_warps(cfg);
  uint64_t S = size ? size : default_size(cfg);
  if (cfg == 3) S = (S / 128) * 128;
  S &= ~1ull;
  const uint64_t nctx = B * W;
  if (nctx == 0 || nctx > (1ull << 32)) return -1;
  const int want_truth = truth_v != NULL && (cfg == 1 || cfg == 2 || cfg == 4);
  if (want_truth && truth_cap < (uint64_t)total / 2) return -3;

  uint64_t* cnt = (uint64_t*)malloc(sizeof(uint64_t) * nctx);
  uint64_t* off = (uint64_t*)malloc(sizeof(uint64_t) * (nctx + 1));
  if (cfg == 5) {
    c5_counts(seed, nctx, (uint64_t)total, cnt);
  } else {
    for (uint64_t c = 0; c < nctx; ++c) cnt[c] = S;
  }
  off[0] = 0;
  for (uint64_t c = 0; c < nctx; ++c) off[c + 1] = off[c] + cnt[c];
  const uint64_t gen_total = off[nctx];

  tg_record* tmp = (tg_record*)malloc(sizeof(tg_record) * (gen_total ? gen_total : 1));
  tg_instance* tru = want_truth ? (tg_instance*)truth_v : NULL;
  if (!tmp) return -4;

  /* per-block bases */
  uint64_t* base = (uint64_t*)malloc(sizeof(uint64_t) * B);
  for (uint64_t b = 0; b < B; ++b) {
    rng_t rb;
    rng_seed(&rb, seed, (uint64_t)cfg * 7919 + 1, b);
    uint64_t range = (cfg == 4) ? (1ull << 32) : (1ull << 20);
    base[b] = rng_below(&rb, range);
  }

#ifdef _OPENMP
  if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int64_t ci = 0; ci < (int64_t)nctx; ++ci) {
    const uint64_t c = (uint64_t)ci;
    rng_t r;
    rng_seed(&r, seed, (uint64_t)cfg, c + 1);
    emitter e;
    memset(&e, 0, sizeof(e));
    e.rec = tmp + off[c];
    e.ctx = (uint32_t)c;
    if (tru) {
      e.tru = tru + off[c] / 2;
      e.tru_base = off[c] / 2;
    }
    const uint32_t warp = (uint32_t)(c % W);
    const uint64_t blk = c / W;
    switch (cfg) {
      case 1: gen_c1(&e, &r, cnt[c]); break;
      case 2: gen_c2(&e, &r, cnt[c], warp, base[blk]); break;
      case 3: gen_c3(&e, &r, cnt[c], base[blk]); break;
      case 4: gen_c4(&e, &r, cnt[c], warp, base[blk]); break;
      case 5: {
        uint64_t ins = 2 * ((cnt[c] + 100) / 200);
        if (ins > cnt[c]) ins = 0;
        gen_c5(&e, &r, cnt[c], ins);
        break;
      }
    }
  }
  (void)threads;

  tg_record* out = (tg_record*)out_v;
  const uint64_t chunk = (cfg == 1 || cfg == 2) ? 1 : 256;
  /* config 3 drops records afterwards, so it interleaves into a buffer of
   * its own first */
  tg_record* lay = out;
  if (cfg == 3) {
    lay = (tg_record*)malloc(sizeof(tg_record) * (gen_total ? gen_total : 1));
    if (!lay) return -4;
  }
  interleave(tmp, off, cnt, nctx, chunk, lay);
  free(tmp);
  free(base);

  if (cfg == 1) { /* Fisher-Yates within each 4 KiB (256-record) chunk */
    rng_t r;
    rng_seed(&r, seed, 1, 0x5F5F);
    for (uint64_t s = 0; s < gen_total; s += SHUF_CHUNK) {
      uint64_t len = gen_total - s < SHUF_CHUNK ? gen_total - s : SHUF_CHUNK;
      for (uint64_t i = len; i > 1; --i) {
        uint64_t j = rng_below(&r, i);
        tg_record t = out[s + i - 1];
        out[s + i - 1] = out[s + j];
        out[s + j] = t;
      }
    }
  }
  if (cfg == 3) { /* drop 0.1% of the END markers, uniformly (selection sampling) */
    uint64_t n_end = 0;
    for (uint64_t i = 0; i < gen_total; ++i) n_end += lay[i].kind == 2;
    uint64_t drop = c3_drops(n_end), seen = 0, o = 0;
    rng_t r;
    rng_seed(&r, seed, 3, 0xD0D0);
    for (uint64_t i = 0; i < gen_total; ++i) {
      if (lay[i].kind == 2) {
        uint64_t left = n_end - seen;
        seen++;
        if (drop > 0 && rng_unit(&r) * (double)left < (double)drop) {
          drop--;
          continue;
        }
      }
      out[o++] = lay[i];
    }
    free(lay);
  }
  free(cnt);
  free(off);
  return total;
}
