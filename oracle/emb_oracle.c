/*
 * Reference oracle for the cached mixed-precision EmbeddingBag training step of
 * "Mixed-Precision Embedding Using a Cache" (Yang, Park, Naumov, Smelyanskiy et al., 2020).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, obviously-correct CPU
 * model of what the GPU library computes.  Only the test-suite, the smoke check
 * and the CPU-baseline leg of the benchmark may load it.  It shares no code,
 * header, table or helper with the HIP library: it has its own Philox, its own
 * FP32->FP16 conversion, its own config struct and its own state layout.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared emb_oracle.c -lm
 * (no fast-math: every float operation below is one IEEE-754 binary32 operation
 * in round-to-nearest-even, and fmaf() is the correctly rounded fused op).
 *
 * What it computes, per the paper:
 *   fetch(T,C,i)   -- Sec. 3: the cached FP32 row if row i is resident in set h(i),
 *                     else the up-converted low-precision row (Alg. 1 dequant).
 *   forward        -- sum of fetched rows per bag (pooling mode is not stated in
 *                     the paper; sum is the reading used here).
 *   update(T,C,i,x) -- Sec. 3 "Cache Replacement Policy" and Alg. 2, applied to the
 *                     de-duplicated rows of the mini-batch (Sec. 5.1 "De-duplicate
 *                     gradients"): sort rows, merge the gradients of the same row,
 *                     apply one update per unique row.
 *   quantization   -- Sec. 3 "Precision" and Alg. 1: row-wise uniform min-max,
 *                     b = min, s = (max-min)/(2^bits-1), codes in [0, 2^bits-1]
 *                     for INT8, INT4 and INT2; or the IEEE binary16 value of each
 *                     element for an FP16 table (no (s,b)).
 *   rounding       -- Sec. 3 "Rounding": nearest with ties to even, or stochastic
 *                     rounding with E[q] = v, between consecutive codes or between
 *                     the two FP16 values one unit in the last place apart.
 *
 * Readings taken where the paper is silent (each is listed in the design notes):
 *   hash h(i) = i mod n_sets; n_sets = max(1, floor(floor(frac*N)/assoc)), 0 when
 *   frac == 0 (no cache); Alg. 2 applied per set in a two-phase batched form
 *   (all priority values updated first, then victims ordered by (PV asc, way asc)
 *   with empty ways lowest, candidates by (PV desc, row asc), the k-th candidate
 *   takes the k-th victim while strictly higher, stopping at the first failure);
 *   LRU timestamp = step counter; LFU count += occurrences, halved every
 *   `lfu_decay_interval` steps; gradient sum of a row in position order: up to
 *   512 occurrences in chunks of 64 (each chunk left to right, then the chunk
 *   partials left to right), more than 512 by bag blocks of 32768/d bags (the
 *   occurrences of each block left to right, then the non-empty block partials
 *   left to right);
 *   row-wise Adagrad G += mean(g^2) with a halving-tree sum; SR uniform from
 *   Philox4x32-10 keyed on (seed, step, table, row, col).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_LRU 0
#define ORC_LFU 1

#define ORC_NSTAT 12
enum {
  ST_LOOKUPS = 0,     /* valid forward occurrences */
  ST_HIT_LOOKUPS,     /* forward occurrences served from the FP32 cache */
  ST_BWD_LOOKUPS,     /* valid occurrences seen by backward_update */
  ST_UNIQUE,          /* unique rows updated */
  ST_UNIQUE_HITS,     /* unique rows resident before the step */
  ST_INSERTS,         /* rows placed in the cache */
  ST_BYPASSES,        /* missed rows written straight to the low-precision table */
  ST_EVICTIONS,       /* valid residents displaced (includes hit-evictions) */
  ST_EMPTY_FILLS,     /* inserts into empty ways */
  ST_HIT_EVICTIONS,   /* residents updated this step and then displaced (LFU) */
  ST_INVALID_FWD,     /* out-of-range indices seen by forward */
  ST_INVALID_BWD      /* out-of-range indices seen by backward_update */
};

typedef struct {
  int32_t num_tables;
  int32_t dim;
  int32_t bits;               /* 8, 4 or 2 (integer codes), or 16 (FP16 table) */
  int32_t sb_fp16;            /* 0: (s,b) in FP32; 1: (s,b) rounded to FP16 */
  double cache_fraction;
  int32_t assoc;
  int32_t policy;             /* ORC_LRU / ORC_LFU */
  int32_t lfu_decay_interval; /* 0 = never */
  int32_t stochastic;         /* 0 nearest-even, 1 stochastic rounding */
  int32_t adagrad;            /* 0 SGD, 1 row-wise Adagrad */
  float lr;
  float eps;
  uint64_t seed;
} orc_config;

typedef struct {
  int64_t N, n_sets, slots;
  uint8_t *code;   /* [N][d], one code per byte (integer precisions) */
  uint16_t *h16;   /* [N][d], binary16 bit patterns (FP16 table) */
  float *scale;    /* [N] (FP16-representable values when sb_fp16) */
  float *bias;     /* [N] */
  float *crow;     /* [slots][d] FP32 cache rows */
  int32_t *tag;    /* [slots], -1 = empty */
  int32_t *ts;     /* [slots], LRU last-access step, -1 = empty */
  int32_t *cnt;    /* [N], LFU access counts */
  float *G;        /* [N], row-wise Adagrad accumulators */
  int64_t stat[ORC_NSTAT];
} orc_table;

typedef struct {
  orc_config cfg;
  uint64_t step;
  orc_table *tab;
} orc_t;

/* ------------------------------------------------------------------------- */
/* Philox4x32-10, from Salmon, Moraes, Dror, Shaw, "Parallel random numbers:   */
/* as easy as 1, 2, 3" (SC'11): ten rounds of two 32x32->64 multiplies and     */
/* xors with a Weyl-sequence key schedule.                                     */
/* ------------------------------------------------------------------------- */
void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint64_t prod0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    uint64_t prod1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
    uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* 24-bit uniform in [0,1) for element (table, row, col) at `step`:
 * counter = (col/4, row, table, step), key = seed; word col%4 of the block. */
float orc_uniform(uint64_t seed, uint32_t step, uint32_t table, uint32_t row, uint32_t col) {
  uint32_t ctr[4] = {col >> 2, row, table, step};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t out[4];
  orc_philox4x32_10(ctr, key, out);
  uint32_t w = out[col & 3u];
  return (float)(w >> 8) * (1.0f / 16777216.0f);
}

/* ------------------------------------------------------------------------- */
/* IEEE binary16 conversion, written from the format definition: 1 sign bit,   */
/* 5 exponent bits (bias 15), 10 fraction bits; subnormals below 2^-14;        */
/* round to nearest, ties to even; overflow to infinity.                        */
/* ------------------------------------------------------------------------- */
uint16_t orc_f32_to_f16_bits(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
  uint32_t exp = (u >> 23) & 0xFFu;
  uint32_t man = u & 0x7FFFFFu;
  if (exp == 0xFFu) {                       /* inf / nan */
    if (man == 0) return sign | 0x7C00u;
    return sign | 0x7E00u;
  }
  /* value = 1.man * 2^(exp-127) for normal inputs */
  int32_t e = (int32_t)exp - 127;
  if (exp == 0) return sign;                /* fp32 subnormals are far below fp16's range */
  if (e > 15) return sign | 0x7C00u;        /* overflow */
  uint32_t full = man | 0x800000u;          /* 24-bit significand */
  int32_t shift;                            /* bits to drop from the 24-bit significand */
  uint32_t he;                              /* biased fp16 exponent of the result */
  if (e >= -14) {
    shift = 13;                             /* keep 11 bits (implicit + 10) */
    he = (uint32_t)(e + 15);
  } else {
    shift = 13 + (-14 - e);                 /* subnormal: value = m * 2^-24 */
    he = 0;
    if (shift > 25) return sign;            /* below half of the smallest subnormal */
  }
  uint32_t kept = full >> shift;
  uint32_t rem = full & ((1u << shift) - 1u);
  uint32_t half = 1u << (shift - 1);
  if (rem > half || (rem == half && (kept & 1u))) kept += 1u;
  uint32_t bits;
  if (he == 0) {
    bits = kept;                            /* may carry into the first normal: still right */
  } else {
    /* kept in [2^10, 2^11]; a carry to 2^11 bumps the exponent */
    if (kept == 0x800u) {
      kept = 0x400u;
      he += 1;
      if (he >= 31) return sign | 0x7C00u;
    }
    bits = (he << 10) | (kept & 0x3FFu);
  }
  return (uint16_t)(sign | bits);
}

float orc_f16_bits_to_f32(uint16_t h) {
  uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
  uint32_t exp = ((uint32_t)h >> 10) & 0x1Fu;
  uint32_t man = (uint32_t)h & 0x3FFu;
  float mag;
  if (exp == 0) {
    mag = ldexpf((float)man, -24);
  } else if (exp == 31) {
    mag = man ? NAN : INFINITY;
  } else {
    mag = ldexpf((float)(man | 0x400u), (int)exp - 25);
  }
  uint32_t u;
  memcpy(&u, &mag, 4);
  u |= sign;
  float out;
  memcpy(&out, &u, 4);
  return out;
}

float orc_round_to_f16(float x) { return orc_f16_bits_to_f32(orc_f32_to_f16_bits(x)); }

/* The binary16 value next to h in increasing (up = 1) or decreasing (up = 0)
 * order, for finite h.  Magnitudes are ordered like their bit patterns; the sign
 * bit flips the direction, and +0 and -0 both step to the smallest subnormal of
 * the stepping direction. */
static uint16_t f16_step(uint16_t h, int up) {
  uint16_t sign = h & 0x8000u, mag = h & 0x7FFFu;
  if (mag == 0) return up ? 0x0001u : 0x8001u;
  int grow = (sign == 0) == (up != 0);      /* moving away from zero */
  return (uint16_t)(sign | (grow ? mag + 1u : mag - 1u));
}

/* Down-conversion of one FP32 value into binary16 (Sec. 3 "Rounding" with FP16
 * as the low-precision domain).  Nearest: IEEE round to nearest, ties to even
 * (overflow to infinity).  Stochastic: x- <= x <= x+ are consecutive finite
 * binary16 values and x+ is taken with probability (x - x-)/(x+ - x-), i.e. when
 * u < (x - x-)/(x+ - x-) for the uniform u of this element; x beyond the largest
 * finite value (65504) saturates to it; an exactly representable x is kept; NaN
 * stays NaN. */
uint16_t orc_f16_round(float x, int stochastic, float u) {
  uint16_t h = orc_f32_to_f16_bits(x);
  if (!stochastic || isnan(x)) return h;
  if (x > 65504.0f) return 0x7BFFu;
  if (x < -65504.0f) return 0xFBFFu;
  float y = orc_f16_bits_to_f32(h);
  if (y == x) return h;
  uint16_t lo_h = y < x ? h : f16_step(h, 0);
  uint16_t hi_h = y < x ? f16_step(h, 1) : h;
  float lo = orc_f16_bits_to_f32(lo_h), hi = orc_f16_bits_to_f32(hi_h);
  return (u < (x - lo) / (hi - lo)) ? hi_h : lo_h;
}

/* ------------------------------------------------------------------------- */
/* Alg. 1 (row-wise IntN quantization with uniform min-max parameters).        */
/* ------------------------------------------------------------------------- */
void orc_quantize_row(const float *x, int d, int bits, int sb_fp16, int stochastic,
                      uint64_t seed, uint32_t step, uint32_t table, uint32_t row,
                      uint8_t *codes, float *scale_out, float *bias_out) {
  const float K = (float)((1 << bits) - 1);
  float mn = x[0], mx = x[0];
  for (int j = 1; j < d; ++j) {
    if (x[j] < mn) mn = x[j];
    if (x[j] > mx) mx = x[j];
  }
  mn = mn + 0.0f; /* a -0 minimum is stored as +0 */
  mx = mx + 0.0f;
  float s = (mx - mn) / K;
  float b = mn;
  if (sb_fp16) {
    s = orc_round_to_f16(s);
    b = orc_round_to_f16(b);
  }
  for (int j = 0; j < d; ++j) {
    float q;
    if (s == 0.0f) {
      q = 0.0f;
    } else {
      float v = (x[j] - b) / s;
      if (stochastic) {
        float f = floorf(v);
        float u = orc_uniform(seed, step, table, row, (uint32_t)j);
        q = (u < v - f) ? f + 1.0f : f;
      } else {
        q = nearbyintf(v); /* default rounding mode: nearest, ties to even */
      }
      if (q < 0.0f) q = 0.0f;
      if (q > K) q = K;
    }
    codes[j] = (uint8_t)(int)q;
  }
  *scale_out = s;
  *bias_out = b;
}

/* Dequantization: q*s + b as one fused multiply-add. */
static float dequant(uint8_t q, float s, float b) { return fmaf((float)q, s, b); }

/* ------------------------------------------------------------------------- */
/* State.                                                                      */
/* ------------------------------------------------------------------------- */
static int64_t n_sets_of(const orc_config *c, int64_t N) {
  if (c->cache_fraction <= 0.0) return 0;
  int64_t cache_rows = (int64_t)floor(c->cache_fraction * (double)N);
  int64_t s = cache_rows / c->assoc;
  return s < 1 ? 1 : s;
}

void orc_destroy(orc_t *o) {
  if (!o) return;
  if (o->tab) {
    for (int t = 0; t < o->cfg.num_tables; ++t) {
      orc_table *tb = &o->tab[t];
      free(tb->code); free(tb->h16); free(tb->scale); free(tb->bias); free(tb->crow);
      free(tb->tag); free(tb->ts); free(tb->cnt); free(tb->G);
    }
    free(o->tab);
  }
  free(o);
}

orc_t *orc_create(const orc_config *cfg, const int64_t *rows) {
  if (cfg->num_tables < 1 || cfg->dim < 1 || cfg->assoc < 1) return NULL;
  if (cfg->bits != 16 && cfg->bits != 8 && cfg->bits != 4 && cfg->bits != 2) return NULL;
  orc_t *o = (orc_t *)calloc(1, sizeof(orc_t));
  o->cfg = *cfg;
  o->tab = (orc_table *)calloc((size_t)cfg->num_tables, sizeof(orc_table));
  int d = cfg->dim;
  for (int t = 0; t < cfg->num_tables; ++t) {
    orc_table *tb = &o->tab[t];
    tb->N = rows[t];
    tb->n_sets = n_sets_of(cfg, tb->N);
    tb->slots = tb->n_sets * cfg->assoc;
    if (cfg->bits == 16) tb->h16 = (uint16_t *)calloc((size_t)(tb->N * d), sizeof(uint16_t));
    else tb->code = (uint8_t *)calloc((size_t)(tb->N * d), 1);
    tb->scale = (float *)calloc((size_t)tb->N, sizeof(float));
    tb->bias = (float *)calloc((size_t)tb->N, sizeof(float));
    tb->crow = (float *)calloc((size_t)(tb->slots * d) + 1, sizeof(float));
    tb->tag = (int32_t *)malloc(sizeof(int32_t) * (size_t)(tb->slots + 1));
    tb->ts = (int32_t *)malloc(sizeof(int32_t) * (size_t)(tb->slots + 1));
    for (int64_t k = 0; k < tb->slots; ++k) { tb->tag[k] = -1; tb->ts[k] = -1; }
    tb->cnt = (int32_t *)calloc((size_t)tb->N, sizeof(int32_t));
    tb->G = (float *)calloc((size_t)tb->N, sizeof(float));
    if (!(tb->code || tb->h16) || !tb->scale || !tb->bias || !tb->crow || !tb->tag || !tb->ts || !tb->cnt || !tb->G) {
      orc_destroy(o);
      return NULL;
    }
  }
  return o;
}

int64_t orc_geometry(const orc_t *o, int t, int64_t *n_sets, int64_t *slots) {
  *n_sets = o->tab[t].n_sets;
  *slots = o->tab[t].slots;
  return o->tab[t].N;
}

uint64_t orc_get_step(const orc_t *o) { return o->step; }
void orc_set_step(orc_t *o, uint64_t s) { o->step = s; }

/* Initial table: x_j = u*(hi-lo) + lo (fused), u the Philox uniform with step
 * word 0xFFFFFFFF and key init_seed; each row quantized with nearest rounding. */
void orc_init_uniform(orc_t *o, float lo, float hi, uint64_t init_seed) {
  int d = o->cfg.dim;
  float *x = (float *)malloc(sizeof(float) * (size_t)d);
  float width = hi - lo;
  for (int t = 0; t < o->cfg.num_tables; ++t) {
    orc_table *tb = &o->tab[t];
    for (int64_t r = 0; r < tb->N; ++r) {
      for (int j = 0; j < d; ++j)
        x[j] = fmaf(orc_uniform(init_seed, 0xFFFFFFFFu, (uint32_t)t, (uint32_t)r, (uint32_t)j), width, lo);
      if (o->cfg.bits == 16) {
        for (int j = 0; j < d; ++j) tb->h16[r * d + j] = orc_f16_round(x[j], 0, 0.0f);
      } else {
        orc_quantize_row(x, d, o->cfg.bits, o->cfg.sb_fp16, 0, 0, 0, 0, 0,
                         tb->code + r * d, &tb->scale[r], &tb->bias[r]);
      }
    }
    for (int64_t k = 0; k < tb->slots; ++k) { tb->tag[k] = -1; tb->ts[k] = -1; }
    memset(tb->crow, 0, sizeof(float) * (size_t)(tb->slots * d));
    memset(tb->cnt, 0, sizeof(int32_t) * (size_t)tb->N);
    memset(tb->G, 0, sizeof(float) * (size_t)tb->N);
  }
  free(x);
}

/* Slot index of row r in its set, or -1 when r is not resident. */
static int64_t find_slot(const orc_t *o, const orc_table *tb, int64_t r) {
  if (tb->n_sets == 0) return -1;
  int64_t s = r % tb->n_sets;
  for (int w = 0; w < o->cfg.assoc; ++w) {
    int64_t k = s * o->cfg.assoc + w;
    if (tb->tag[k] == (int32_t)r) return k;
  }
  return -1;
}

/* fetch(T,C,i): FP32 cache row if resident, else the dequantized row. */
static void fetch_row(const orc_t *o, const orc_table *tb, int64_t r, float *x) {
  int d = o->cfg.dim;
  int64_t k = find_slot(o, tb, r);
  if (k >= 0) {
    memcpy(x, tb->crow + k * d, sizeof(float) * (size_t)d);
  } else if (o->cfg.bits == 16) {
    for (int j = 0; j < d; ++j) x[j] = orc_f16_bits_to_f32(tb->h16[r * d + j]);
  } else {
    for (int j = 0; j < d; ++j) x[j] = dequant(tb->code[r * d + j], tb->scale[r], tb->bias[r]);
  }
}

/* Down-convert an FP32 row into the low-precision table T. */
static void store_low_precision(orc_t *o, int t, int64_t r, const float *x) {
  orc_table *tb = &o->tab[t];
  if (o->cfg.bits == 16) {
    for (int j = 0; j < o->cfg.dim; ++j) {
      float u = o->cfg.stochastic ? orc_uniform(o->cfg.seed, (uint32_t)o->step, (uint32_t)t, (uint32_t)r, (uint32_t)j)
                                  : 0.0f;
      tb->h16[r * o->cfg.dim + j] = orc_f16_round(x[j], o->cfg.stochastic, u);
    }
    return;
  }
  orc_quantize_row(x, o->cfg.dim, o->cfg.bits, o->cfg.sb_fp16, o->cfg.stochastic, o->cfg.seed,
                   (uint32_t)o->step, (uint32_t)t, (uint32_t)r, tb->code + r * o->cfg.dim,
                   &tb->scale[r], &tb->bias[r]);
}

/* ------------------------------------------------------------------------- */
/* Forward: out[b][t][:] = left-to-right sum of fetch() over the bag's valid    */
/* positions, first term as the seed; an empty bag gives +0.                    */
/* indices: flat int32; offsets: [T*B+1], table-major bags; out: [B][T][d].     */
/* ------------------------------------------------------------------------- */
void orc_forward(orc_t *o, const int32_t *idx, int64_t n_idx, const int32_t *off, int32_t B, float *out) {
  int T = o->cfg.num_tables, d = o->cfg.dim;
  float *x = (float *)malloc(sizeof(float) * (size_t)d);
  for (int t = 0; t < T; ++t) {
    orc_table *tb = &o->tab[t];
    tb->stat[ST_LOOKUPS] = 0;
    tb->stat[ST_HIT_LOOKUPS] = 0;
    tb->stat[ST_INVALID_FWD] = 0;
    for (int32_t b = 0; b < B; ++b) {
      float *acc = out + ((int64_t)b * T + t) * d;
      for (int j = 0; j < d; ++j) acc[j] = 0.0f;
      int first = 1;
      int64_t p0 = off[(int64_t)t * B + b], p1 = off[(int64_t)t * B + b + 1];
      if (p0 < 0) p0 = 0;
      if (p1 > n_idx) p1 = n_idx;
      for (int64_t p = p0; p < p1; ++p) {
        int64_t r = idx[p];
        if (r < 0 || r >= tb->N) { tb->stat[ST_INVALID_FWD]++; continue; }
        tb->stat[ST_LOOKUPS]++;
        if (find_slot(o, tb, r) >= 0) tb->stat[ST_HIT_LOOKUPS]++;
        fetch_row(o, tb, r, x);
        if (first) {
          for (int j = 0; j < d; ++j) acc[j] = x[j];
          first = 0;
        } else {
          for (int j = 0; j < d; ++j) acc[j] = acc[j] + x[j];
        }
      }
    }
  }
  free(x);
}

/* ------------------------------------------------------------------------- */
/* Backward + update.                                                          */
/* ------------------------------------------------------------------------- */
typedef struct { int64_t row; int64_t pos; int32_t bag; } occ_t;

static int occ_cmp(const void *a, const void *b) {
  const occ_t *x = (const occ_t *)a, *y = (const occ_t *)b;
  if (x->row != y->row) return x->row < y->row ? -1 : 1;
  if (x->pos != y->pos) return x->pos < y->pos ? -1 : 1;
  return 0;
}

typedef struct { int64_t pv; int32_t way; } victim_t;
typedef struct { int64_t pv; int64_t row; int64_t u; } cand_t;

static int victim_cmp(const void *a, const void *b) { /* PV ascending, way ascending */
  const victim_t *x = (const victim_t *)a, *y = (const victim_t *)b;
  if (x->pv != y->pv) return x->pv < y->pv ? -1 : 1;
  return x->way < y->way ? -1 : (x->way > y->way);
}
static int cand_cmp(const void *a, const void *b) { /* PV descending, row ascending */
  const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
  if (x->pv != y->pv) return x->pv > y->pv ? -1 : 1;
  return x->row < y->row ? -1 : (x->row > y->row);
}

enum { ACT_HIT_STAY = 0, ACT_HIT_EVICT = 1, ACT_INSERT = 2, ACT_BYPASS = 3 };

#define SUM_CHUNK 64        /* occurrences per chunk of a merged-gradient sum */
#define SUM_BLOCK_ABOVE 512 /* rows with more occurrences sum by bag blocks */
#define BLOCK_FLOATS 32768  /* a bag block spans 32768/d bags */

/* Returns 0, or 1 when the call is rejected: offsets that are negative, decrease,
 * or point past the end of the indices make the call change no table, cache,
 * count or accumulator (not even the LFU decay of that step); the backward
 * statistics read 0 and the step counter still advances. */
int orc_backward_update(orc_t *o, const int32_t *idx, int64_t n_idx, const int32_t *off, int32_t B,
                        const float *grad) {
  const orc_config *c = &o->cfg;
  int T = c->num_tables, d = c->dim, A = c->assoc;
  uint64_t step = o->step;

  for (int64_t i = 0; i < (int64_t)T * B; ++i) {
    if (off[i] < 0 || off[i + 1] < off[i] || off[i + 1] > n_idx) {
      for (int t = 0; t < T; ++t) {
        for (int k = ST_BWD_LOOKUPS; k <= ST_HIT_EVICTIONS; ++k) o->tab[t].stat[k] = 0;
        o->tab[t].stat[ST_INVALID_BWD] = 0;
      }
      o->step = step + 1;
      return 1;
    }
  }

  /* Decay of LFU counts: halve every count at the start of every K-th step. */
  if (c->policy == ORC_LFU && c->lfu_decay_interval > 0 && step > 0 &&
      step % (uint64_t)c->lfu_decay_interval == 0) {
    for (int t = 0; t < T; ++t)
      for (int64_t r = 0; r < o->tab[t].N; ++r) o->tab[t].cnt[r] >>= 1;
  }

  for (int t = 0; t < T; ++t) {
    orc_table *tb = &o->tab[t];
    for (int k = ST_BWD_LOOKUPS; k <= ST_HIT_EVICTIONS; ++k) tb->stat[k] = 0;
    tb->stat[ST_INVALID_BWD] = 0;

    /* 1. occurrences (row, position, bag) of the valid indices of table t */
    int64_t n_occ = 0, cap = 0;
    for (int32_t b = 0; b < B; ++b) {
      int64_t p0 = off[(int64_t)t * B + b], p1 = off[(int64_t)t * B + b + 1];
      if (p0 < 0) p0 = 0;
      if (p1 > n_idx) p1 = n_idx;
      if (p1 > p0) cap += p1 - p0;
    }
    occ_t *occ = (occ_t *)malloc(sizeof(occ_t) * (size_t)(cap + 1));
    for (int32_t b = 0; b < B; ++b) {
      int64_t p0 = off[(int64_t)t * B + b], p1 = off[(int64_t)t * B + b + 1];
      if (p0 < 0) p0 = 0;
      if (p1 > n_idx) p1 = n_idx;
      for (int64_t p = p0; p < p1; ++p) {
        int64_t r = idx[p];
        if (r < 0 || r >= tb->N) { tb->stat[ST_INVALID_BWD]++; continue; }
        occ[n_occ].row = r; occ[n_occ].pos = p; occ[n_occ].bag = b;
        ++n_occ;
      }
    }
    tb->stat[ST_BWD_LOOKUPS] = n_occ;

    /* 2. de-duplicate: sort by row, occurrences of a row in position order */
    qsort(occ, (size_t)n_occ, sizeof(occ_t), occ_cmp);
    int64_t U = 0;
    int64_t *ustart = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_occ + 1));
    for (int64_t i = 0; i < n_occ; ++i)
      if (i == 0 || occ[i].row != occ[i - 1].row) ustart[U++] = i;
    ustart[U] = n_occ;
    tb->stat[ST_UNIQUE] = U;

    int64_t *urow = (int64_t *)malloc(sizeof(int64_t) * (size_t)(U + 1));
    int64_t *uslot = (int64_t *)malloc(sizeof(int64_t) * (size_t)(U + 1));
    int *uact = (int *)malloc(sizeof(int) * (size_t)(U + 1));
    int64_t *udst = (int64_t *)malloc(sizeof(int64_t) * (size_t)(U + 1));
    float *g = (float *)malloc(sizeof(float) * (size_t)(U * d + 1));
    float *x = (float *)malloc(sizeof(float) * (size_t)(U * d + 1));
    float *part = (float *)malloc(sizeof(float) * (size_t)d);

    /* 3. merged gradient of each unique row, occurrences in position order.  Up to
     *    512 occurrences: groups of 64 consecutive occurrences (one group when there
     *    are at most 64), each summed left to right, then the group sums left to
     *    right.  More than 512: groups by bag block (bags [k*NB, (k+1)*NB) with
     *    NB = 32768/d), each non-empty group summed left to right, then the group
     *    sums left to right in block order. */
    const int32_t NB = BLOCK_FLOATS / d;
    for (int64_t u = 0; u < U; ++u) {
      urow[u] = occ[ustart[u]].row;
      float *gu = g + u * d;
      const int by_block = ustart[u + 1] - ustart[u] > SUM_BLOCK_ABOVE;
      int64_t first_chunk = 1;
      for (int64_t c0 = ustart[u], c1; c0 < ustart[u + 1]; c0 = c1) {
        if (by_block) {
          c1 = c0 + 1;
          while (c1 < ustart[u + 1] && occ[c1].bag / NB == occ[c0].bag / NB) ++c1;
        } else {
          c1 = c0 + SUM_CHUNK < ustart[u + 1] ? c0 + SUM_CHUNK : ustart[u + 1];
        }
        const float *g0 = grad + ((int64_t)occ[c0].bag * T + t) * d;
        for (int j = 0; j < d; ++j) part[j] = g0[j];
        for (int64_t i = c0 + 1; i < c1; ++i) {
          const float *gi = grad + ((int64_t)occ[i].bag * T + t) * d;
          for (int j = 0; j < d; ++j) part[j] = part[j] + gi[j];
        }
        if (first_chunk) {
          for (int j = 0; j < d; ++j) gu[j] = part[j];
          first_chunk = 0;
        } else {
          for (int j = 0; j < d; ++j) gu[j] = gu[j] + part[j];
        }
      }
    }

    /* 4. residency before the step; priority-value update (Alg. 2, first line
     *    of the loop body): LRU stamps hit slots with the step, LFU adds the
     *    row's occurrence count (saturating) */
    for (int64_t u = 0; u < U; ++u) {
      uslot[u] = find_slot(o, tb, urow[u]);
      uact[u] = uslot[u] >= 0 ? ACT_HIT_STAY : ACT_BYPASS;
      udst[u] = uslot[u];
      if (uslot[u] >= 0) tb->stat[ST_UNIQUE_HITS]++;
      if (c->policy == ORC_LRU) {
        if (uslot[u] >= 0) tb->ts[uslot[u]] = (int32_t)step;
      } else {
        int64_t nc = (int64_t)tb->cnt[urow[u]] + (ustart[u + 1] - ustart[u]);
        tb->cnt[urow[u]] = nc > INT32_MAX ? INT32_MAX : (int32_t)nc;
      }
    }

    /* 5. new FP32 value of every unique row from the pre-step state:
     *    x = fetch(T,C,r), then the optimizer step in FP32 */
    for (int64_t u = 0; u < U; ++u) {
      float *xu = x + u * d;
      const float *gu = g + u * d;
      int64_t r = urow[u];
      if (uslot[u] >= 0) {
        memcpy(xu, tb->crow + uslot[u] * d, sizeof(float) * (size_t)d);
      } else if (c->bits == 16) {
        for (int j = 0; j < d; ++j) xu[j] = orc_f16_bits_to_f32(tb->h16[r * d + j]);
      } else {
        for (int j = 0; j < d; ++j) xu[j] = dequant(tb->code[r * d + j], tb->scale[r], tb->bias[r]);
      }
      if (c->adagrad) {
        /* sum of squares by halving: a[j] += a[j + h] for h = d/2, d/4, ..., 1 */
        float *a = part;
        for (int j = 0; j < d; ++j) a[j] = gu[j] * gu[j];
        for (int h = d / 2; h >= 1; h /= 2)
          for (int j = 0; j < h; ++j) a[j] = a[j] + a[j + h];
        tb->G[r] = tb->G[r] + a[0] * (1.0f / (float)d);
        float rate = c->lr / (sqrtf(tb->G[r]) + c->eps);
        for (int j = 0; j < d; ++j) xu[j] = fmaf(-rate, gu[j], xu[j]);
      } else {
        for (int j = 0; j < d; ++j) xu[j] = fmaf(-c->lr, gu[j], xu[j]);
      }
    }

    /* 6. replacement decision per set that saw a miss (Sec. 3 policy, Alg. 2) */
    int64_t *ev_slot = (int64_t *)malloc(sizeof(int64_t) * (size_t)(U + 1));
    int64_t *ev_row = (int64_t *)malloc(sizeof(int64_t) * (size_t)(U + 1));
    int64_t n_ev = 0;
    if (tb->n_sets > 0) {
      /* group the unique rows by set: collect per set in row order */
      int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(U + 1));
      int64_t *set_of = (int64_t *)malloc(sizeof(int64_t) * (size_t)(U + 1));
      for (int64_t u = 0; u < U; ++u) { order[u] = u; set_of[u] = urow[u] % tb->n_sets; }
      /* insertion sort would be quadratic; sort indices by (set, row) via qsort on pairs */
      occ_t *tmp = (occ_t *)malloc(sizeof(occ_t) * (size_t)(U + 1));
      for (int64_t u = 0; u < U; ++u) { tmp[u].row = set_of[u]; tmp[u].pos = urow[u]; tmp[u].bag = (int32_t)u; }
      qsort(tmp, (size_t)U, sizeof(occ_t), occ_cmp);
      for (int64_t u = 0; u < U; ++u) order[u] = tmp[u].bag;
      free(tmp);

      victim_t *vic = (victim_t *)malloc(sizeof(victim_t) * (size_t)A);
      cand_t *cand = (cand_t *)malloc(sizeof(cand_t) * (size_t)(U + 1));
      int64_t i = 0;
      while (i < U) {
        int64_t s = set_of[order[i]];
        int64_t j = i;
        while (j < U && set_of[order[j]] == s) ++j;
        int64_t nm = 0;
        for (int64_t k = i; k < j; ++k) {
          int64_t u = order[k];
          if (uslot[u] < 0) {
            cand[nm].row = urow[u];
            cand[nm].u = u;
            cand[nm].pv = c->policy == ORC_LRU ? (int64_t)step : (int64_t)tb->cnt[urow[u]];
            ++nm;
          }
        }
        if (nm > 0) {
          if (A == 1 && c->policy == ORC_LRU) {
            /* direct-mapped LRU: no priority test, every missed row replaces the
             * resident in turn (rows in ascending order); the last one stays */
            int64_t k0 = s;
            int32_t old = tb->tag[k0];
            if (old >= 0) {
              tb->stat[ST_EVICTIONS]++;
              int64_t hu = -1;
              for (int64_t k = i; k < j; ++k)
                if (uslot[order[k]] == k0) hu = order[k];
              if (hu >= 0) {
                uact[hu] = ACT_HIT_EVICT;
                tb->stat[ST_HIT_EVICTIONS]++;
              } else {
                ev_slot[n_ev] = k0; ev_row[n_ev] = old; ++n_ev;
              }
            } else {
              tb->stat[ST_EMPTY_FILLS]++;
            }
            /* candidates are in row order within the set: the largest row wins */
            int64_t win = -1;
            for (int64_t k = 0; k < nm; ++k)
              if (win < 0 || cand[k].row > cand[win].row) win = k;
            for (int64_t k = 0; k < nm; ++k) {
              if (k == win) {
                uact[cand[k].u] = ACT_INSERT;
                udst[cand[k].u] = k0;
                tb->stat[ST_INSERTS]++;
              } else {
                uact[cand[k].u] = ACT_BYPASS;
                tb->stat[ST_BYPASSES]++;
              }
            }
          } else {
            for (int w = 0; w < A; ++w) {
              int64_t k0 = s * A + w;
              vic[w].way = w;
              if (tb->tag[k0] < 0) vic[w].pv = INT64_MIN;
              else if (c->policy == ORC_LRU) vic[w].pv = tb->ts[k0];
              else vic[w].pv = tb->cnt[tb->tag[k0]];
            }
            qsort(vic, (size_t)A, sizeof(victim_t), victim_cmp);
            qsort(cand, (size_t)nm, sizeof(cand_t), cand_cmp);
            int64_t k = 0;
            for (; k < nm && k < A; ++k) {
              if (!(cand[k].pv > vic[k].pv)) break;
              int64_t k0 = s * A + vic[k].way;
              int32_t old = tb->tag[k0];
              uact[cand[k].u] = ACT_INSERT;
              udst[cand[k].u] = k0;
              tb->stat[ST_INSERTS]++;
              if (old < 0) {
                tb->stat[ST_EMPTY_FILLS]++;
              } else {
                tb->stat[ST_EVICTIONS]++;
                int64_t hu = -1;
                for (int64_t q = i; q < j; ++q)
                  if (uslot[order[q]] == k0) hu = order[q];
                if (hu >= 0) {
                  uact[hu] = ACT_HIT_EVICT;
                  tb->stat[ST_HIT_EVICTIONS]++;
                } else {
                  ev_slot[n_ev] = k0; ev_row[n_ev] = old; ++n_ev;
                }
              }
            }
            for (; k < nm; ++k) {
              uact[cand[k].u] = ACT_BYPASS;
              tb->stat[ST_BYPASSES]++;
            }
          }
        }
        i = j;
      }
      free(vic); free(cand); free(order); free(set_of);
    } else {
      for (int64_t u = 0; u < U; ++u) tb->stat[ST_BYPASSES]++;
    }

    /* 7. writes.  Displaced residents that were not updated this step go to T
     *    first (their FP32 row is read before an insert overwrites the way). */
    for (int64_t e = 0; e < n_ev; ++e)
      store_low_precision(o, t, ev_row[e], tb->crow + ev_slot[e] * d);
    for (int64_t u = 0; u < U; ++u) {
      const float *xu = x + u * d;
      switch (uact[u]) {
        case ACT_HIT_STAY:
          memcpy(tb->crow + uslot[u] * d, xu, sizeof(float) * (size_t)d);
          break;
        case ACT_HIT_EVICT:
        case ACT_BYPASS:
          store_low_precision(o, t, urow[u], xu);
          break;
        case ACT_INSERT:
          memcpy(tb->crow + udst[u] * d, xu, sizeof(float) * (size_t)d);
          tb->tag[udst[u]] = (int32_t)urow[u];
          tb->ts[udst[u]] = c->policy == ORC_LRU ? (int32_t)step : -1;
          break;
      }
    }
    /* under LFU the timestamp array is unused; keep it at -1 */
    free(ev_slot); free(ev_row);
    free(occ); free(ustart); free(urow); free(uslot); free(uact); free(udst);
    free(g); free(x); free(part);
  }
  o->step = step + 1;
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Inspection.                                                                 */
/* ------------------------------------------------------------------------- */
void orc_stats(const orc_t *o, int t, int64_t *out) {
  for (int k = 0; k < ORC_NSTAT; ++k) out[k] = o->tab[t].stat[k];
}

/* Rows [row0, row0+n) of table t: codes [n][d] (one per byte; for an FP16 table
 * the binary16 bit patterns, two bytes each), scale, bias (0 for FP16), LFU counts
 * and Adagrad accumulators.  NULL outputs are skipped. */
void orc_export_rows(const orc_t *o, int t, int64_t row0, int64_t n, void *codes, float *scale,
                     float *bias, int32_t *cnt, float *G) {
  const orc_table *tb = &o->tab[t];
  int d = o->cfg.dim;
  if (codes && o->cfg.bits == 16) memcpy(codes, tb->h16 + row0 * d, sizeof(uint16_t) * (size_t)(n * d));
  else if (codes) memcpy(codes, tb->code + row0 * d, (size_t)(n * d));
  if (scale) memcpy(scale, tb->scale + row0, sizeof(float) * (size_t)n);
  if (bias) memcpy(bias, tb->bias + row0, sizeof(float) * (size_t)n);
  if (cnt) memcpy(cnt, tb->cnt + row0, sizeof(int32_t) * (size_t)n);
  if (G) memcpy(G, tb->G + row0, sizeof(float) * (size_t)n);
}

void orc_import_rows(orc_t *o, int t, int64_t row0, int64_t n, const void *codes, const float *scale,
                     const float *bias, const int32_t *cnt, const float *G) {
  orc_table *tb = &o->tab[t];
  int d = o->cfg.dim;
  if (codes && o->cfg.bits == 16) memcpy(tb->h16 + row0 * d, codes, sizeof(uint16_t) * (size_t)(n * d));
  else if (codes) memcpy(tb->code + row0 * d, codes, (size_t)(n * d));
  if (scale) memcpy(tb->scale + row0, scale, sizeof(float) * (size_t)n);
  if (bias) memcpy(tb->bias + row0, bias, sizeof(float) * (size_t)n);
  if (cnt) memcpy(tb->cnt + row0, cnt, sizeof(int32_t) * (size_t)n);
  if (G) memcpy(tb->G + row0, G, sizeof(float) * (size_t)n);
}

/* Whole cache of table t: rows [slots][d], tags [slots], LRU stamps [slots]. */
void orc_export_cache(const orc_t *o, int t, float *crow, int32_t *tag, int32_t *ts) {
  const orc_table *tb = &o->tab[t];
  int d = o->cfg.dim;
  if (crow) memcpy(crow, tb->crow, sizeof(float) * (size_t)(tb->slots * d));
  if (tag) memcpy(tag, tb->tag, sizeof(int32_t) * (size_t)tb->slots);
  if (ts) memcpy(ts, tb->ts, sizeof(int32_t) * (size_t)tb->slots);
}

void orc_import_cache(orc_t *o, int t, const float *crow, const int32_t *tag, const int32_t *ts) {
  orc_table *tb = &o->tab[t];
  int d = o->cfg.dim;
  if (crow) memcpy(tb->crow, crow, sizeof(float) * (size_t)(tb->slots * d));
  if (tag) memcpy(tb->tag, tag, sizeof(int32_t) * (size_t)tb->slots);
  if (ts) memcpy(tb->ts, ts, sizeof(int32_t) * (size_t)tb->slots);
}

/* ------------------------------------------------------------------------- */
/* Appendix "Memory Compression Factor": (M_T_lowprec + M_C + M_tags + M_cnt)  */
/* / M_T_FP32, counted in bits per embedding row.  A row of the low-precision  */
/* table costs bits*D plus 64 bits of FP32 (s,b); the cache costs ratio*32*D   */
/* and ratio*32 of INT32 tags; LFU adds one INT32 counter per row.  Without a  */
/* cache there are neither tags nor counters.                                  */
/* ------------------------------------------------------------------------- */
double orc_compression_factor(int bits, int D, double ratio, int counters, int sb_bits) {
  double row = (double)bits * D + 2.0 * sb_bits;
  double cache = ratio * 32.0 * D;
  double tags = ratio * 32.0;
  double cnt = (ratio > 0.0 && counters) ? 32.0 : 0.0;
  return (row + cache + tags + cnt) / (32.0 * D);
}
