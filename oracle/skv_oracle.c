/*
 * skv_oracle.c -- CPU oracle for the SpectrumKV per-token mixed-precision KV
 * transfer codec (arXiv 2606.08635).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, single-threaded
 * implementation of what the codec computes, written from the paper; where
 * the paper leaves a choice open, the function that makes it states the
 * reading taken.  Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load it.  It shares no code,
 * header, table or constant with the GPU library: it has its own binary16
 * conversions (written from IEEE 754), its own plan arithmetic and its own
 * payload writer and reader.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -shared -fPIC.
 * Floating point follows the C abstract machine on x86-64 (SSE2,
 * FLT_EVAL_METHOD == 0, round-to-nearest-even): every float or double
 * operation below is one correctly rounded IEEE 754 operation.
 *
 * Functions and the passages they follow:
 *   ora_plan            normalized budget (Sec. 2.1, eq. "budget"), the
 *                       budget-to-tier mapping (Sec. 4.4), sink reservation
 *                       (Sec. 4.4, Algorithm 1, scoring), the 2-tier drop rule
 *                       (Sec. 7.4.3 / probe ablation).
 *   ora_decay_table     the recency factor exp(-lambda*Delta) of eq.
 *                       "importance" (Sec. 4.3).
 *   ora_score           I_j = A_j exp(-lambda Delta_j) (Sec. 4.3) with the
 *                       KV-norm fallback or an observation-window attention
 *                       statistic (Sec. 3, Sec. 4.3).
 *   ora_assign          sink pinning + importance-sorted assignment
 *                       (Sec. 2.3 Prop. 1 "exchange argument"; Algorithm 1
 *                       steps 2-3).
 *   ora_pack            per-tier quantization of K and V, independently,
 *                       into one mixed-precision payload (Algorithm 1, transfer;
 *                       "standard symmetric" quantizer, Sec. 8).
 *   ora_unpack          decode-side dequantization into a paged fp16 cache
 *                       (Sec. 4.2, Fig. "sysarch").
 * Every parity claim of the GPU path is made against these functions.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Types and constants (the oracle's own copies; values are fixed by the      */
/* payload format, not shared with the library).                              */
/* ------------------------------------------------------------------------ */

typedef struct {
  int32_t num_layers;   /* L   */
  int32_t num_kv_heads; /* H   */
  int32_t head_dim;     /* d   */
  int32_t num_tokens;   /* n   */
  float budget;         /* b   */
  float first_ratio;    /* rho */
  int32_t num_sink;     /* -1: ceil(rho*n); >= 0: explicit */
  float decay;          /* lambda */
  int32_t num_tiers;    /* 2 or 3 */
  int32_t score_mode;   /* 0 kv-norm, 1 attention, 2 recency */
  int32_t num_q_heads;  /* attention mode */
  int32_t obs_window;   /* attention mode */
  int32_t quant_int8;   /* quantizer variant of the INT8 tier (0: row-wise symmetric, fp32 scale) */
  int32_t quant_int4;   /* quantizer variant of the INT4 tier */
} ora_config;

typedef struct {
  int32_t n_sink, n_fp16, n_int8, n_int4, n_drop;
  int64_t budget_units, used_units;
} ora_plan_t;

enum { ORA_OK = 0, ORA_ERR_INVALID_ARG = 1, ORA_ERR_BUDGET = 2,
       ORA_ERR_CAPACITY = 3, ORA_ERR_FORMAT = 4 };
enum { T_FP16 = 0, T_INT8 = 1, T_INT4 = 2, T_DROP = 3 };
enum { MODE_KVNORM = 0, MODE_ATTN = 1, MODE_RECENCY = 2 };

#define ORA_MAGIC 0x31564B53u /* bytes 'S','K','V','1' */
#define ORA_VERSION 1u
#define ORA_CHUNK 256          /* tokens per chunk-index entry */
#define ORA_MAX_TOKENS (1 << 21)

typedef unsigned __int128 u128;

static uint64_t up256(uint64_t x) { return (x + 255u) & ~(uint64_t)255u; }

/* ------------------------------------------------------------------------ */
/* binary16 <-> binary32 / binary64, written from the IEEE 754 definition.     */
/* ------------------------------------------------------------------------ */

/* Exact value of a binary16 encoding. */
double ora_half_to_double(uint16_t h) {
  int sign = h >> 15, e = (h >> 10) & 31, m = h & 1023;
  double v;
  if (e == 0) v = ldexp((double)m, -24);              /* subnormal or zero */
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexp((double)(m + 1024), e - 25);         /* (1.m) * 2^(e-15) */
  return sign ? -v : v;
}

/* Round a binary32 value to binary16, nearest-even.  NaN maps to 0x7E00. */
uint16_t ora_float_to_half(float f) {
  double x = (double)f; /* exact */
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs(x);
  if (isnan(x)) return 0x7E00;
  if (a >= 65520.0) return sign | 0x7C00;            /* rounds to infinity */
  if (a < ldexp(1.0, -14)) {                         /* subnormal range */
    double q = nearbyint(ldexp(a, 24));              /* exact scaling, RNE */
    return sign | (uint16_t)q;                       /* q==1024 -> min normal */
  }
  int E;
  (void)frexp(a, &E);               /* a = f*2^E, f in [0.5,1): exponent E-1 */
  int ex = E - 1;
  double q = nearbyint(ldexp(a, 10 - ex));           /* in [1024, 2048] */
  if (q == 2048.0) { q = 1024.0; ex += 1; }
  if (ex + 15 >= 31) return sign | 0x7C00;
  return sign | (uint16_t)(((ex + 15) << 10) | ((int)q - 1024));
}

static float half_to_float(uint16_t h) { return (float)ora_half_to_double(h); }

/* ------------------------------------------------------------------------ */
/* Quantizer variants within a tier.  The paper leaves the quantizer of each  */
/* tier open (Sec. 6.10 and Sec. 8: any per-tier scheme applies within a tier, */
/* e.g. KIVI-style asymmetric quantization; Sec. 10 on KIVI and KVQuant).  A   */
/* variant descriptor selects, per quantized tier:                             */
/*   bits 0-1  elements per scale group: 0 the whole row (d), 1 64, 2 32       */
/*             (capped at d);                                                  */
/*   bit 2     asymmetric: per group minimum lo and scale (max - min)/M, codes */
/*             0..M (M = 255 or 15), instead of symmetric absmax codes -Q..Q;  */
/*   bit 3     group scale (and minimum) stored as binary16 instead of fp32;   */
/*   bit 4     per-channel key scales (KIVI-style key quantization, Sec. 8 and */
/*             Sec. 10): the K rows of the tier inside each 256-token chunk    */
/*             form one group per channel (the chunk's rows of that tier, one  */
/*             element each), quantized with bits 2-3; V rows keep the        */
/*             per-row groups of bits 0-3.                                     */
/* Descriptor 0 is the row-wise symmetric quantizer with fp32 scales used      */
/* everywhere else in this file.                                               */
/* ------------------------------------------------------------------------ */

enum { QV_ASYM = 4, QV_FP16 = 8, QV_CHANNEL = 16 };

static int qv_valid(int32_t q) { return (q & ~31) == 0 && (q & 3) != 3; }

static int32_t qv_group(int32_t q, int32_t d) {
  int32_t g = (q & 3) == 0 ? d : (q & 3) == 1 ? 64 : 32;
  return g < d ? g : d;
}

/* Bytes of one group's metadata (s, then lo if asymmetric). */
static uint64_t qv_group_entry(int32_t q) { return ((q & QV_ASYM) ? 2u : 1u) * ((q & QV_FP16) ? 2u : 4u); }

/* Per-row metadata bytes of one quantized row under descriptor q (the row's
 * groups); K rows of a per-channel tier carry none (is_k). */
static uint64_t qv_entry_bytes(int32_t q, int32_t d) {
  return (uint64_t)(d / qv_group(q, d)) * qv_group_entry(q);
}
static uint64_t qv_row_bytes(int32_t q, int32_t d, int is_k) {
  return (is_k && (q & QV_CHANNEL)) ? 0u : qv_entry_bytes(q, d);
}

/* ------------------------------------------------------------------------ */
/* Validation and plan (Sec. 2.1 eq. "budget"; Sec. 4.4).                      */
/* ------------------------------------------------------------------------ */

static int valid_head_dim(int d) { return d == 32 || d == 64 || d == 128 || d == 256; }

int ora_validate(const ora_config* c) {
  if (!c) return ORA_ERR_INVALID_ARG;
  if (c->num_layers < 1 || c->num_kv_heads < 1) return ORA_ERR_INVALID_ARG;
  if (!valid_head_dim(c->head_dim)) return ORA_ERR_INVALID_ARG;
  if (c->num_tokens < 1 || c->num_tokens > ORA_MAX_TOKENS) return ORA_ERR_INVALID_ARG;
  if ((int64_t)c->num_layers * c->num_kv_heads > 65536) return ORA_ERR_INVALID_ARG;
  if (!(c->budget > 0.0f && c->budget <= 1.0f)) return ORA_ERR_INVALID_ARG;
  if (!(c->first_ratio >= 0.0f && c->first_ratio <= 1.0f)) return ORA_ERR_INVALID_ARG;
  if (c->num_sink < -1) return ORA_ERR_INVALID_ARG;
  if (!(c->decay >= 0.0f) || isinf(c->decay)) return ORA_ERR_INVALID_ARG;
  if (2.0 * (double)c->decay * (double)(c->num_tokens - 1) > 700.0) return ORA_ERR_INVALID_ARG;
  if (c->num_tiers != 2 && c->num_tiers != 3) return ORA_ERR_INVALID_ARG;
  if (c->score_mode < MODE_KVNORM || c->score_mode > MODE_RECENCY) return ORA_ERR_INVALID_ARG;
  if (!qv_valid(c->quant_int8) || !qv_valid(c->quant_int4)) return ORA_ERR_INVALID_ARG;
  if (c->score_mode == MODE_ATTN) {
    if (c->num_q_heads < 1 || c->num_q_heads % c->num_kv_heads != 0) return ORA_ERR_INVALID_ARG;
    if (c->obs_window < 1) return ORA_ERR_INVALID_ARG;
    if ((c->num_q_heads / c->num_kv_heads) * c->obs_window > 256) return ORA_ERR_INVALID_ARG;
  }
  return ORA_OK;
}

/* Tier counts.  Costs in quarter units: fp16 4, int8 2, int4 1, drop 0, so the
 * normalized budget b (eq. "budget") becomes the integer B = floor(4 b n). */
int ora_plan(const ora_config* c, ora_plan_t* p) {
  int st = ora_validate(c);
  if (st) return st;
  int64_t n = c->num_tokens;
  int64_t s;
  if (c->num_sink >= 0) s = c->num_sink < n ? c->num_sink : n;
  else {
    double want = ceil((double)c->first_ratio * (double)n); /* exact product */
    s = want < (double)n ? (int64_t)want : n;
  }
  int64_t B = (int64_t)floor(4.0 * (double)c->budget * (double)n); /* exact */
  if (4 * s > B) return ORA_ERR_BUDGET;
  int64_t m = n - s, R = B - 4 * s;
  int64_t n16 = 0, n8 = 0, n4 = 0, nd = 0;
  if (R >= 2 * m) {                       /* b' >= 1/2: f16 = 2b'-1, f8 = 2-2b' */
    n16 = (R - 2 * m) / 2;
    n8 = m - n16;
  } else if (c->num_tiers == 3 && R >= m) { /* 1/4 <= b' < 1/2: f8 = 4b'-1, f4 = 2-4b' */
    n8 = R - m;
    n4 = 2 * m - R;
  } else if (c->num_tiers == 3) {          /* b' < 1/4: int4 first, drop the rest */
    n4 = R;
    nd = m - R;
  } else {                                 /* 2-tier: int8 lowest, drop the rest */
    n8 = R / 2;
    nd = m - n8;
  }
  if (p) {
    p->n_sink = (int32_t)s; p->n_fp16 = (int32_t)n16; p->n_int8 = (int32_t)n8;
    p->n_int4 = (int32_t)n4; p->n_drop = (int32_t)nd;
    p->budget_units = B;
    p->used_units = 4 * (s + n16) + 2 * n8 + n4;
  }
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Payload geometry (format version 1, little-endian).                         */
/* ------------------------------------------------------------------------ */

typedef struct {
  uint64_t tiermap_off, chunkidx_off, layers_off;
  uint64_t seg_bytes, seg_stride, scales_bytes, layer_stride, total;
  int64_t nq, nchunks;
  uint64_t e8, e4;            /* per-row metadata bytes of a V row (INT8 / INT4) */
  uint64_t ek8, ek4;          /* the same for a K row (0 for a per-channel tier) */
  uint64_t seg_scale_bytes;   /* per-row metadata of one V segment: n8 e8 + n4 e4 */
  uint64_t seg_scale_bytes_k; /* the same for a K segment: n8 ek8 + n4 ek4 */
  uint64_t chan_block;        /* per-channel parameters of one (head, chunk) */
  uint64_t channel_bytes;     /* the layer's per-channel area (256-aligned) */
  uint64_t cidx_entry;        /* chunk-index entry bytes: 8 (both descriptors 0) or 16 */
} ora_geom;

static void geometry(const ora_config* c, const ora_plan_t* p, ora_geom* g) {
  uint64_t n = (uint64_t)c->num_tokens, d = (uint64_t)c->head_dim, H = (uint64_t)c->num_kv_heads;
  g->nq = p->n_int8 + p->n_int4;
  g->nchunks = (int64_t)((n + ORA_CHUNK - 1) / ORA_CHUNK);
  g->e8 = qv_row_bytes(c->quant_int8, (int32_t)d, 0);
  g->e4 = qv_row_bytes(c->quant_int4, (int32_t)d, 0);
  g->ek8 = qv_row_bytes(c->quant_int8, (int32_t)d, 1);
  g->ek4 = qv_row_bytes(c->quant_int4, (int32_t)d, 1);
  g->seg_scale_bytes = (uint64_t)p->n_int8 * g->e8 + (uint64_t)p->n_int4 * g->e4;
  g->seg_scale_bytes_k = (uint64_t)p->n_int8 * g->ek8 + (uint64_t)p->n_int4 * g->ek4;
  g->chan_block = ((c->quant_int8 & QV_CHANNEL) ? d * qv_group_entry(c->quant_int8) : 0u) +
                  ((c->quant_int4 & QV_CHANNEL) ? d * qv_group_entry(c->quant_int4) : 0u);
  g->channel_bytes = up256(H * (uint64_t)g->nchunks * g->chan_block);
  g->cidx_entry = (c->quant_int8 || c->quant_int4) ? 16u : 8u;
  g->tiermap_off = 256;
  g->chunkidx_off = g->tiermap_off + up256((n + 3) / 4);
  g->layers_off = g->chunkidx_off + up256((uint64_t)g->nchunks * g->cidx_entry);
  g->seg_bytes = (uint64_t)(p->n_sink + p->n_fp16) * 2 * d + (uint64_t)p->n_int8 * d +
                 (uint64_t)p->n_int4 * (d / 2);
  g->seg_stride = up256(g->seg_bytes);
  g->scales_bytes = up256(H * (g->seg_scale_bytes_k + g->seg_scale_bytes));
  g->layer_stride = g->scales_bytes + g->channel_bytes + 2 * H * g->seg_stride;
  g->total = g->layers_off + (uint64_t)c->num_layers * g->layer_stride;
}

int ora_payload_size(const ora_config* c, uint64_t* bytes) {
  ora_plan_t p;
  int st = ora_plan(c, &p);
  if (st) return st;
  ora_geom g;
  geometry(c, &p, &g);
  *bytes = g.total;
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Recency factor (Sec. 4.3, eq. "importance"): Delta = n-1-t for 0-based t.   */
/* which == 1: exp(-lambda*Delta); which == 2: exp(-2*lambda*Delta).           */
/* ------------------------------------------------------------------------ */

void ora_decay_table(float decay, int which, int32_t count, double* out) {
  double lam = (double)decay * (which == 2 ? 2.0 : 1.0);
  for (int32_t dlt = 0; dlt < count; ++dlt) out[dlt] = exp(-(lam * (double)dlt));
}

/* ------------------------------------------------------------------------ */
/* Scores (Sec. 4.3).                                                          */
/* ------------------------------------------------------------------------ */

/* (x * 2^24)^2 as an exact integer for a finite binary16 x; 0 for inf/NaN. */
static u128 square_units(uint16_t h) {
  int e = (h >> 10) & 31, m = h & 1023;
  if (e == 31) return 0;
  uint64_t mant = e ? (uint64_t)(m + 1024) : (uint64_t)m;
  int sh = e ? e - 1 : 0;
  u128 X = (u128)mant << sh;
  return X * X;
}

/* Exact S_t = sum over layers, heads, K and V, and channels of x^2, in units
 * of 2^-48, returned as two 64-bit halves. */
int ora_sumsq(const ora_config* c, const uint16_t* k, const uint16_t* v, int32_t t,
              uint64_t* hi, uint64_t* lo) {
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  u128 S = 0;
  for (int64_t l = 0; l < L; ++l)
    for (int64_t h = 0; h < H; ++h) {
      const uint16_t* kr = k + (((l * H + h) * n + t) * d);
      const uint16_t* vr = v + (((l * H + h) * n + t) * d);
      for (int64_t i = 0; i < d; ++i) S += square_units(kr[i]) + square_units(vr[i]);
    }
  *hi = (uint64_t)(S >> 64);
  *lo = (uint64_t)S;
  return ORA_OK;
}

/* The exact values of `count` binary16 elements (a key plane is decoded once
 * and read by every query of the heads that share it). */
static void decode_plane(const uint16_t* src, int64_t count, double* out) {
  for (int64_t i = 0; i < count; ++i) out[i] = ora_half_to_double(src[i]);
}

/* Mean attention mass of every key over the observation queries of all layers
 * and query heads (Sec. 3: aggregate over layers, heads and decode
 * observations; Sec. 4.3: A_j observed or approximated).  Binary64 throughout.
 * Query head hq reads KV head hq / (Hq/H).  No causal mask: the observation
 * queries stand for decode steps, which see every prompt token. */
static void attention_mass(const ora_config* c, const uint16_t* k, const uint16_t* q, double* A) {
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  int64_t Hq = c->num_q_heads, W = c->obs_window, grp = Hq / H;
  double inv_sqrt_d = 1.0 / sqrt((double)d);
  double* z = (double*)malloc((size_t)n * sizeof(double));
  double* qv = (double*)malloc((size_t)d * sizeof(double));
  double* kv = (double*)malloc((size_t)(n * d) * sizeof(double));
  for (int64_t t = 0; t < n; ++t) A[t] = 0.0;
  for (int64_t l = 0; l < L; ++l)
    for (int64_t hq = 0; hq < Hq; ++hq) {
      int64_t h = hq / grp;
      if (hq % grp == 0) decode_plane(k + (l * H + h) * n * d, n * d, kv);
      for (int64_t w = 0; w < W; ++w) {
        const uint16_t* qr = q + ((l * Hq + hq) * W + w) * d;
        for (int64_t i = 0; i < d; ++i) qv[i] = ora_half_to_double(qr[i]);
        double zmax = -INFINITY;
        for (int64_t t = 0; t < n; ++t) {
          const double* kr = kv + t * d;
          double dot = 0.0;
          for (int64_t i = 0; i < d; ++i) dot += qv[i] * kr[i];
          z[t] = dot * inv_sqrt_d;
          if (z[t] > zmax) zmax = z[t];
        }
        double den = 0.0;
        for (int64_t t = 0; t < n; ++t) { z[t] = exp(z[t] - zmax); den += z[t]; }
        for (int64_t t = 0; t < n; ++t) A[t] += z[t] / den;
      }
    }
  double count = (double)(L * Hq * W);
  for (int64_t t = 0; t < n; ++t) A[t] /= count;
  free(z);
  free(qv);
  free(kv);
}

/* key[t] for every token.  KV-norm mode ranks by I_t^2 = ||KV_t||^2 e^{-2 lambda Delta}
 * (same order as I_t = ||KV_t|| e^{-lambda Delta}); attention mode by
 * A_t e^{-lambda Delta}; recency mode by e^{-lambda Delta} (A = 1). */
int ora_score(const ora_config* c, const uint16_t* k, const uint16_t* v, const uint16_t* q,
              double* key) {
  int st = ora_validate(c);
  if (st) return st;
  int32_t n = c->num_tokens;
  double* w = (double*)malloc((size_t)n * sizeof(double));
  if (c->score_mode == MODE_KVNORM) {
    ora_decay_table(c->decay, 2, n, w);
    for (int32_t t = 0; t < n; ++t) {
      uint64_t hi, lo;
      ora_sumsq(c, k, v, t, &hi, &lo);
      u128 S = ((u128)hi << 64) | lo;
      double s = ldexp((double)S, -48);  /* one rounding (u128 -> double), exact scaling */
      key[t] = s * w[n - 1 - t];
    }
  } else if (c->score_mode == MODE_ATTN) {
    if (!q) { free(w); return ORA_ERR_INVALID_ARG; }
    ora_decay_table(c->decay, 1, n, w);
    double* A = (double*)malloc((size_t)n * sizeof(double));
    attention_mass(c, k, q, A);
    for (int32_t t = 0; t < n; ++t) key[t] = A[t] * w[n - 1 - t];
    free(A);
  } else {
    ora_decay_table(c->decay, 1, n, w);
    for (int32_t t = 0; t < n; ++t) key[t] = w[n - 1 - t];
  }
  free(w);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Tier assignment (Sec. 2.3 Prop. 1; Algorithm 1, scoring and tier assignment).                  */
/* ------------------------------------------------------------------------ */

/* Ranking key: the score's binary64 pattern cut to 32 fraction bits, with the
 * token index below it, so equal (cut) scores rank the more recent token
 * higher.  Scores that are NaN or not positive rank as +0. */
uint64_t ora_composite(double key, int32_t t) {
  uint64_t bits = 0;
  if (key > 0.0) memcpy(&bits, &key, 8);
  return ((bits >> 20) << 21) | (uint64_t)(uint32_t)t;
}

static int desc_u64(const void* a, const void* b) {
  uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
  return x < y ? 1 : (x > y ? -1 : 0);
}

int ora_assign(const ora_config* c, const double* key, uint8_t* tier) {
  ora_plan_t p;
  int st = ora_plan(c, &p);
  if (st) return st;
  int32_t n = c->num_tokens, s = p.n_sink, m = n - s;
  for (int32_t t = 0; t < s; ++t) tier[t] = T_FP16; /* sinks pinned before ranking */
  uint64_t* cs = (uint64_t*)malloc((size_t)(m > 0 ? m : 1) * sizeof(uint64_t));
  for (int32_t t = s; t < n; ++t) cs[t - s] = ora_composite(key[t], t);
  qsort(cs, (size_t)m, sizeof(uint64_t), desc_u64);
  for (int32_t r = 0; r < m; ++r) {
    int32_t t = (int32_t)(cs[r] & ((1u << 21) - 1));
    uint8_t tr;
    if (r < p.n_fp16) tr = T_FP16;
    else if (r < p.n_fp16 + p.n_int8) tr = T_INT8;
    else if (r < p.n_fp16 + p.n_int8 + p.n_int4) tr = T_INT4;
    else tr = T_DROP;
    tier[t] = tr;
  }
  free(cs);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Row offsets and row codec.                                                  */
/* ------------------------------------------------------------------------ */

static int width_units(int tr) { return tr == T_FP16 ? 4 : tr == T_INT8 ? 2 : tr == T_INT4 ? 1 : 0; }

/* units[t] = sum over u < t of the row width in units of d/2 bytes;
 * qrank[t] = number of quantized (int8/int4) rows before t. */
void ora_offsets(int32_t n, const uint8_t* tier, uint32_t* units, uint32_t* qrank) {
  uint32_t u = 0, q = 0;
  for (int32_t t = 0; t < n; ++t) {
    units[t] = u;
    qrank[t] = q;
    u += (uint32_t)width_units(tier[t]);
    q += (tier[t] == T_INT8 || tier[t] == T_INT4);
  }
}

/* sbytes[t] = metadata bytes of the quantized rows before t (e8 per INT8
 * row, e4 per INT4 row): where row t's scales start inside its segment's
 * metadata. */
void ora_scale_offsets(int32_t n, const uint8_t* tier, uint64_t e8, uint64_t e4, uint32_t* sbytes) {
  uint64_t b = 0;
  for (int32_t t = 0; t < n; ++t) {
    sbytes[t] = (uint32_t)b;
    b += tier[t] == T_INT8 ? e8 : tier[t] == T_INT4 ? e4 : 0;
  }
}

/* Symmetric per-row absmax quantizer ("standard symmetric", Sec. 8).  Writes
 * the row's payload bytes to out and its scale to *scale; returns 1 if the
 * row holds a non-finite element (scale NaN, codes zero), else 0. */
int ora_encode_row(int tr, int32_t d, const uint16_t* x, uint8_t* out, float* scale) {
  if (tr == T_FP16) {
    for (int32_t i = 0; i < d; ++i) { out[2 * i] = (uint8_t)x[i]; out[2 * i + 1] = (uint8_t)(x[i] >> 8); }
    return 0;
  }
  if (tr == T_DROP) return 0;
  const int Q = tr == T_INT8 ? 127 : 7;
  uint16_t amax = 0;
  for (int32_t i = 0; i < d; ++i) {
    uint16_t mag = x[i] & 0x7FFF;
    if (mag > amax) amax = mag;
  }
  int32_t codes[256];
  int bad = 0;
  if (amax >= 0x7C00) {                 /* inf or NaN somewhere in the row */
    uint32_t nanbits = 0x7FC00000u;
    memcpy(scale, &nanbits, 4);
    for (int32_t i = 0; i < d; ++i) codes[i] = 0;
    bad = 1;
  } else if (amax == 0) {
    *scale = 0.0f;
    for (int32_t i = 0; i < d; ++i) codes[i] = 0;
  } else {
    float a = half_to_float(amax);
    *scale = a / (float)Q;
    float r = (float)Q / a;
    for (int32_t i = 0; i < d; ++i) {
      float y = half_to_float(x[i]) * r;
      float c = nearbyintf(y);
      if (c > (float)Q) c = (float)Q;
      if (c < (float)-Q) c = (float)-Q;
      codes[i] = (int32_t)c;
    }
  }
  if (tr == T_INT8) {
    for (int32_t i = 0; i < d; ++i) out[i] = (uint8_t)(codes[i] & 0xFF);
  } else {
    for (int32_t i = 0; i < d / 2; ++i)
      out[i] = (uint8_t)((codes[2 * i] & 0xF) | ((codes[2 * i + 1] & 0xF) << 4));
  }
  return bad;
}

/* Inverse of ora_encode_row: fp16 bits of the reconstructed row. */
void ora_decode_row(int tr, int32_t d, const uint8_t* in, float scale, uint16_t* y) {
  if (tr == T_FP16) {
    for (int32_t i = 0; i < d; ++i) y[i] = (uint16_t)(in[2 * i] | (in[2 * i + 1] << 8));
    return;
  }
  if (tr == T_DROP) {
    for (int32_t i = 0; i < d; ++i) y[i] = 0;
    return;
  }
  if (isnan(scale)) {
    for (int32_t i = 0; i < d; ++i) y[i] = 0x7E00;
    return;
  }
  for (int32_t i = 0; i < d; ++i) {
    int32_t code;
    if (tr == T_INT8) code = (int32_t)(int8_t)in[i];
    else {
      int32_t nib = (in[i / 2] >> (4 * (i & 1))) & 0xF;
      code = nib >= 8 ? nib - 16 : nib;
    }
    y[i] = ora_float_to_half((float)code * scale);
  }
}

static void put32(uint8_t* p, uint32_t v);
static uint32_t get32(const uint8_t* p);
static uint32_t fbits(float f);

/* Order key of a binary16 pattern that sorts finite values numerically with
 * -0 below +0 (IEEE totalOrder restricted to finite values). */
static uint32_t order_key(uint16_t h) { return (h & 0x8000u) ? (uint32_t)(~h & 0xFFFFu) : (uint32_t)(h | 0x8000u); }

static void put16(uint8_t* p, uint16_t v) { memcpy(p, &v, 2); }
static uint16_t get16(const uint8_t* p) { uint16_t v; memcpy(&v, p, 2); return v; }

/* One quantization group under descriptor q's bits 2-3 (tier tr): the cnt
 * binary16 values x[0], x[stride], ...  Writes the codes to codes[0..cnt) and
 * the group's metadata (s, then lo if asymmetric; fp32 or binary16) at m.
 *   symmetric: a = max |x|; a non-finite element gives a NaN scale and zero
 *     codes, a = 0 a zero scale and zero codes; otherwise with an fp32 scale
 *     s = RN32(a/Q), r = RN32(Q/a), and with a binary16 scale s = RN16(RN32(a/Q))
 *     (zero codes if that underflows to 0), r = RN32(1/s);
 *     code = clamp(rne(RN32(x r)), -Q, Q).
 *   asymmetric: lo = min x, hi = max x (-0 below +0); non-finite gives NaN
 *     scale and minimum and zero codes; range = RN32(hi - lo); range = 0 gives
 *     a zero scale and zero codes; otherwise s = RN32(range/M) (binary16: RN16
 *     of that, zero codes on underflow), r = RN32(M/range) (binary16:
 *     RN32(1/s)); code = clamp(rne(RN32(RN32(x - lo) r)), 0, M).
 * Returns 1 if the group held a non-finite element. */
static int quant_group(int tr, int32_t q, const uint16_t* x, int64_t stride, int64_t cnt, int32_t* codes,
                       uint8_t* m) {
  const int asym = (q & QV_ASYM) != 0, f16 = (q & QV_FP16) != 0;
  const int Q = tr == T_INT8 ? 127 : 7, M = tr == T_INT8 ? 255 : 15;
  int bad = 0;
  uint16_t amax = 0, lo = x[0], hi = x[0];
  for (int64_t i = 0; i < cnt; ++i) {
    uint16_t v = x[i * stride];
    if ((v & 0x7C00u) == 0x7C00u) bad = 1;
    if ((v & 0x7FFFu) > amax) amax = v & 0x7FFFu;
    if (order_key(v) < order_key(lo)) lo = v;
    if (order_key(v) > order_key(hi)) hi = v;
  }
  float scale = 0.0f, r = 0.0f, lof = 0.0f;
  uint16_t s16 = 0;
  int zero = 0;
  if (bad) {
    uint32_t nanbits = 0x7FC00000u;
    memcpy(&scale, &nanbits, 4);
    memcpy(&lof, &nanbits, 4);
    s16 = 0x7E00;
    zero = 1;
  } else if (!asym) {
    if (amax == 0) {
      zero = 1;
    } else {
      float a = half_to_float(amax);
      scale = a / (float)Q;
      if (f16) {
        s16 = ora_float_to_half(scale);
        scale = half_to_float(s16);
        if (s16 == 0) zero = 1;
        else r = 1.0f / scale;
      } else {
        r = (float)Q / a;
      }
    }
  } else {
    lof = half_to_float(lo);
    float range = half_to_float(hi) - lof;
    if (range == 0.0f) {
      zero = 1;
    } else {
      scale = range / (float)M;
      if (f16) {
        s16 = ora_float_to_half(scale);
        scale = half_to_float(s16);
        if (s16 == 0) zero = 1;
        else r = 1.0f / scale;
      } else {
        r = (float)M / range;
      }
    }
  }
  for (int64_t i = 0; i < cnt; ++i) {
    if (zero) { codes[i] = 0; continue; }
    float c, xv = half_to_float(x[i * stride]);
    if (!asym) {
      c = nearbyintf(xv * r);
      if (c > (float)Q) c = (float)Q;
      if (c < (float)-Q) c = (float)-Q;
    } else {
      float dlt = xv - lof;
      c = nearbyintf(dlt * r);
      if (c > (float)M) c = (float)M;
      if (c < 0.0f) c = 0.0f;
    }
    codes[i] = (int32_t)c;
  }
  if (f16) {
    put16(m, bad ? (uint16_t)0x7E00 : s16);
    if (asym) put16(m + 2, bad ? (uint16_t)0x7E00 : lo);
  } else {
    put32(m, fbits(scale));
    if (asym) put32(m + 4, fbits(lof));
  }
  return bad;
}

/* One quantization group of cnt contiguous values (exported for tests): codes
 * and the group's metadata entry, as quant_group. */
int ora_quant_group(int tr, int32_t q, int64_t cnt, const uint16_t* x, int32_t* codes, uint8_t* meta) {
  return quant_group(tr, q, x, 1, cnt, codes, meta);
}

/* Stores d codes of tier tr: a byte each (INT8), or two nibbles per byte,
 * even element in the low nibble (INT4). */
static void store_codes(int tr, int32_t d, const int32_t* codes, uint8_t* out) {
  if (tr == T_INT8) {
    for (int32_t i = 0; i < d; ++i) out[i] = (uint8_t)(codes[i] & 0xFF);
  } else {
    for (int32_t i = 0; i < d / 2; ++i)
      out[i] = (uint8_t)((codes[2 * i] & 0xF) | ((codes[2 * i + 1] & 0xF) << 4));
  }
}

/* Row quantizer under variant descriptor q (see the variant section above):
 * the row's groups of qv_group(q, d) elements, each by quant_group.  Codes are
 * stored as for descriptor 0 (signed byte / nibble), asymmetric codes as
 * unsigned byte / nibble.  Metadata: per group s, then lo if asymmetric.
 * Returns 1 if a group held a non-finite element.  Descriptor 0 is
 * ora_encode_row with its fp32 scale in the metadata.  Bit 4 (per-channel K)
 * does not enter a row's own quantization. */
int ora_encode_row_q(int tr, int32_t q, int32_t d, const uint16_t* x, uint8_t* out, uint8_t* meta) {
  q &= ~QV_CHANNEL;
  if (tr == T_FP16 || tr == T_DROP || q == 0) {
    float scale = 0.0f;
    int bad = ora_encode_row(tr, d, x, out, &scale);
    if (tr == T_INT8 || tr == T_INT4) put32(meta, fbits(scale));
    return bad;
  }
  const int32_t gs = qv_group(q, d);
  int32_t codes[256];
  int bad_any = 0;
  for (int32_t g0 = 0; g0 < d; g0 += gs)
    bad_any |= quant_group(tr, q, x + g0, 1, gs, codes + g0, meta + (uint64_t)(g0 / gs) * qv_group_entry(q));
  store_codes(tr, d, codes, out);
  return bad_any;
}

/* Decodes one code of tier tr under descriptor bits 2 (asymmetric) with the
 * group's s and lo: a NaN s gives 0x7E00; symmetric x^ = RN16(RN32(code s));
 * asymmetric x^ = RN16(RN32(RN32(code s) + lo)).  raw is the stored byte
 * (INT8) or nibble (INT4). */
static uint16_t decode_code(int tr, int asym, uint32_t raw, float scale, float lo) {
  if (isnan(scale)) return 0x7E00;
  int32_t code = asym ? (int32_t)raw
                      : tr == T_INT8 ? (int32_t)(int8_t)(uint8_t)raw : ((int32_t)raw >= 8 ? (int32_t)raw - 16 : (int32_t)raw);
  float v = (float)code * scale;
  if (asym) v = v + lo;
  return ora_float_to_half(v);
}

/* Inverse of ora_encode_row_q: per group, decode_code with the group's s, lo. */
void ora_decode_row_q(int tr, int32_t q, int32_t d, const uint8_t* in, const uint8_t* meta, uint16_t* y) {
  q &= ~QV_CHANNEL;
  if (tr == T_FP16 || tr == T_DROP || q == 0) {
    float scale = 0.0f;
    if (tr == T_INT8 || tr == T_INT4) {
      uint32_t b = get32(meta);
      memcpy(&scale, &b, 4);
    }
    ora_decode_row(tr, d, in, scale, y);
    return;
  }
  const int asym = (q & QV_ASYM) != 0, f16 = (q & QV_FP16) != 0;
  const int32_t gs = qv_group(q, d);
  for (int32_t g0 = 0; g0 < d; g0 += gs) {
    const uint8_t* m = meta + (uint64_t)(g0 / gs) * qv_group_entry(q);
    float scale, lo = 0.0f;
    if (f16) {
      scale = half_to_float(get16(m));
      if (asym) lo = half_to_float(get16(m + 2));
    } else {
      uint32_t b = get32(m);
      memcpy(&scale, &b, 4);
      if (asym) { b = get32(m + 4); memcpy(&lo, &b, 4); }
    }
    for (int32_t i = g0; i < g0 + gs; ++i) {
      uint32_t raw = tr == T_INT8 ? in[i] : (uint32_t)(in[i / 2] >> (4 * (i & 1))) & 0xFu;
      y[i] = decode_code(tr, asym, raw, scale, lo);
    }
  }
}

/* Decodes a per-channel K row: element i with channel i's entry (s, then lo)
 * in blk, by decode_code. */
void ora_decode_row_channel(int tr, int32_t q, int32_t d, const uint8_t* in, const uint8_t* blk, uint16_t* y) {
  const int asym = (q & QV_ASYM) != 0, f16 = (q & QV_FP16) != 0;
  for (int32_t i = 0; i < d; ++i) {
    const uint8_t* m = blk + (uint64_t)i * qv_group_entry(q);
    float scale, lo = 0.0f;
    if (f16) {
      scale = half_to_float(get16(m));
      if (asym) lo = half_to_float(get16(m + 2));
    } else {
      uint32_t b = get32(m);
      memcpy(&scale, &b, 4);
      if (asym) { b = get32(m + 4); memcpy(&lo, &b, 4); }
    }
    uint32_t raw = tr == T_INT8 ? in[i] : (uint32_t)(in[i / 2] >> (4 * (i & 1))) & 0xFu;
    y[i] = decode_code(tr, asym, raw, scale, lo);
  }
}

/* ------------------------------------------------------------------------ */
/* Payload writer (Algorithm 1, transfer) and reader (decode side, Sec. 4.2).     */
/* ------------------------------------------------------------------------ */

static void put32(uint8_t* p, uint32_t v) { memcpy(p, &v, 4); }
static void put64(uint8_t* p, uint64_t v) { memcpy(p, &v, 8); }
static uint32_t get32(const uint8_t* p) { uint32_t v; memcpy(&v, p, 4); return v; }
static uint32_t fbits(float f) { uint32_t v; memcpy(&v, &f, 4); return v; }

static void write_header(const ora_config* c, const ora_plan_t* p, const ora_geom* g, uint8_t* h) {
  memset(h, 0, 256);
  put32(h + 0, ORA_MAGIC);
  put32(h + 4, ORA_VERSION);
  put32(h + 8, (uint32_t)c->num_layers);
  put32(h + 12, (uint32_t)c->num_kv_heads);
  put32(h + 16, (uint32_t)c->head_dim);
  put32(h + 20, (uint32_t)c->num_tokens);
  put32(h + 24, (uint32_t)p->n_sink);
  put32(h + 28, (uint32_t)c->num_tiers);
  put32(h + 32, fbits(c->budget));
  put32(h + 36, fbits(c->first_ratio));
  put32(h + 40, fbits(c->decay));
  put32(h + 44, (uint32_t)c->score_mode);
  put32(h + 48, (uint32_t)p->n_fp16);
  put32(h + 52, (uint32_t)p->n_int8);
  put32(h + 56, (uint32_t)p->n_int4);
  put32(h + 60, (uint32_t)p->n_drop);
  put64(h + 64, (uint64_t)p->budget_units);
  put64(h + 72, (uint64_t)p->used_units);
  put64(h + 80, g->tiermap_off);
  put64(h + 88, g->chunkidx_off);
  put64(h + 96, g->layers_off);
  put64(h + 104, g->seg_bytes);
  put64(h + 112, g->seg_stride);
  put64(h + 120, g->scales_bytes);
  put64(h + 128, g->layer_stride);
  put64(h + 136, g->total);
  put32(h + 144, 0);             /* non-finite quantized rows */
  put32(h + 148, 0);             /* status */
  put32(h + 152, ORA_CHUNK);
  put32(h + 156, (uint32_t)c->quant_int8);
  put32(h + 160, (uint32_t)c->quant_int4);
  put64(h + 168, g->channel_bytes);
}

static int any_channel(const ora_config* c) { return ((c->quant_int8 | c->quant_int4) & QV_CHANNEL) != 0; }

/* Header, 2-bit tier map and chunk index (the payload bytes before layer 0);
 * also returns the per-token row offsets, scale ranks and per-row metadata
 * offsets of V segments (sbytes) and K segments (sbytes_k). */
static void write_meta(const ora_config* c, const ora_plan_t* p, const ora_geom* g, const uint8_t* tier,
                       uint32_t* units, uint32_t* qrank, uint32_t* sbytes, uint32_t* sbytes_k, uint8_t* payload) {
  int64_t n = c->num_tokens;
  write_header(c, p, g, payload);
  for (int64_t t = 0; t < n; ++t)
    payload[g->tiermap_off + (uint64_t)t / 4] |= (uint8_t)(tier[t] << (2 * (t % 4)));
  ora_offsets((int32_t)n, tier, units, qrank);
  ora_scale_offsets((int32_t)n, tier, g->e8, g->e4, sbytes);
  ora_scale_offsets((int32_t)n, tier, g->ek8, g->ek4, sbytes_k);
  for (int64_t ch = 0; ch < g->nchunks; ++ch) {
    uint8_t* e = payload + g->chunkidx_off + g->cidx_entry * (uint64_t)ch;
    put32(e, units[ch * ORA_CHUNK]);
    put32(e + 4, qrank[ch * ORA_CHUNK]);
    if (g->cidx_entry == 16) {
      put32(e + 8, sbytes[ch * ORA_CHUNK]); /* V-side metadata bytes before the chunk */
      put32(e + 12, any_channel(c) ? sbytes_k[ch * ORA_CHUNK] : 0u); /* K side, if it differs */
    }
  }
}

/* Per-row metadata of segment (kv, h) within its layer: the H K segments, then
 * the H V segments. */
static uint64_t seg_meta_off(const ora_geom* g, int64_t H, int kv, int64_t h) {
  return kv == 0 ? (uint64_t)h * g->seg_scale_bytes_k
                 : (uint64_t)H * g->seg_scale_bytes_k + (uint64_t)h * g->seg_scale_bytes;
}

/* Per-channel parameters of K head h, chunk ch, tier tr within its layer:
 * after the per-row metadata, one block per (head, chunk), the INT8 entries
 * (if that tier is per-channel) before the INT4 entries. */
static uint64_t chan_off(const ora_config* c, const ora_geom* g, int64_t h, int64_t ch, int tr) {
  uint64_t off = g->scales_bytes + ((uint64_t)h * (uint64_t)g->nchunks + (uint64_t)ch) * g->chan_block;
  if (tr == T_INT4 && (c->quant_int8 & QV_CHANNEL))
    off += (uint64_t)c->head_dim * qv_group_entry(c->quant_int8);
  return off;
}

/* Per-channel K quantization of chunk [t0, t1) for tier tr (descriptor q with
 * bit 4): channel i's group is {src[t][i] : t in the chunk, tier[t] == tr},
 * quantized by quant_group; codes go to each row's data slot, the d group
 * entries to blk (left zero when the chunk has no row of the tier).  Returns
 * the number of those rows holding a non-finite element. */
static uint32_t pack_channel_chunk(int tr, int32_t q, int32_t d, const uint16_t* src, const uint8_t* tier,
                                   int64_t t0, int64_t t1, const uint32_t* units, uint8_t* seg, uint8_t* blk) {
  int64_t rows[ORA_CHUNK], cnt = 0;
  for (int64_t t = t0; t < t1; ++t)
    if (tier[t] == tr) rows[cnt++] = t;
  if (cnt == 0) return 0;
  uint16_t vals[ORA_CHUNK];
  int32_t codes[ORA_CHUNK];
  int32_t* rc = (int32_t*)malloc((size_t)cnt * (size_t)d * sizeof(int32_t));
  for (int32_t i = 0; i < d; ++i) {
    for (int64_t j = 0; j < cnt; ++j) vals[j] = src[rows[j] * d + i];
    quant_group(tr, q, vals, 1, cnt, codes, blk + (uint64_t)i * qv_group_entry(q));
    for (int64_t j = 0; j < cnt; ++j) rc[j * d + i] = codes[j];
  }
  uint32_t bad = 0;
  for (int64_t j = 0; j < cnt; ++j) {
    store_codes(tr, d, rc + j * d, seg + (uint64_t)units[rows[j]] * ((uint64_t)d / 2));
    for (int32_t i = 0; i < d; ++i)
      if ((src[rows[j] * d + i] & 0x7C00u) == 0x7C00u) { ++bad; break; }
  }
  free(rc);
  return bad;
}

/* Payload geometry: out = {tiermap_off, chunkidx_off, layers_off, seg_bytes,
 * seg_stride, scales_bytes, layer_stride, total, nq, seg_scale_bytes,
 * seg_scale_bytes_k, chan_block, channel_bytes}. */
int ora_geometry(const ora_config* c, uint64_t* out) {
  ora_plan_t p;
  int st = ora_plan(c, &p);
  if (st) return st;
  ora_geom g;
  geometry(c, &p, &g);
  uint64_t v[13] = {g.tiermap_off, g.chunkidx_off, g.layers_off, g.seg_bytes, g.seg_stride,
                    g.scales_bytes, g.layer_stride, g.total, (uint64_t)g.nq, g.seg_scale_bytes,
                    g.seg_scale_bytes_k, g.chan_block, g.channel_bytes};
  memcpy(out, v, sizeof(v));
  return ORA_OK;
}

/* The payload's first layers_off bytes (header with a zero non-finite count,
 * tier map, chunk index) for a tier map that is on plan. */
int ora_pack_meta(const ora_config* c, const uint8_t* tier, uint8_t* out, uint64_t capacity) {
  ora_plan_t p;
  int st = ora_plan(c, &p);
  if (st) return st;
  ora_geom g;
  geometry(c, &p, &g);
  if (capacity < g.layers_off) return ORA_ERR_CAPACITY;
  int64_t n = c->num_tokens;
  uint32_t* units = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* qrank = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* sbytes = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* sbytes_k = (uint32_t*)malloc((size_t)n * 4);
  memset(out, 0, g.layers_off);
  write_meta(c, &p, &g, tier, units, qrank, sbytes, sbytes_k, out);
  free(units);
  free(qrank);
  free(sbytes);
  free(sbytes_k);
  return ORA_OK;
}

int ora_pack(const ora_config* c, const uint16_t* k, const uint16_t* v, const uint8_t* tier,
             uint8_t* payload, uint64_t capacity) {
  ora_plan_t p;
  int st = ora_plan(c, &p);
  if (st) return st;
  ora_geom g;
  geometry(c, &p, &g);
  if (capacity < g.total) return ORA_ERR_CAPACITY;
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  /* The tier map must carry exactly the planned counts (sizes depend on them). */
  int64_t cnt[4] = {0, 0, 0, 0};
  for (int64_t t = 0; t < n; ++t) {
    if (tier[t] > 3) return ORA_ERR_INVALID_ARG;
    cnt[tier[t]]++;
  }
  if (cnt[T_FP16] != p.n_sink + p.n_fp16 || cnt[T_INT8] != p.n_int8 ||
      cnt[T_INT4] != p.n_int4 || cnt[T_DROP] != p.n_drop)
    return ORA_ERR_INVALID_ARG;

  memset(payload, 0, g.total);
  uint32_t* units = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* qrank = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* sbytes = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* sbytes_k = (uint32_t*)malloc((size_t)n * 4);
  write_meta(c, &p, &g, tier, units, qrank, sbytes, sbytes_k, payload);
  uint32_t nonfinite = 0;
  uint64_t rowunit = (uint64_t)d / 2;
  for (int64_t l = 0; l < L; ++l) {
    uint8_t* lb = payload + g.layers_off + (uint64_t)l * g.layer_stride;
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        const uint16_t* src = (kv == 0 ? k : v) + ((l * H + h) * n) * d;
        uint8_t* seg = lb + g.scales_bytes + g.channel_bytes + (uint64_t)(kv * H + h) * g.seg_stride;
        uint8_t* sc = lb + seg_meta_off(&g, H, kv, h);
        const uint32_t* so = kv == 0 ? sbytes_k : sbytes;
        for (int64_t t = 0; t < n; ++t) {
          int32_t q = tier[t] == T_INT8 ? c->quant_int8 : c->quant_int4;
          int quant = tier[t] == T_INT8 || tier[t] == T_INT4;
          if (kv == 0 && quant && (q & QV_CHANNEL)) continue; /* per-channel K rows: per chunk below */
          int bad = ora_encode_row_q(tier[t], q, (int32_t)d, src + t * d, seg + units[t] * rowunit, sc + so[t]);
          if (quant) nonfinite += (uint32_t)bad;
        }
        if (kv == 0)
          for (int64_t ch = 0; ch < g.nchunks; ++ch)
            for (int tr = T_INT8; tr <= T_INT4; ++tr) {
              int32_t q = tr == T_INT8 ? c->quant_int8 : c->quant_int4;
              if (!(q & QV_CHANNEL)) continue;
              int64_t t1 = (ch + 1) * ORA_CHUNK < n ? (ch + 1) * ORA_CHUNK : n;
              nonfinite += pack_channel_chunk(tr, q, (int32_t)d, src, tier, ch * ORA_CHUNK, t1, units, seg,
                                              lb + chan_off(c, &g, h, ch, tr));
            }
      }
  }
  put32(payload + 144, nonfinite);
  free(units);
  free(qrank);
  free(sbytes);
  free(sbytes_k);
  return ORA_OK;
}

/* Checks a payload header against the configuration. */
int ora_check_header(const ora_config* c, const uint8_t* payload, uint64_t bytes) {
  ora_plan_t p;
  int st = ora_plan(c, &p);
  if (st) return st;
  ora_geom g;
  geometry(c, &p, &g);
  if (bytes < 256) return ORA_ERR_FORMAT;
  uint8_t want[256];
  write_header(c, &p, &g, want);
  /* every field but the non-finite row count must match exactly */
  if (memcmp(want, payload, 144) != 0) return ORA_ERR_FORMAT;
  if (get32(payload + 148) != 0) return ORA_ERR_FORMAT;
  if (memcmp(want + 152, payload + 152, 256 - 152) != 0) return ORA_ERR_FORMAT;
  if (bytes < g.total) return ORA_ERR_FORMAT;
  return ORA_OK;
}

int ora_unpack(const ora_config* c, const uint8_t* payload, uint64_t bytes, uint16_t* kc,
               uint16_t* vc, const int32_t* block_table, int32_t num_blocks, int32_t block_size) {
  int st = ora_check_header(c, payload, bytes);
  if (st) return st;
  if (block_size < 1 || num_blocks < 1) return ORA_ERR_INVALID_ARG;
  ora_plan_t p;
  ora_plan(c, &p);
  ora_geom g;
  geometry(c, &p, &g);
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  uint8_t* tier = (uint8_t*)malloc((size_t)n);
  int64_t cnt[4] = {0, 0, 0, 0};
  for (int64_t t = 0; t < n; ++t) {
    tier[t] = (payload[g.tiermap_off + (uint64_t)t / 4] >> (2 * (t % 4))) & 3;
    cnt[tier[t]]++;
  }
  uint32_t* units = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* qrank = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* sbytes = (uint32_t*)malloc((size_t)n * 4);
  uint32_t* sbytes_k = (uint32_t*)malloc((size_t)n * 4);
  ora_offsets((int32_t)n, tier, units, qrank);
  ora_scale_offsets((int32_t)n, tier, g.e8, g.e4, sbytes);
  ora_scale_offsets((int32_t)n, tier, g.ek8, g.ek4, sbytes_k);
  int bad = cnt[T_FP16] != p.n_sink + p.n_fp16 || cnt[T_INT8] != p.n_int8 ||
            cnt[T_INT4] != p.n_int4 || cnt[T_DROP] != p.n_drop;
  for (int64_t ch = 0; ch < g.nchunks && !bad; ++ch) {
    const uint8_t* e = payload + g.chunkidx_off + g.cidx_entry * (uint64_t)ch;
    bad = get32(e) != units[ch * ORA_CHUNK] || get32(e + 4) != qrank[ch * ORA_CHUNK];
    if (!bad && g.cidx_entry == 16)
      bad = get32(e + 8) != sbytes[ch * ORA_CHUNK] ||
            get32(e + 12) != (any_channel(c) ? sbytes_k[ch * ORA_CHUNK] : 0u);
  }
  for (int64_t t = 0; t < (n + block_size - 1) / block_size && !bad; ++t)
    bad = block_table[t] < 0 || block_table[t] >= num_blocks;
  if (bad) {
    free(tier); free(units); free(qrank); free(sbytes); free(sbytes_k);
    return ORA_ERR_FORMAT;
  }
  uint64_t rowunit = (uint64_t)d / 2;
  for (int64_t l = 0; l < L; ++l) {
    const uint8_t* lb = payload + g.layers_off + (uint64_t)l * g.layer_stride;
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        const uint8_t* seg = lb + g.scales_bytes + g.channel_bytes + (uint64_t)(kv * H + h) * g.seg_stride;
        const uint8_t* sc = lb + seg_meta_off(&g, H, kv, h);
        const uint32_t* so = kv == 0 ? sbytes_k : sbytes;
        uint16_t* cache = kv == 0 ? kc : vc;
        for (int64_t t = 0; t < n; ++t) {
          int32_t q = tier[t] == T_INT8 ? c->quant_int8 : c->quant_int4;
          int64_t blk = block_table[t / block_size], slot = t % block_size;
          uint16_t* dst = cache + (((l * num_blocks + blk) * block_size + slot) * H + h) * d;
          const uint8_t* row = seg + units[t] * rowunit;
          if (kv == 0 && (tier[t] == T_INT8 || tier[t] == T_INT4) && (q & QV_CHANNEL)) {
            /* per-channel K row: element i with channel i's entry of the chunk */
            ora_decode_row_channel(tier[t], q, (int32_t)d, row, lb + chan_off(c, &g, h, t / ORA_CHUNK, tier[t]), dst);
          } else {
            ora_decode_row_q(tier[t], q, (int32_t)d, row, sc + so[t], dst);
          }
        }
      }
  }
  free(tier); free(units); free(qrank); free(sbytes); free(sbytes_k);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Cold-tier precision upgrade (Sec. 4.2, Fig. "sysarch": on-demand fetch that */
/* upgrades tokens already present at low precision; Sec. 8 "cold-tier fetch */
/* design").  The prefill side, which still holds the fp16 K/V and the tier   */
/* map, sends for a listed set of tokens either the fp16 rows themselves       */
/* (mode 0, exact) or the INT8-quantized residual between the fp16 row and    */
/* the row the decoder reconstructed (mode 1); the decoder applies it in      */
/* place in its paged cache.                                                   */
/*                                                                             */
/* Upgrade payload (version 1, little-endian, sections 256-byte aligned):     */
/*   [header 256 B: u32 magic 0x55564B53 ("SKVU"), u32 version, i32 L, H, d,   */
/*    n, m (listed tokens), mode; u64 offsets of tokens, tiers, scales, data;  */
/*    u64 total; u32 status]                                                   */
/*   [tokens: i32[m], ascending] [tiers: u8[m], each token's tier in the       */
/*   original payload] [scales: fp32 [L][2][H][m], mode 1 only]                */
/*   [data: [L][2][H][m] rows, 2d bytes (mode 0) or d bytes (mode 1)]          */
/* ------------------------------------------------------------------------ */

#define ORA_UPG_MAGIC 0x55564B53u /* bytes 'S','K','V','U' */

typedef struct {
  uint64_t tokens_off, tiers_off, scales_off, data_off, total, row_bytes;
} ora_upg_geom;

static int upg_geometry(const ora_config* c, int32_t m, int32_t mode, ora_upg_geom* g) {
  int st = ora_validate(c);
  if (st) return st;
  if (c->quant_int8 || c->quant_int4) return ORA_ERR_INVALID_ARG; /* held rows use descriptor 0 */
  if (m < 1 || m > c->num_tokens || (mode != 0 && mode != 1)) return ORA_ERR_INVALID_ARG;
  uint64_t L = (uint64_t)c->num_layers, H = (uint64_t)c->num_kv_heads, d = (uint64_t)c->head_dim;
  g->tokens_off = 256;
  g->tiers_off = g->tokens_off + up256(4 * (uint64_t)m);
  g->scales_off = g->tiers_off + up256((uint64_t)m);
  g->data_off = g->scales_off + (mode == 1 ? up256(L * 2 * H * (uint64_t)m * 4) : 0);
  g->row_bytes = mode == 0 ? 2 * d : d;
  g->total = g->data_off + L * 2 * H * (uint64_t)m * g->row_bytes;
  return ORA_OK;
}

int ora_upgrade_size(const ora_config* c, int32_t m, int32_t mode, uint64_t* bytes) {
  ora_upg_geom g;
  int st = upg_geometry(c, m, mode, &g);
  if (st == ORA_OK) *bytes = g.total;
  return st;
}

/* Reconstruction the decoder holds for one row after the original transfer. */
static void held_row(int tr, int32_t d, const uint16_t* x, uint16_t* out) {
  uint8_t enc[512];
  float scale = 0.0f;
  ora_encode_row(tr, d, x, enc, &scale);
  ora_decode_row(tr, d, enc, scale, out);
}

static int upg_tokens_ok(int32_t n, const int32_t* tokens, int32_t m) {
  for (int32_t i = 0; i < m; ++i) {
    if (tokens[i] < 0 || tokens[i] >= n) return 0;
    if (i > 0 && tokens[i] <= tokens[i - 1]) return 0;
  }
  return 1;
}

int ora_pack_upgrade(const ora_config* c, const uint16_t* k, const uint16_t* v, const uint8_t* tier,
                     const int32_t* tokens, int32_t m, int32_t mode, uint8_t* out, uint64_t capacity) {
  ora_upg_geom g;
  int st = upg_geometry(c, m, mode, &g);
  if (st) return st;
  if (capacity < g.total) return ORA_ERR_CAPACITY;
  if (!upg_tokens_ok(c->num_tokens, tokens, m)) return ORA_ERR_INVALID_ARG;
  for (int32_t i = 0; i < m; ++i)
    if (tier[tokens[i]] > 3) return ORA_ERR_INVALID_ARG;
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  memset(out, 0, g.total);
  put32(out + 0, ORA_UPG_MAGIC);
  put32(out + 4, 1);
  put32(out + 8, (uint32_t)L);
  put32(out + 12, (uint32_t)H);
  put32(out + 16, (uint32_t)d);
  put32(out + 20, (uint32_t)n);
  put32(out + 24, (uint32_t)m);
  put32(out + 28, (uint32_t)mode);
  memcpy(out + 32, &g.tokens_off, 8);
  memcpy(out + 40, &g.tiers_off, 8);
  memcpy(out + 48, &g.scales_off, 8);
  memcpy(out + 56, &g.data_off, 8);
  memcpy(out + 64, &g.total, 8);
  for (int32_t i = 0; i < m; ++i) {
    put32(out + g.tokens_off + 4 * (uint64_t)i, (uint32_t)tokens[i]);
    out[g.tiers_off + (uint64_t)i] = tier[tokens[i]];
  }
  uint16_t held[256];
  for (int64_t l = 0; l < L; ++l)
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        const uint16_t* src = (kv == 0 ? k : v) + ((l * H + h) * n) * d;
        uint64_t seg = (uint64_t)((l * 2 + kv) * H + h);
        for (int32_t i = 0; i < m; ++i) {
          const uint16_t* x = src + (int64_t)tokens[i] * d;
          uint8_t* row = out + g.data_off + (seg * (uint64_t)m + (uint64_t)i) * g.row_bytes;
          if (mode == 0) {
            for (int64_t e = 0; e < d; ++e) { row[2 * e] = (uint8_t)x[e]; row[2 * e + 1] = (uint8_t)(x[e] >> 8); }
            continue;
          }
          /* residual e = RN32(x - held) of every element, INT8 absmax quantized */
          held_row(tier[tokens[i]], (int32_t)d, x, held);
          float res[256];
          int finite = 1;
          float amax = 0.0f;
          for (int64_t e = 0; e < d; ++e) {
            float xf = half_to_float(x[e]), hf = half_to_float(held[e]);
            res[e] = xf - hf;
            if (!isfinite(res[e])) finite = 0;
            else if (fabsf(res[e]) > amax) amax = fabsf(res[e]);
          }
          float scale;
          uint8_t* sc = out + g.scales_off + (seg * (uint64_t)m + (uint64_t)i) * 4;
          if (!finite) {
            uint32_t nanbits = 0x7FC00000u;
            memcpy(&scale, &nanbits, 4);
            for (int64_t e = 0; e < d; ++e) row[e] = 0;
          } else if (amax == 0.0f) {
            scale = 0.0f;
            for (int64_t e = 0; e < d; ++e) row[e] = 0;
          } else {
            scale = amax / 127.0f;
            float r = 127.0f / amax;
            for (int64_t e = 0; e < d; ++e) {
              float q = nearbyintf(res[e] * r);
              if (q > 127.0f) q = 127.0f;
              if (q < -127.0f) q = -127.0f;
              row[e] = (uint8_t)((int32_t)q & 0xFF);
            }
          }
          put32(sc, fbits(scale));
        }
      }
  return ORA_OK;
}

int ora_unpack_upgrade(const ora_config* c, const uint8_t* up, uint64_t bytes, uint16_t* kc, uint16_t* vc,
                       const int32_t* block_table, int32_t num_blocks, int32_t block_size) {
  int st = ora_validate(c);
  if (st) return st;
  if (bytes < 256 || get32(up) != ORA_UPG_MAGIC || get32(up + 4) != 1) return ORA_ERR_FORMAT;
  int32_t m = (int32_t)get32(up + 24), mode = (int32_t)get32(up + 28);
  ora_upg_geom g;
  if (upg_geometry(c, m, mode, &g)) return ORA_ERR_FORMAT;
  if (get32(up + 8) != (uint32_t)c->num_layers || get32(up + 12) != (uint32_t)c->num_kv_heads ||
      get32(up + 16) != (uint32_t)c->head_dim || get32(up + 20) != (uint32_t)c->num_tokens)
    return ORA_ERR_FORMAT;
  uint64_t f[5];
  memcpy(f, up + 32, 40);
  if (f[0] != g.tokens_off || f[1] != g.tiers_off || f[2] != g.scales_off || f[3] != g.data_off || f[4] != g.total ||
      bytes < g.total || get32(up + 72) != 0)
    return ORA_ERR_FORMAT;
  int32_t* tokens = (int32_t*)malloc((size_t)m * 4);
  for (int32_t i = 0; i < m; ++i) tokens[i] = (int32_t)get32(up + g.tokens_off + 4 * (uint64_t)i);
  int ok = upg_tokens_ok(c->num_tokens, tokens, m);
  for (int32_t i = 0; i < m && ok; ++i) ok = up[g.tiers_off + (uint64_t)i] <= 3;
  if (ok && (block_size < 1 || num_blocks < 1)) ok = 0;
  for (int64_t b = 0; ok && b < ((int64_t)c->num_tokens + block_size - 1) / block_size; ++b)
    ok = block_table[b] >= 0 && block_table[b] < num_blocks;
  if (!ok) { free(tokens); return ORA_ERR_FORMAT; }
  int64_t L = c->num_layers, H = c->num_kv_heads, d = c->head_dim;
  for (int64_t l = 0; l < L; ++l)
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        uint64_t seg = (uint64_t)((l * 2 + kv) * H + h);
        uint16_t* cache = kv == 0 ? kc : vc;
        for (int32_t i = 0; i < m; ++i) {
          int64_t t = tokens[i], blk = block_table[t / block_size], slot = t % block_size;
          uint16_t* dst = cache + (((l * num_blocks + blk) * block_size + slot) * H + h) * d;
          const uint8_t* row = up + g.data_off + (seg * (uint64_t)m + (uint64_t)i) * g.row_bytes;
          if (mode == 0) {
            for (int64_t e = 0; e < d; ++e) dst[e] = (uint16_t)(row[2 * e] | (row[2 * e + 1] << 8));
            continue;
          }
          float scale;
          uint32_t sb = get32(up + g.scales_off + (seg * (uint64_t)m + (uint64_t)i) * 4);
          memcpy(&scale, &sb, 4);
          if (isnan(scale)) continue; /* no usable residual: keep the held row */
          for (int64_t e = 0; e < d; ++e) {
            float corr = (float)(int32_t)(int8_t)row[e] * scale;
            dst[e] = ora_float_to_half(half_to_float(dst[e]) + corr);
          }
        }
      }
  free(tokens);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Per-layer and per-head tier maps.  The paper keeps one tier per token for  */
/* every layer and head and names finer maps as the next step: a per-layer    */
/* budget allocation favouring layers whose errors propagate furthest         */
/* (Sec. 2.6, Sec. 6.10) and per-head or per-layer importance scores          */
/* (Sec. 7.5, Sec. 9 (iii)).  Here the (layer, head) pairs are partitioned    */
/* into groups -- one group (granularity 0, the paper's map), one per layer   */
/* (1) or one per (layer, head) (2) -- and every group gets its own score,    */
/* its own budget b_g, its own plan (the Sec. 4.4 mapping with sinks pinned,  */
/* as above) and its own tier map; K and V of a pair share their group's map. */
/*                                                                             */
/* Grouped payload (version 1, little-endian, sections 256-byte aligned,      */
/* zero padding):                                                              */
/*   header 256 B: u32 words 0 magic 0x47564B53 ("SKVG"), 1 version, 2-5 L, H, */
/*     d, n, 6 granularity, 7 G, 8 num_tiers, 9 score_mode, 10-12 bits of b,   */
/*     rho, lambda, 13 num_sink (as configured), 14 chunk tokens (256),        */
/*     15 zero; u64 at words 16, 18, ..., 30: group table, tier maps, tier-map */
/*     stride, chunk indexes, chunk-index stride, segment table, layers,       */
/*     total; u32 word 32 non-finite quantized rows, 33 status                 */
/*   group table: G x 32 B, u32 [sinks, fp16, int8, int4, drop, bits of b_g,   */
/*     quantized rows nq_g, zero]                                              */
/*   G tier maps (2 bits per token, token t at bits 2(t%4) of byte t/4), each  */
/*     padded to the tier-map stride                                           */
/*   G chunk indexes (u32 row-width units and u32 quantized rows before every  */
/*     256th token), each padded to the chunk-index stride                     */
/*   segment table: for (layer, K/V, head) in that order, u64 offsets of the   */
/*     segment's scales and of its rows                                        */
/*   layers: [fp32 scales of the 2H segments, nq_g each, back to back, padded] */
/*     [the 2H segments, rows in token order at their group's tier widths,     */
/*     each padded to 256 B]                                                   */
/* ------------------------------------------------------------------------ */

#define ORA_GRP_MAGIC 0x47564B53u /* bytes 'S','K','V','G' */
enum { GRAN_TOKEN = 0, GRAN_LAYER = 1, GRAN_HEAD = 2 };

int32_t ora_group_count(const ora_config* c, int32_t gran) {
  if (gran == GRAN_TOKEN) return 1;
  if (gran == GRAN_LAYER) return c->num_layers;
  if (gran == GRAN_HEAD) return c->num_layers * c->num_kv_heads;
  return -1;
}

static int64_t group_of(const ora_config* c, int32_t gran, int64_t l, int64_t h) {
  return gran == GRAN_TOKEN ? 0 : gran == GRAN_LAYER ? l : l * c->num_kv_heads + h;
}

/* Validates cfg, the granularity and every group budget, then plans every
 * group (plans: G entries). */
static int plan_groups(const ora_config* c, int32_t gran, const float* budgets, ora_plan_t* plans) {
  int st = ora_validate(c);
  if (st) return st;
  if (c->quant_int8 || c->quant_int4) return ORA_ERR_INVALID_ARG; /* grouped payloads use descriptor 0 */
  int32_t G = ora_group_count(c, gran);
  if (G < 1) return ORA_ERR_INVALID_ARG;
  for (int32_t g = 0; g < G; ++g) {
    ora_config cg = *c;
    if (budgets) cg.budget = budgets[g];
    st = ora_plan(&cg, plans ? &plans[g] : NULL);
    if (st) return st;
  }
  return ORA_OK;
}

int ora_plan_group(const ora_config* c, int32_t gran, const float* budgets, int32_t g, ora_plan_t* p) {
  int32_t G = ora_group_count(c, gran);
  if (G < 1 || g < 0 || g >= G) return ORA_ERR_INVALID_ARG;
  ora_plan_t* all = (ora_plan_t*)malloc((size_t)G * sizeof(ora_plan_t));
  int st = plan_groups(c, gran, budgets, all);
  if (!st) *p = all[g];
  free(all);
  return st;
}

typedef struct {
  int32_t G;
  int64_t nchunks;
  uint64_t group_off, tiermaps_off, tiermap_stride, chunkidx_off, chunkidx_stride, segtab_off,
      layers_off, total;
} ora_ggeom;

static uint64_t group_seg_bytes(const ora_plan_t* p, uint64_t d) {
  return (uint64_t)(p->n_sink + p->n_fp16) * 2 * d + (uint64_t)p->n_int8 * d + (uint64_t)p->n_int4 * (d / 2);
}

/* Section offsets; segtab (optional, 2LH pairs of u64) receives every
 * segment's scale and row offsets. */
static void grouped_layout(const ora_config* c, int32_t gran, const ora_plan_t* plans, ora_ggeom* g,
                           uint64_t* segtab) {
  uint64_t L = (uint64_t)c->num_layers, H = (uint64_t)c->num_kv_heads, d = (uint64_t)c->head_dim;
  uint64_t n = (uint64_t)c->num_tokens;
  g->G = ora_group_count(c, gran);
  g->nchunks = (int64_t)((n + ORA_CHUNK - 1) / ORA_CHUNK);
  g->group_off = 256;
  g->tiermaps_off = g->group_off + up256(32 * (uint64_t)g->G);
  g->tiermap_stride = up256((n + 3) / 4);
  g->chunkidx_off = g->tiermaps_off + (uint64_t)g->G * g->tiermap_stride;
  g->chunkidx_stride = up256(8 * (uint64_t)g->nchunks);
  g->segtab_off = g->chunkidx_off + (uint64_t)g->G * g->chunkidx_stride;
  g->layers_off = g->segtab_off + up256(2 * L * H * 16);
  uint64_t off = g->layers_off;
  for (uint64_t l = 0; l < L; ++l) {
    uint64_t nscales = 0;
    for (int kv = 0; kv < 2; ++kv)
      for (uint64_t h = 0; h < H; ++h) {
        const ora_plan_t* p = &plans[group_of(c, gran, (int64_t)l, (int64_t)h)];
        if (segtab) segtab[2 * ((l * 2 + (uint64_t)kv) * H + h)] = off + 4 * nscales;
        nscales += (uint64_t)(p->n_int8 + p->n_int4);
      }
    uint64_t data = off + up256(4 * nscales);
    for (int kv = 0; kv < 2; ++kv)
      for (uint64_t h = 0; h < H; ++h) {
        const ora_plan_t* p = &plans[group_of(c, gran, (int64_t)l, (int64_t)h)];
        if (segtab) segtab[2 * ((l * 2 + (uint64_t)kv) * H + h) + 1] = data;
        data += up256(group_seg_bytes(p, d));
      }
    off = data;
  }
  g->total = off;
}

int ora_grouped_size(const ora_config* c, int32_t gran, const float* budgets, uint64_t* bytes) {
  int32_t G = ora_group_count(c, gran);
  if (G < 1) return ORA_ERR_INVALID_ARG;
  ora_plan_t* plans = (ora_plan_t*)malloc((size_t)G * sizeof(ora_plan_t));
  int st = plan_groups(c, gran, budgets, plans);
  if (!st) {
    ora_ggeom g;
    grouped_layout(c, gran, plans, &g, NULL);
    *bytes = g.total;
  }
  free(plans);
  return st;
}

/* Exact sum of squares of token t over the K and V elements of the pairs in
 * group grp, in units of 2^-48. */
int ora_sumsq_group(const ora_config* c, int32_t gran, const uint16_t* k, const uint16_t* v, int32_t grp,
                    int32_t t, uint64_t* hi, uint64_t* lo) {
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  u128 S = 0;
  for (int64_t l = 0; l < L; ++l)
    for (int64_t h = 0; h < H; ++h) {
      if (group_of(c, gran, l, h) != grp) continue;
      const uint16_t* kr = k + (((l * H + h) * n + t) * d);
      const uint16_t* vr = v + (((l * H + h) * n + t) * d);
      for (int64_t i = 0; i < d; ++i) S += square_units(kr[i]) + square_units(vr[i]);
    }
  *hi = (uint64_t)(S >> 64);
  *lo = (uint64_t)S;
  return ORA_OK;
}

/* Mean attention mass of every key over the observation rows of the query
 * heads that read the group's KV heads (a layer: all Hq query heads of the
 * layer; a (layer, KV head): its Hq/H query heads), binary64.  Same
 * statistic and conventions as attention_mass, restricted to the group. */
static void attention_mass_groups(const ora_config* c, int32_t gran, const uint16_t* k, const uint16_t* q,
                                  double* A) {
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  int64_t Hq = c->num_q_heads, W = c->obs_window, grp = Hq / H;
  int64_t G = ora_group_count(c, gran);
  double inv_sqrt_d = 1.0 / sqrt((double)d);
  double* z = (double*)malloc((size_t)n * sizeof(double));
  double* qv = (double*)malloc((size_t)d * sizeof(double));
  double* kv = (double*)malloc((size_t)(n * d) * sizeof(double));
  for (int64_t i = 0; i < G * n; ++i) A[i] = 0.0;
  for (int64_t l = 0; l < L; ++l)
    for (int64_t hq = 0; hq < Hq; ++hq) {
      int64_t h = hq / grp;
      double* Ag = A + group_of(c, gran, l, h) * n;
      if (hq % grp == 0) decode_plane(k + (l * H + h) * n * d, n * d, kv);
      for (int64_t w = 0; w < W; ++w) {
        const uint16_t* qr = q + ((l * Hq + hq) * W + w) * d;
        for (int64_t i = 0; i < d; ++i) qv[i] = ora_half_to_double(qr[i]);
        double zmax = -INFINITY;
        for (int64_t t = 0; t < n; ++t) {
          const double* kr = kv + t * d;
          double dot = 0.0;
          for (int64_t i = 0; i < d; ++i) dot += qv[i] * kr[i];
          z[t] = dot * inv_sqrt_d;
          if (z[t] > zmax) zmax = z[t];
        }
        double den = 0.0;
        for (int64_t t = 0; t < n; ++t) { z[t] = exp(z[t] - zmax); den += z[t]; }
        for (int64_t t = 0; t < n; ++t) Ag[t] += z[t] / den;
      }
    }
  double rows = (double)(gran == GRAN_TOKEN ? L * Hq * W : gran == GRAN_LAYER ? Hq * W : grp * W);
  for (int64_t i = 0; i < G * n; ++i) A[i] /= rows;
  free(z);
  free(qv);
  free(kv);
}

/* key[g*n + t]: the score of token t in group g (eq. "importance" with the
 * statistic restricted to the group's pairs). */
int ora_score_groups(const ora_config* c, int32_t gran, const uint16_t* k, const uint16_t* v,
                     const uint16_t* q, double* key) {
  int st = ora_validate(c);
  if (st) return st;
  int32_t G = ora_group_count(c, gran);
  if (G < 1) return ORA_ERR_INVALID_ARG;
  int32_t n = c->num_tokens;
  double* w = (double*)malloc((size_t)n * sizeof(double));
  if (c->score_mode == MODE_KVNORM) {
    ora_decay_table(c->decay, 2, n, w);
    for (int32_t g = 0; g < G; ++g)
      for (int32_t t = 0; t < n; ++t) {
        uint64_t hi, lo;
        ora_sumsq_group(c, gran, k, v, g, t, &hi, &lo);
        u128 S = ((u128)hi << 64) | lo;
        key[(int64_t)g * n + t] = ldexp((double)S, -48) * w[n - 1 - t];
      }
  } else if (c->score_mode == MODE_ATTN) {
    if (!q) { free(w); return ORA_ERR_INVALID_ARG; }
    ora_decay_table(c->decay, 1, n, w);
    double* A = (double*)malloc((size_t)G * (size_t)n * sizeof(double));
    attention_mass_groups(c, gran, k, q, A);
    for (int32_t g = 0; g < G; ++g)
      for (int32_t t = 0; t < n; ++t) key[(int64_t)g * n + t] = A[(int64_t)g * n + t] * w[n - 1 - t];
    free(A);
  } else {
    ora_decay_table(c->decay, 1, n, w);
    for (int32_t g = 0; g < G; ++g)
      for (int32_t t = 0; t < n; ++t) key[(int64_t)g * n + t] = w[n - 1 - t];
  }
  free(w);
  return ORA_OK;
}

/* tier[g*n + t]: Prop. 1's assignment within every group, under its budget. */
int ora_assign_groups(const ora_config* c, int32_t gran, const float* budgets, const double* key,
                      uint8_t* tier) {
  int32_t G = ora_group_count(c, gran);
  if (G < 1) return ORA_ERR_INVALID_ARG;
  int st = plan_groups(c, gran, budgets, NULL);
  if (st) return st;
  int64_t n = c->num_tokens;
  for (int32_t g = 0; g < G; ++g) {
    ora_config cg = *c;
    if (budgets) cg.budget = budgets[g];
    st = ora_assign(&cg, key + g * n, tier + g * n);
    if (st) return st;
  }
  return ORA_OK;
}

static void write_grouped_header(const ora_config* c, int32_t gran, const ora_ggeom* g, uint8_t* h) {
  memset(h, 0, 256);
  put32(h + 0, ORA_GRP_MAGIC);
  put32(h + 4, ORA_VERSION);
  put32(h + 8, (uint32_t)c->num_layers);
  put32(h + 12, (uint32_t)c->num_kv_heads);
  put32(h + 16, (uint32_t)c->head_dim);
  put32(h + 20, (uint32_t)c->num_tokens);
  put32(h + 24, (uint32_t)gran);
  put32(h + 28, (uint32_t)g->G);
  put32(h + 32, (uint32_t)c->num_tiers);
  put32(h + 36, (uint32_t)c->score_mode);
  put32(h + 40, fbits(c->budget));
  put32(h + 44, fbits(c->first_ratio));
  put32(h + 48, fbits(c->decay));
  put32(h + 52, (uint32_t)c->num_sink);
  put32(h + 56, ORA_CHUNK);
  put64(h + 64, g->group_off);
  put64(h + 72, g->tiermaps_off);
  put64(h + 80, g->tiermap_stride);
  put64(h + 88, g->chunkidx_off);
  put64(h + 96, g->chunkidx_stride);
  put64(h + 104, g->segtab_off);
  put64(h + 112, g->layers_off);
  put64(h + 120, g->total);
  put32(h + 128, 0); /* non-finite quantized rows */
  put32(h + 132, 0); /* status */
}

/* Everything before the layers: header, group table, tier maps, chunk
 * indexes, segment table.  units/qrank receive every group's row offsets. */
static void write_grouped_meta(const ora_config* c, int32_t gran, const float* budgets, const ora_plan_t* plans,
                               const ora_ggeom* g, const uint64_t* segtab, const uint8_t* tier,
                               uint32_t* units, uint32_t* qrank, uint8_t* out) {
  int64_t n = c->num_tokens, L = c->num_layers, H = c->num_kv_heads;
  write_grouped_header(c, gran, g, out);
  for (int32_t grp = 0; grp < g->G; ++grp) {
    const ora_plan_t* p = &plans[grp];
    uint8_t* e = out + g->group_off + 32 * (uint64_t)grp;
    put32(e + 0, (uint32_t)p->n_sink);
    put32(e + 4, (uint32_t)p->n_fp16);
    put32(e + 8, (uint32_t)p->n_int8);
    put32(e + 12, (uint32_t)p->n_int4);
    put32(e + 16, (uint32_t)p->n_drop);
    put32(e + 20, fbits(budgets ? budgets[grp] : c->budget));
    put32(e + 24, (uint32_t)(p->n_int8 + p->n_int4));
    const uint8_t* tg = tier + (int64_t)grp * n;
    uint8_t* map = out + g->tiermaps_off + (uint64_t)grp * g->tiermap_stride;
    for (int64_t t = 0; t < n; ++t) map[t / 4] |= (uint8_t)(tg[t] << (2 * (t % 4)));
    uint32_t* ug = units + (int64_t)grp * n;
    uint32_t* qg = qrank + (int64_t)grp * n;
    ora_offsets((int32_t)n, tg, ug, qg);
    uint8_t* ci = out + g->chunkidx_off + (uint64_t)grp * g->chunkidx_stride;
    for (int64_t ch = 0; ch < g->nchunks; ++ch) {
      put32(ci + 8 * ch, ug[ch * ORA_CHUNK]);
      put32(ci + 8 * ch + 4, qg[ch * ORA_CHUNK]);
    }
  }
  for (int64_t s = 0; s < 2 * L * H; ++s) {
    put64(out + g->segtab_off + 16 * (uint64_t)s, segtab[2 * s]);
    put64(out + g->segtab_off + 16 * (uint64_t)s + 8, segtab[2 * s + 1]);
  }
}

int ora_pack_groups(const ora_config* c, int32_t gran, const float* budgets, const uint16_t* k,
                    const uint16_t* v, const uint8_t* tier, uint8_t* payload, uint64_t capacity) {
  int32_t G = ora_group_count(c, gran);
  if (G < 1) return ORA_ERR_INVALID_ARG;
  ora_plan_t* plans = (ora_plan_t*)malloc((size_t)G * sizeof(ora_plan_t));
  int st = plan_groups(c, gran, budgets, plans);
  if (st) { free(plans); return st; }
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  uint64_t* segtab = (uint64_t*)malloc((size_t)(4 * L * H) * sizeof(uint64_t));
  ora_ggeom g;
  grouped_layout(c, gran, plans, &g, segtab);
  st = capacity < g.total ? ORA_ERR_CAPACITY : ORA_OK;
  /* every group's map must carry exactly its planned counts */
  for (int32_t grp = 0; grp < G && !st; ++grp) {
    int64_t cnt[4] = {0, 0, 0, 0};
    for (int64_t t = 0; t < n && !st; ++t) {
      uint8_t tr = tier[(int64_t)grp * n + t];
      if (tr > 3) st = ORA_ERR_INVALID_ARG;
      else cnt[tr]++;
    }
    const ora_plan_t* p = &plans[grp];
    if (!st && (cnt[T_FP16] != p->n_sink + p->n_fp16 || cnt[T_INT8] != p->n_int8 ||
                cnt[T_INT4] != p->n_int4 || cnt[T_DROP] != p->n_drop))
      st = ORA_ERR_INVALID_ARG;
  }
  if (st) { free(plans); free(segtab); return st; }
  memset(payload, 0, g.total);
  uint32_t* units = (uint32_t*)malloc((size_t)G * (size_t)n * 4);
  uint32_t* qrank = (uint32_t*)malloc((size_t)G * (size_t)n * 4);
  write_grouped_meta(c, gran, budgets, plans, &g, segtab, tier, units, qrank, payload);
  uint32_t nonfinite = 0;
  uint64_t rowunit = (uint64_t)d / 2;
  for (int64_t l = 0; l < L; ++l)
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        int64_t grp = group_of(c, gran, l, h), s = (l * 2 + kv) * H + h;
        const uint8_t* tg = tier + grp * n;
        const uint32_t* ug = units + grp * n;
        const uint32_t* qg = qrank + grp * n;
        const uint16_t* src = (kv == 0 ? k : v) + ((l * H + h) * n) * d;
        uint8_t* sc = payload + segtab[2 * s];
        uint8_t* seg = payload + segtab[2 * s + 1];
        for (int64_t t = 0; t < n; ++t) {
          float scale = 0.0f;
          int bad = ora_encode_row(tg[t], (int32_t)d, src + t * d, seg + ug[t] * rowunit, &scale);
          if (tg[t] == T_INT8 || tg[t] == T_INT4) {
            put32(sc + 4 * (uint64_t)qg[t], fbits(scale));
            nonfinite += (uint32_t)bad;
          }
        }
      }
  put32(payload + 128, nonfinite);
  free(units); free(qrank); free(plans); free(segtab);
  return ORA_OK;
}

int ora_unpack_groups(const ora_config* c, int32_t gran, const float* budgets, const uint8_t* payload,
                      uint64_t bytes, uint16_t* kc, uint16_t* vc, const int32_t* block_table,
                      int32_t num_blocks, int32_t block_size) {
  int32_t G = ora_group_count(c, gran);
  if (G < 1) return ORA_ERR_INVALID_ARG;
  if (block_size < 1 || num_blocks < 1) return ORA_ERR_INVALID_ARG;
  ora_plan_t* plans = (ora_plan_t*)malloc((size_t)G * sizeof(ora_plan_t));
  int st = plan_groups(c, gran, budgets, plans);
  if (st) { free(plans); return st; }
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens, d = c->head_dim;
  uint64_t* segtab = (uint64_t*)malloc((size_t)(4 * L * H) * sizeof(uint64_t));
  ora_ggeom g;
  grouped_layout(c, gran, plans, &g, segtab);
  int bad = bytes < g.layers_off || bytes < g.total;
  uint8_t* want = NULL;
  uint8_t* tier = (uint8_t*)malloc((size_t)G * (size_t)n);
  uint32_t* units = (uint32_t*)malloc((size_t)G * (size_t)n * 4);
  uint32_t* qrank = (uint32_t*)malloc((size_t)G * (size_t)n * 4);
  if (!bad) {
    /* header (but the non-finite count), group table and segment table must be
     * exactly what cfg, the granularity and the budgets imply */
    uint8_t h[256];
    write_grouped_header(c, gran, &g, h);
    bad = memcmp(h, payload, 128) != 0 || get32(payload + 132) != 0 ||
          memcmp(h + 136, payload + 136, 256 - 136) != 0;
  }
  for (int32_t grp = 0; grp < G && !bad; ++grp) {
    const uint8_t* map = payload + g.tiermaps_off + (uint64_t)grp * g.tiermap_stride;
    int64_t cnt[4] = {0, 0, 0, 0};
    for (int64_t t = 0; t < n; ++t) {
      uint8_t tr = (map[t / 4] >> (2 * (t % 4))) & 3;
      tier[(int64_t)grp * n + t] = tr;
      cnt[tr]++;
    }
    const ora_plan_t* p = &plans[grp];
    bad = cnt[T_FP16] != p->n_sink + p->n_fp16 || cnt[T_INT8] != p->n_int8 ||
          cnt[T_INT4] != p->n_int4 || cnt[T_DROP] != p->n_drop;
  }
  if (!bad) {
    /* rebuild the metadata from the decoded maps and compare byte for byte */
    want = (uint8_t*)calloc((size_t)g.layers_off, 1);
    write_grouped_meta(c, gran, budgets, plans, &g, segtab, tier, units, qrank, want);
    bad = memcmp(want + 136, payload + 136, (size_t)(g.layers_off - 136)) != 0;
  }
  for (int64_t b = 0; b < (n + block_size - 1) / block_size && !bad; ++b)
    bad = block_table[b] < 0 || block_table[b] >= num_blocks;
  if (bad) {
    free(want); free(tier); free(units); free(qrank); free(plans); free(segtab);
    return ORA_ERR_FORMAT;
  }
  uint64_t rowunit = (uint64_t)d / 2;
  for (int64_t l = 0; l < L; ++l)
    for (int kv = 0; kv < 2; ++kv)
      for (int64_t h = 0; h < H; ++h) {
        int64_t grp = group_of(c, gran, l, h), s = (l * 2 + kv) * H + h;
        const uint8_t* tg = tier + grp * n;
        const uint32_t* ug = units + grp * n;
        const uint32_t* qg = qrank + grp * n;
        const uint8_t* sc = payload + segtab[2 * s];
        const uint8_t* seg = payload + segtab[2 * s + 1];
        uint16_t* cache = kv == 0 ? kc : vc;
        for (int64_t t = 0; t < n; ++t) {
          float scale = 0.0f;
          if (tg[t] == T_INT8 || tg[t] == T_INT4) {
            uint32_t bits = get32(sc + 4 * (uint64_t)qg[t]);
            memcpy(&scale, &bits, 4);
          }
          int64_t blk = block_table[t / block_size], slot = t % block_size;
          uint16_t* dst = cache + (((l * num_blocks + blk) * block_size + slot) * H + h) * d;
          ora_decode_row(tg[t], (int32_t)d, seg + ug[t] * rowunit, scale, dst);
        }
      }
  free(want); free(tier); free(units); free(qrank); free(plans); free(segtab);
  return ORA_OK;
}

/* The grouped payload's first layers_off bytes (header with a zero non-finite
 * count, group table, tier maps, chunk indexes, segment table) for tier maps
 * on their plans; *layers_off receives their size. */
int ora_pack_groups_meta(const ora_config* c, int32_t gran, const float* budgets, const uint8_t* tier,
                         uint8_t* out, uint64_t capacity, uint64_t* layers_off) {
  int32_t G = ora_group_count(c, gran);
  if (G < 1) return ORA_ERR_INVALID_ARG;
  ora_plan_t* plans = (ora_plan_t*)malloc((size_t)G * sizeof(ora_plan_t));
  int st = plan_groups(c, gran, budgets, plans);
  if (st) { free(plans); return st; }
  int64_t L = c->num_layers, H = c->num_kv_heads, n = c->num_tokens;
  uint64_t* segtab = (uint64_t*)malloc((size_t)(4 * L * H) * sizeof(uint64_t));
  ora_ggeom g;
  grouped_layout(c, gran, plans, &g, segtab);
  *layers_off = g.layers_off;
  if (capacity < g.layers_off) { free(plans); free(segtab); return ORA_ERR_CAPACITY; }
  uint32_t* units = (uint32_t*)malloc((size_t)G * (size_t)n * 4);
  uint32_t* qrank = (uint32_t*)malloc((size_t)G * (size_t)n * 4);
  memset(out, 0, g.layers_off);
  write_grouped_meta(c, gran, budgets, plans, &g, segtab, tier, units, qrank, out);
  free(units); free(qrank); free(plans); free(segtab);
  return ORA_OK;
}
