/*
 * OSCAR CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU implementation of what the OSCAR serving
 * hot path computes (arXiv 2605.17757):
 *   - the cache update: rotate a bf16 key/value row by a fixed orthogonal matrix,
 *     clip it, quantize it to asymmetric INT2 per channel group with an fp16
 *     scale and zero, and pack four 2-bit codes per byte into a page
 *     (Sec. 4 "KV Cache Update"; App. "Scale Determination and Per-token
 *     Clipping Details"; Alg. 1 QuantizeAndWrite);
 *   - decode attention over the packed cache (Alg. 1 DecodeStep; Sec. 2
 *     attention definition), evaluated in fp64 in the rotated basis, plus a
 *     brute-force evaluation in the original basis;
 *   - plain fp64 attention over a bf16 paged cache (the bf16 baseline);
 *   - the mixed-precision cache of Sec. 4 "KV Cache Layout": bf16 sink and
 *     recent window around the INT2 history, the per-step demotion of the
 *     oldest window token (Alg. 1 DecodeStep) and decode attention over it;
 *   - quantizer variants: the per-token quantile clip of App. "Scale
 *     Determination and Per-token Clipping Details", bfloat16 scale/zero
 *     metadata, any group size dividing d, and an identity rotation (a NULL
 *     matrix: R_V absorbed into the projection weights, Sec. 4 "KV Cache Update").
 *
 * Only the test suite, the package smoke check and the benchmark's CPU-baseline
 * leg may load this library.  It shares no code, header or table with the GPU
 * library; the page byte layout is re-implemented here from its written
 * definition.
 *
 * Build: gcc -O2 -std=c11 -fopenmp -ffp-contract=off -fno-fast-math -shared -fPIC
 * (no FMA contraction, IEEE single/double arithmetic on SSE2).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------- */
/* Number formats (IEEE 754 binary16, bfloat16), written from the definitions */
/* ------------------------------------------------------------------------- */

static float f32_from_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t bits_from_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* bfloat16 is the upper half of a binary32: widening is exact. */
float oracle_bf16_to_f32(uint16_t h) { return f32_from_bits(((uint32_t)h) << 16); }

/* binary16 -> binary32 (exact). */
float oracle_f16_to_f32(uint16_t h) {
  uint32_t sign = (uint32_t)(h >> 15) & 1u;
  int32_t exp = (h >> 10) & 0x1f;
  uint32_t man = h & 0x3ffu;
  double v;
  if (exp == 0x1f) {
    if (man) return f32_from_bits(0x7fc00000u | (sign << 31));
    return sign ? -INFINITY : INFINITY;
  }
  if (exp == 0) v = ldexp((double)man, -24);                 /* subnormal: man * 2^-24 */
  else v = ldexp((double)(man | 0x400u), exp - 25);          /* (1.man) * 2^(exp-15) */
  return (float)(sign ? -v : v);
}

/* binary32 -> binary16, round to nearest, ties to even.  Values whose rounded
 * magnitude exceeds the largest finite binary16 become infinity (IEEE). */
uint16_t oracle_f32_to_f16_rne(float f) {
  uint32_t u = bits_from_f32(f);
  uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
  double a = fabs((double)f);                  /* exact */
  if (isnan(f)) return (uint16_t)(sign | 0x7e00u);
  if (isinf(f)) return (uint16_t)(sign | 0x7c00u);
  /* Quantum of the binary16 grid at magnitude a: 2^-24 below 2^-14 (subnormal
   * range), else 2^(floor(log2 a) - 10). */
  int e;
  frexp(a, &e);                                /* a = m * 2^e, m in [0.5,1) */
  int q_exp = (a < ldexp(1.0, -14)) ? -24 : (e - 1) - 10;
  double q = ldexp(1.0, q_exp);
  double n = a / q;                            /* exact: power-of-two division */
  double fl = floor(n);
  double r = n - fl;                           /* exact */
  double k = fl;
  if (r > 0.5 || (r == 0.5 && fmod(fl, 2.0) != 0.0)) k = fl + 1.0;
  double res = k * q;                          /* exact */
  if (res > 65504.0) return (uint16_t)(sign | 0x7c00u);
  if (res == 0.0) return sign;
  /* Encode res (a multiple of q, representable in binary16). */
  if (res < ldexp(1.0, -14)) {
    uint16_t man = (uint16_t)(res / ldexp(1.0, -24));
    return (uint16_t)(sign | man);
  }
  int re;
  double rm = frexp(res, &re);                 /* res = rm * 2^re, rm in [0.5,1) */
  int ebias = (re - 1) + 15;
  uint16_t man = (uint16_t)((rm * 2.0 - 1.0) * 1024.0);
  return (uint16_t)(sign | (uint16_t)(ebias << 10) | man);
}

/* binary32 -> bfloat16, round to nearest, ties to even: bfloat16 keeps the
 * binary32 exponent range and 8 significant bits, so the grid quantum at
 * magnitude a is 2^(floor(log2 a) - 7) for normal a and 2^-133 below 2^-126.
 * Values that round beyond the largest finite bfloat16 become infinity. */
uint16_t oracle_f32_to_bf16_rne(float f) {
  uint32_t u = bits_from_f32(f);
  uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
  double a = fabs((double)f);
  if (isnan(f)) return (uint16_t)(sign | 0x7fc0u);
  if (isinf(f)) return (uint16_t)(sign | 0x7f80u);
  if (a == 0.0) return sign;
  int e;
  frexp(a, &e);                                /* a = m * 2^e, m in [0.5,1) */
  int q_exp = (a < ldexp(1.0, -126)) ? -133 : (e - 1) - 7;
  double q = ldexp(1.0, q_exp);
  double n = a / q;                            /* exact */
  double fl = floor(n);
  double r = n - fl;
  double k = fl;
  if (r > 0.5 || (r == 0.5 && fmod(fl, 2.0) != 0.0)) k = fl + 1.0;
  double res = k * q;                          /* exact in double */
  double maxf = ldexp(255.0, 127 - 7);         /* (2 - 2^-7) * 2^127 */
  if (res > maxf) return (uint16_t)(sign | 0x7f80u);
  if (res == 0.0) return sign;
  /* res is on the bfloat16 grid, hence exactly a binary32 value whose low 16
   * bits are zero. */
  return (uint16_t)(sign | (uint16_t)(bits_from_f32((float)res) >> 16));
}

/* Saturating binary16 conversion used for stored scale and zero: finite values
 * beyond +-65504 are clamped to +-65504 first, then rounded. */
static uint16_t f16_sat(float f) {
  if (f > 65504.0f) f = 65504.0f;
  if (f < -65504.0f) f = -65504.0f;
  return oracle_f32_to_f16_rne(f);
}

/* Saturating bfloat16 conversion for stored scale and zero (a finite value
 * that would round to infinity is stored as the largest finite bfloat16). */
static uint16_t bf16_sat(float f) {
  uint16_t h = oracle_f32_to_bf16_rne(f);
  if ((h & 0x7fffu) == 0x7f80u) h = (uint16_t)((h & 0x8000u) | 0x7f7fu);
  return h;
}

/* Stored metadata formats: 0 = binary16, 1 = bfloat16. */
static uint16_t meta_store(int meta, float f) { return meta ? bf16_sat(f) : f16_sat(f); }
static float meta_load(int meta, uint16_t h) { return meta ? oracle_bf16_to_f32(h) : oracle_f16_to_f32(h); }
static int meta_saturates(int meta, float f) {
  if (!meta) return fabsf(f) > 65504.0f;
  return (oracle_f32_to_bf16_rne(f) & 0x7fffu) == 0x7f80u;
}

/* ------------------------------------------------------------------------- */
/* Page layout (the ABI, re-implemented from its definition)                  */
/* ------------------------------------------------------------------------- */
/*
 * The pool is num_pages pages; each page holds P token slots of Hkv heads.
 * Page-head block (page p, kv-head h) starts at byte (p*Hkv + h) * B_ph where
 * B_ph = 2*P*d/4 + 2*(d/G)*P*4.  Inside a block:
 *   [K codes]  P*d/4 bytes, token-major: byte t*(d/4) + c/4
 *   [V codes]  P*d/4 bytes, quad-major:  byte (c/4)*P + t
 *   [K s,z]    (d/G)*P entries of 4 bytes, group-major: entry g*P + t
 *   [V s,z]    same
 * A code byte holds channels 4j..4j+3 of one token, channel c in bits 2*(c%4)
 * (least significant first).  An s,z entry is two little-endian 16-bit values
 * (binary16 or bfloat16 by the metadata format): scale, then zero.
 */
size_t oracle_page_head_bytes(int d, int P, int G) {
  return (size_t)2 * P * (d / 4) + (size_t)2 * (d / G) * P * 4;
}

typedef struct { int d, Hkv, P, G, meta; } geo_t;

/* Rotation of KV head h: one shared [d][d] matrix (rph = 0) or one per KV head,
 * [Hkv][d][d] (rph = 1); NULL stays the identity. */
static const float *head_rot(const float *R, int rph, int h, int d) {
  return (R && rph) ? R + (size_t)h * d * d : R;
}

static size_t kcode_off(geo_t g, int t, int c) { return (size_t)t * (g.d / 4) + (size_t)(c / 4); }
static size_t vcode_off(geo_t g, int t, int c) {
  return (size_t)g.P * (g.d / 4) + (size_t)(c / 4) * g.P + (size_t)t;
}
static size_t sz_off(geo_t g, int is_v, int grp, int t) {
  size_t base = (size_t)2 * g.P * (g.d / 4) + (is_v ? (size_t)(g.d / g.G) * g.P * 4 : 0);
  return base + ((size_t)grp * g.P + (size_t)t) * 4;
}
static uint8_t *block_ptr(geo_t g, uint8_t *pages, int64_t page, int h) {
  return pages + ((size_t)page * g.Hkv + (size_t)h) * oracle_page_head_bytes(g.d, g.P, g.G);
}

static void put_code(geo_t g, uint8_t *blk, int is_v, int t, int c, unsigned code) {
  size_t off = is_v ? vcode_off(g, t, c) : kcode_off(g, t, c);
  unsigned sh = 2u * (unsigned)(c % 4);
  blk[off] = (uint8_t)((blk[off] & ~(3u << sh)) | ((code & 3u) << sh));
}
static unsigned get_code(geo_t g, const uint8_t *blk, int is_v, int t, int c) {
  size_t off = is_v ? vcode_off(g, t, c) : kcode_off(g, t, c);
  return (blk[off] >> (2u * (unsigned)(c % 4))) & 3u;
}
static void put_sz(geo_t g, uint8_t *blk, int is_v, int grp, int t, uint16_t s, uint16_t z) {
  uint8_t *p = blk + sz_off(g, is_v, grp, t);
  p[0] = (uint8_t)(s & 0xff); p[1] = (uint8_t)(s >> 8);
  p[2] = (uint8_t)(z & 0xff); p[3] = (uint8_t)(z >> 8);
}
static void get_sz(geo_t g, const uint8_t *blk, int is_v, int grp, int t, uint16_t *s, uint16_t *z) {
  const uint8_t *p = blk + sz_off(g, is_v, grp, t);
  *s = (uint16_t)(p[0] | (p[1] << 8));
  *z = (uint16_t)(p[2] | (p[3] << 8));
}

/* ------------------------------------------------------------------------- */
/* Cache update                                                               */
/* ------------------------------------------------------------------------- */

/* Rotation x~ = x R in row-vector convention (Sec. 2; App. scale determination):
 * x~_j = sum_c x_c R[c][j].  Products of a bf16-exact input and an fp32 matrix
 * entry are exact in fp64; they are summed in fp64 in ascending c and the sum is
 * rounded once to fp32.  R == NULL is the identity (x~ = x). */
void oracle_rotate_row(const float *x, const float *R, int d, float *out) {
  if (!R) {
    for (int j = 0; j < d; ++j) out[j] = x[j];
    return;
  }
  for (int j = 0; j < d; ++j) {
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc = acc + (double)x[c] * (double)R[(size_t)c * d + j];
    out[j] = (float)acc;
  }
}

/* Token-wise percentile clip threshold (App. "Scale Determination and Per-token
 * Clipping Details"): tau = quantile_rho of {|x~_c|, c < d}, read as the linear
 * interpolation between order statistics at position rho (d - 1) of the sorted
 * values a_0 <= ... <= a_{d-1}, in fp32 operations:
 *   pos = rho * (d - 1), k = floor(pos), f = pos - k,
 *   tau = a_k + f * (a_{k+1} - a_k)   (tau = a_k when k = d - 1). */
float oracle_token_quantile(const float *xt, int d, float rho) {
  float *a = (float *)malloc(sizeof(float) * (size_t)d);
  for (int c = 0; c < d; ++c) a[c] = fabsf(xt[c]);
  for (int i = 1; i < d; ++i) {                   /* insertion sort, ascending */
    float v = a[i];
    int j = i - 1;
    while (j >= 0 && a[j] > v) { a[j + 1] = a[j]; --j; }
    a[j + 1] = v;
  }
  float pos = rho * (float)(d - 1);
  int k = (int)floorf(pos);
  if (k > d - 1) k = d - 1;
  float tau;
  if (k >= d - 1) {
    tau = a[d - 1];
  } else {
    float f = pos - (float)k;
    float diff = a[k + 1] - a[k];
    float prod = f * diff;
    tau = a[k] + prod;
  }
  free(a);
  return tau;
}

/* Clip and quantize one rotated row (App. scale determination, per token and
 * per group of G channels):
 *   clip = 0: tau = rho * max|x~| over the group;
 *   clip = 1: tau = the token's rho-quantile of |x~| over all d channels
 *             (oracle_token_quantile), the same for every group;
 *   y = clip(x~, -tau, tau), a = min y, b = max y, s = (b - a)/3, z = -a/s,
 *   code = clip(round(y/s + z), 0, 3)
 * s and z are stored in the metadata format (meta 0: binary16, 1: bfloat16) and
 * the codes are computed with the stored values, so that dequantizing a code and
 * quantizing it again returns it.  A group whose stored scale would be zero gets
 * s = 1, z = -a, codes 0.  A zero point of zero is stored as +0.  Returns the
 * number of saturated metadata stores. */
int oracle_quantize_row(const float *xt, int d, int G, float rho, int meta, int clip,
                        uint8_t *codes, uint16_t *s_out, uint16_t *z_out) {
  int sat = 0;
  const float tau_tok = clip ? oracle_token_quantile(xt, d, rho) : 0.0f;
  for (int grp = 0; grp < d / G; ++grp) {
    const float *x = xt + grp * G;
    float tau;
    if (clip) {
      tau = tau_tok;
    } else {
      float m = 0.0f;
      for (int c = 0; c < G; ++c) { float ax = fabsf(x[c]); if (ax > m) m = ax; }
      tau = rho * m;
    }
    float a = 0.0f, b = 0.0f;
    for (int c = 0; c < G; ++c) {
      float y = fminf(fmaxf(x[c], -tau), tau);
      if (c == 0 || y < a) a = y;
      if (c == 0 || y > b) b = y;
    }
    float s = (b - a) / 3.0f;
    sat += meta_saturates(meta, s);
    uint16_t s16 = meta_store(meta, s);
    uint16_t z16;
    if ((s16 & 0x7fffu) == 0) {
      s16 = meta ? 0x3f80u : 0x3c00u;                 /* 1.0 */
      float na = -a + 0.0f;                           /* +0, never -0 */
      sat += meta_saturates(meta, na);
      z16 = meta_store(meta, na);
      for (int c = 0; c < G; ++c) codes[grp * G + c] = 0;
    } else {
      float sf = meta_load(meta, s16);
      float z = -a / sf;
      z = z + 0.0f;                                   /* +0, never -0 */
      sat += meta_saturates(meta, z);
      z16 = meta_store(meta, z);
      float zf = meta_load(meta, z16);
      for (int c = 0; c < G; ++c) {
        float y = fminf(fmaxf(x[c], -tau), tau);
        float u = y / sf;
        u = u + zf;
        float r = rintf(u);                           /* ties to even */
        if (r < 0.0f) r = 0.0f;
        if (r > 3.0f) r = 3.0f;
        codes[grp * G + c] = (uint8_t)r;
      }
    }
    s_out[grp] = s16;
    z_out[grp] = z16;
  }
  return sat;
}

/* Quantize n_tok new rows into the paged cache (Alg. 1 QuantizeAndWrite; the
 * fused cache-write of Sec. 4).  k, v: bf16 [n_tok, Hkv, d]; slot_mapping[i] =
 * page*P + offset.  Rk, Rv: fp32 [d, d] row-major (rph = 0) or [Hkv, d, d], one
 * per KV head (rph = 1), or NULL for the identity.
 * meta, clip: metadata format and clip rule of oracle_quantize_row.  Returns the
 * number of saturated metadata stores, or -1 on a slot outside the pool. */
int64_t oracle_kv_append(int d, int Hkv, int P, int G, int meta, int clip, int64_t num_pages,
                         uint8_t *pages, const uint16_t *k, const uint16_t *v,
                         const int64_t *slot_mapping, int n_tok, const float *Rk,
                         const float *Rv, float clip_k, float clip_v, int rph) {
  geo_t g = {d, Hkv, P, G, meta};
  int64_t sat = 0, bad = 0;
#pragma omp parallel for reduction(+ : sat, bad) schedule(static)
  for (int i = 0; i < n_tok; ++i) {
    int64_t slot = slot_mapping[i];
    if (slot < 0 || slot >= num_pages * (int64_t)P) { bad += 1; continue; }
    int64_t page = slot / P;
    int t = (int)(slot % P);
    float *x = (float *)malloc(sizeof(float) * (size_t)d * 2);
    float *xt = x + d;
    uint8_t *codes = (uint8_t *)malloc((size_t)d);
    uint16_t *s16 = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)(d / G) * 2);
    uint16_t *z16 = s16 + d / G;
    for (int h = 0; h < Hkv; ++h) {
      uint8_t *blk = block_ptr(g, pages, page, h);
      for (int is_v = 0; is_v < 2; ++is_v) {
        const uint16_t *src = (is_v ? v : k) + ((size_t)i * Hkv + (size_t)h) * d;
        for (int c = 0; c < d; ++c) x[c] = oracle_bf16_to_f32(src[c]);
        oracle_rotate_row(x, head_rot(is_v ? Rv : Rk, rph, h, d), d, xt);
        sat += oracle_quantize_row(xt, d, G, is_v ? clip_v : clip_k, meta, clip, codes, s16, z16);
        for (int c = 0; c < d; ++c) put_code(g, blk, is_v, t, c, codes[c]);
        for (int grp = 0; grp < d / G; ++grp) put_sz(g, blk, is_v, grp, t, s16[grp], z16[grp]);
      }
    }
    free(x); free(codes); free(s16);
  }
  return bad ? -1 : sat;
}

/* Read one token's codes and stored s,z back out of the cache (for tests). */
void oracle_read_token(int d, int Hkv, int P, int G, const uint8_t *pages, int64_t page, int h,
                       int t, int is_v, uint8_t *codes, uint16_t *s16, uint16_t *z16) {
  geo_t g = {d, Hkv, P, G, 0};
  const uint8_t *blk = block_ptr(g, (uint8_t *)pages, page, h);
  for (int c = 0; c < d; ++c) codes[c] = (uint8_t)get_code(g, blk, is_v, t, c);
  for (int grp = 0; grp < d / G; ++grp) get_sz(g, blk, is_v, grp, t, &s16[grp], &z16[grp]);
}

/* Dequantized rotated row Q(x~)_c = s*(code - z) in fp64 (App. scale
 * determination, dequantization map). */
static void dequant_rotated(geo_t g, const uint8_t *blk, int is_v, int t, double *out) {
  for (int grp = 0; grp < g.d / g.G; ++grp) {
    uint16_t s16, z16;
    get_sz(g, blk, is_v, grp, t, &s16, &z16);
    double s = (double)meta_load(g.meta, s16), z = (double)meta_load(g.meta, z16);
    for (int c = grp * g.G; c < (grp + 1) * g.G; ++c)
      out[c] = s * ((double)get_code(g, blk, is_v, t, c) - z);
  }
}

/* ------------------------------------------------------------------------- */
/* Decode attention                                                           */
/* ------------------------------------------------------------------------- */
/*
 * One decode step for B sequences (Alg. 1 DecodeStep; attention of Sec. 2).
 * Query head h reads KV head h / (Hq/Hkv).  Sequence b attends to its tokens
 * t < seq_lens[b]; token t lives in page block_table[b*max_pages + t/P] at slot
 * t % P.  The cached keys and values are K^ = Q(K~) Rk^T and V^ = Q(V~) Rv^T,
 * and the output is softmax(sm_scale * q K^T) V^.
 *
 * oracle_decode evaluates it in the rotated basis, using q K^T = (q Rk) Q(K~)^T
 * and S V^ = (S Q(V~)) Rv^T, all in fp64.  Output o[pair][d] (fp64) for the
 * listed (b, h) pairs; pairs == NULL means every (b, h) in order b-major.
 * Returns 0, or -1 on a page id outside the pool / a bad length.
 */
static int decode_pair(geo_t g, const uint8_t *pages, int64_t num_pages, const uint16_t *q,
                       int Hq, const int32_t *block_table, int max_pages,
                       const int32_t *seq_lens, const float *Rk, const float *Rv,
                       double sm_scale, int b, int h, double *o, int rph) {
  int d = g.d, group = Hq / g.Hkv, kvh = h / group;
  Rk = head_rot(Rk, rph, kvh, d);
  Rv = head_rot(Rv, rph, kvh, d);
  int len = seq_lens[b];
  if (len < 1 || len > max_pages * g.P) return -1;
  double *qt = (double *)calloc((size_t)d, sizeof(double));
  double *ot = (double *)calloc((size_t)d, sizeof(double));
  double *row = (double *)malloc(sizeof(double) * (size_t)d);
  double *score = (double *)malloc(sizeof(double) * (size_t)len);
  int rc = 0;
  const uint16_t *qr = q + ((size_t)b * Hq + (size_t)h) * d;
  for (int j = 0; j < d; ++j) {
    double acc = 0.0;
    if (!Rk) acc = (double)oracle_bf16_to_f32(qr[j]);     /* identity rotation */
    else
      for (int c = 0; c < d; ++c) acc += (double)oracle_bf16_to_f32(qr[c]) * (double)Rk[(size_t)c * d + j];
    qt[j] = acc;
  }
  double m = -INFINITY;
  for (int t = 0; t < len; ++t) {
    int32_t page = block_table[(size_t)b * max_pages + t / g.P];
    if (page < 0 || page >= num_pages) { rc = -1; goto done; }
    dequant_rotated(g, block_ptr(g, (uint8_t *)pages, page, kvh), 0, t % g.P, row);
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += qt[c] * row[c];
    score[t] = sm_scale * acc;
    if (score[t] > m) m = score[t];
  }
  double l = 0.0;
  for (int t = 0; t < len; ++t) {
    double p = exp(score[t] - m);
    l += p;
    int32_t page = block_table[(size_t)b * max_pages + t / g.P];
    dequant_rotated(g, block_ptr(g, (uint8_t *)pages, page, kvh), 1, t % g.P, row);
    for (int c = 0; c < d; ++c) ot[c] += p * row[c];
  }
  /* o = (ot / l) Rv^T, i.e. o_j = sum_c ot_c Rv[j][c] / l (Rv NULL: identity) */
  for (int j = 0; j < d; ++j) {
    double acc = 0.0;
    if (!Rv) acc = ot[j];
    else
      for (int c = 0; c < d; ++c) acc += ot[c] * (double)Rv[(size_t)j * d + c];
    o[j] = acc / l;
  }
done:
  free(qt); free(ot); free(row); free(score);
  return rc;
}

int oracle_decode(int d, int Hkv, int P, int G, int meta, int64_t num_pages,
                  const uint8_t *pages, const uint16_t *q, int B, int Hq,
                  const int32_t *block_table, int max_pages, const int32_t *seq_lens,
                  const float *Rk, const float *Rv, double sm_scale, const int32_t *pairs,
                  int n_pairs, double *out, int rph) {
  geo_t g = {d, Hkv, P, G, meta};
  if (Hq % Hkv) return -1;
  int n = pairs ? n_pairs : B * Hq;
  int bad = 0;
#pragma omp parallel for reduction(+ : bad) schedule(dynamic, 1)
  for (int i = 0; i < n; ++i) {
    int b = pairs ? pairs[2 * i] : i / Hq;
    int h = pairs ? pairs[2 * i + 1] : i % Hq;
    if (b < 0 || b >= B || h < 0 || h >= Hq) { bad += 1; continue; }
    if (decode_pair(g, pages, num_pages, q, Hq, block_table, max_pages, seq_lens, Rk, Rv,
                    sm_scale, b, h, out + (size_t)i * d, rph))
      bad += 1;
  }
  return bad ? -1 : 0;
}

/* Brute force in the original basis, following Alg. 1 DecodeStep literally:
 * dequantize the history, rotate it back (k^ = Q(k~) Rk^T, v^ = Q(v~) Rv^T),
 * then o = softmax(sm_scale * q k^T) v^.  O(len * d^2) per pair: tiny inputs. */
int oracle_decode_brute(int d, int Hkv, int P, int G, int meta, int64_t num_pages,
                        const uint8_t *pages, const uint16_t *q, int B, int Hq,
                        const int32_t *block_table, int max_pages, const int32_t *seq_lens,
                        const float *Rk, const float *Rv, double sm_scale, double *out,
                        int rph) {
  geo_t g = {d, Hkv, P, G, meta};
  if (Hq % Hkv) return -1;
  int group = Hq / Hkv;
  double *rot = (double *)malloc(sizeof(double) * (size_t)d);
  double *khat = (double *)malloc(sizeof(double) * (size_t)d);
  int rc = 0;
  for (int b = 0; b < B && !rc; ++b) {
    int len = seq_lens[b];
    if (len < 1 || len > max_pages * P) { rc = -1; break; }
    double *vhat = (double *)malloc(sizeof(double) * (size_t)len * d);
    double *score = (double *)malloc(sizeof(double) * (size_t)len);
    for (int h = 0; h < Hq && !rc; ++h) {
      int kvh = h / group;
      const float *Rkh = head_rot(Rk, rph, kvh, d), *Rvh = head_rot(Rv, rph, kvh, d);
      const uint16_t *qr = q + ((size_t)b * Hq + h) * d;
      double m = -INFINITY;
      for (int t = 0; t < len; ++t) {
        int32_t page = block_table[(size_t)b * max_pages + t / P];
        if (page < 0 || page >= num_pages) { rc = -1; break; }
        const uint8_t *blk = block_ptr(g, (uint8_t *)pages, page, kvh);
        dequant_rotated(g, blk, 0, t % P, rot);
        for (int j = 0; j < d; ++j) {          /* k^_j = sum_c Q(k~)_c Rk[j][c] */
          double acc = 0.0;
          if (!Rkh) acc = rot[j];
          else
            for (int c = 0; c < d; ++c) acc += rot[c] * (double)Rkh[(size_t)j * d + c];
          khat[j] = acc;
        }
        dequant_rotated(g, blk, 1, t % P, rot);
        for (int j = 0; j < d; ++j) {
          double acc = 0.0;
          if (!Rvh) acc = rot[j];
          else
            for (int c = 0; c < d; ++c) acc += rot[c] * (double)Rvh[(size_t)j * d + c];
          vhat[(size_t)t * d + j] = acc;
        }
        double s = 0.0;
        for (int j = 0; j < d; ++j) s += (double)oracle_bf16_to_f32(qr[j]) * khat[j];
        score[t] = sm_scale * s;
        if (score[t] > m) m = score[t];
      }
      if (rc) break;
      double l = 0.0;
      double *o = out + ((size_t)b * Hq + h) * d;
      for (int j = 0; j < d; ++j) o[j] = 0.0;
      for (int t = 0; t < len; ++t) {
        double p = exp(score[t] - m);
        l += p;
        for (int j = 0; j < d; ++j) o[j] += p * vhat[(size_t)t * d + j];
      }
      for (int j = 0; j < d; ++j) o[j] /= l;
    }
    free(vhat); free(score);
  }
  free(rot); free(khat);
  return rc;
}

/* ------------------------------------------------------------------------- */
/* bf16 baseline: plain attention over a bf16 paged cache                     */
/* ------------------------------------------------------------------------- */
/* bf16 page-head block (page p, kv-head h) at element (p*Hkv + h) * 2*P*d, for
 * P = 64, d = 128, in the library's tiled order (K then V, each as 16 tiles of
 * 64 x 8 elements):
 *   K(t, c) at ((u*4 + kc)*64 + lo + 16*hi)*8 + e,   t = 4*lo + u, c = 32*hi + 8*kc + e
 *   V(t, c) at P*d + ((ct*2 + kt)*64 + lo + 16*hi)*8 + e,
 *                                                  t = 16*hi + 8*kt + e, c = 16*ct + lo */
static size_t bf16_k_index(int t, int c) {
  int u = t & 3, lo = t >> 2, hi = c >> 5, kc = (c >> 3) & 3, e = c & 7;
  return ((size_t)(u * 4 + kc) * 64 + lo + 16 * hi) * 8 + e;
}
static size_t bf16_v_index(int t, int c) {
  int hi = t >> 4, kt = (t >> 3) & 1, e = t & 7, ct = c >> 4, lo = c & 15;
  return (size_t)64 * 128 + ((size_t)(ct * 2 + kt) * 64 + lo + 16 * hi) * 8 + e;
}
int oracle_bf16_decode(int d, int Hkv, int P, int64_t num_pages, const uint16_t *pages,
                       const uint16_t *q, int B, int Hq, const int32_t *block_table,
                       int max_pages, const int32_t *seq_lens, double sm_scale,
                       const int32_t *pairs, int n_pairs, double *out) {
  if (Hq % Hkv || d != 128 || P != 64) return -1;
  int group = Hq / Hkv;
  int n = pairs ? n_pairs : B * Hq;
  int bad = 0;
#pragma omp parallel for reduction(+ : bad) schedule(dynamic, 1)
  for (int i = 0; i < n; ++i) {
    int b = pairs ? pairs[2 * i] : i / Hq;
    int h = pairs ? pairs[2 * i + 1] : i % Hq;
    int len = (b >= 0 && b < B) ? seq_lens[b] : 0;
    if (h < 0 || h >= Hq || len < 1 || len > max_pages * P) { bad += 1; continue; }
    int kvh = h / group;
    const uint16_t *qr = q + ((size_t)b * Hq + h) * d;
    double *score = (double *)malloc(sizeof(double) * (size_t)len);
    double *o = out + (size_t)i * d;
    double m = -INFINITY;
    int ok = 1;
    for (int t = 0; t < len && ok; ++t) {
      int32_t page = block_table[(size_t)b * max_pages + t / P];
      if (page < 0 || page >= num_pages) { ok = 0; break; }
      const uint16_t *kb = pages + ((size_t)page * Hkv + kvh) * 2 * P * d;
      double s = 0.0;
      for (int c = 0; c < d; ++c)
        s += (double)oracle_bf16_to_f32(qr[c]) * (double)oracle_bf16_to_f32(kb[bf16_k_index(t % P, c)]);
      score[t] = sm_scale * s;
      if (score[t] > m) m = score[t];
    }
    if (ok) {
      double l = 0.0;
      for (int j = 0; j < d; ++j) o[j] = 0.0;
      for (int t = 0; t < len; ++t) {
        int32_t page = block_table[(size_t)b * max_pages + t / P];
        const uint16_t *vb = pages + ((size_t)page * Hkv + kvh) * 2 * P * d;
        double p = exp(score[t] - m);
        l += p;
        for (int j = 0; j < d; ++j) o[j] += p * (double)oracle_bf16_to_f32(vb[bf16_v_index(t % P, j)]);
      }
      for (int j = 0; j < d; ++j) o[j] /= l;
    } else {
      bad += 1;
    }
    free(score);
  }
  return bad ? -1 : 0;
}

/* Write bf16 rows into the bf16 paged cache (plain copy at slot_mapping). */
int oracle_bf16_append(int d, int Hkv, int P, int64_t num_pages, uint16_t *pages,
                       const uint16_t *k, const uint16_t *v, const int64_t *slot_mapping,
                       int n_tok) {
  if (d != 128 || P != 64) return -1;
  for (int i = 0; i < n_tok; ++i) {
    int64_t slot = slot_mapping[i];
    if (slot < 0 || slot >= num_pages * (int64_t)P) return -1;
    int64_t page = slot / P;
    int t = (int)(slot % P);
    for (int h = 0; h < Hkv; ++h) {
      uint16_t *blk = pages + ((size_t)page * Hkv + h) * 2 * P * d;
      const uint16_t *ks = k + ((size_t)i * Hkv + h) * d;
      const uint16_t *vs = v + ((size_t)i * Hkv + h) * d;
      for (int c = 0; c < d; ++c) {
        blk[bf16_k_index(t, c)] = ks[c];
        blk[bf16_v_index(t, c)] = vs[c];
      }
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Mixed-precision cache: bf16 sink, INT2 history, bf16 recent window         */
/* ------------------------------------------------------------------------- */
/*
 * Sec. 4 "KV Cache Layout": at decode length n the logical cache of a sequence
 * is the bf16 sink [0, S0), the INT2 history [S0, n - W) and the bf16 recent
 * window [n - W, n), with the bounds clamped: lo = min(S0, n), hi = max(lo, n - W);
 * history tokens live in the paged INT2 pool at their own positions.
 *
 * bf16 segment store (a layout of this library, not of the paper): for each
 * (sequence b, kv-head h) a block of 2*(S0+W) rows of d bf16 values, the K rows of
 * all slots and then the V rows:
 *   K(b, h, slot, c) at element (((b*Hkv + h)*2 + 0)*(S0+W) + slot)*d + c
 *   V(b, h, slot, c) at element (((b*Hkv + h)*2 + 1)*(S0+W) + slot)*d + c
 * A sink position p < S0 uses slot p; a position p >= S0 of the recent window
 * uses slot S0 + (p - S0) mod W.
 */
static int64_t seg_slot(int S0, int W, int64_t p) {
  if (p < 0) return -1;
  if (p < S0) return p;
  if (W <= 0) return -1;
  return S0 + (p - S0) % W;
}

static size_t seg_row(int d, int Hkv, int S0, int W, int b, int h, int is_v, int64_t slot) {
  return ((((size_t)b * Hkv + (size_t)h) * 2 + (size_t)is_v) * (size_t)(S0 + W) + (size_t)slot) *
         (size_t)d;
}

/* Copy bf16 rows (token i: k/v[i][Hkv][d]) of sequence seq_idx[i] at position
 * pos[i] into their sink or window slot.  Returns 0, or -1 on a bad index or a
 * position that has no bf16 slot (p >= S0 with W = 0). */
int oracle_seg_write(int d, int Hkv, int S0, int W, int B, uint16_t *seg, const uint16_t *k,
                     const uint16_t *v, const int32_t *seq_idx, const int64_t *pos, int n_tok) {
  for (int i = 0; i < n_tok; ++i) {
    int b = seq_idx[i];
    int64_t slot = seg_slot(S0, W, pos[i]);
    if (b < 0 || b >= B || slot < 0) return -1;
    for (int h = 0; h < Hkv; ++h) {
      memcpy(seg + seg_row(d, Hkv, S0, W, b, h, 0, slot), k + ((size_t)i * Hkv + h) * d,
             sizeof(uint16_t) * (size_t)d);
      memcpy(seg + seg_row(d, Hkv, S0, W, b, h, 1, slot), v + ((size_t)i * Hkv + h) * d,
             sizeof(uint16_t) * (size_t)d);
    }
  }
  return 0;
}

/* The cache side of Alg. 1 DecodeStep for one new token per sequence, at
 * position p = seq_lens[b] - 1 (k_new, v_new: bf16 [B][Hkv][d]):
 *   p < S0          -> the token joins the bf16 sink;
 *   p >= S0, W = 0  -> the token is quantized into the INT2 history at once;
 *   otherwise       -> the token joins the recent window; if the window then
 *                      holds more than W tokens (p - W >= S0), its oldest token,
 *                      at position p - W, is quantized into the INT2 history
 *                      (QuantizeAndWrite) before its slot is reused.
 * Quantization is the cache update above (rotation from the bf16 row).
 * Returns the number of saturated fp16 stores, or -1 on a bad length / page. */
int64_t oracle_mixed_update(int d, int Hkv, int P, int G, int meta, int clip, int64_t num_pages,
                            uint8_t *pages,
                            uint16_t *seg, int S0, int W, int B, const uint16_t *k_new,
                            const uint16_t *v_new, const int32_t *block_table, int max_pages,
                            const int32_t *seq_lens, const float *Rk, const float *Rv,
                            float clip_k, float clip_v, int rph) {
  int64_t sat = 0;
  uint16_t *ko = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)Hkv * d);
  uint16_t *vo = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)Hkv * d);
  int rc = 0;
  for (int b = 0; b < B && !rc; ++b) {
    int64_t p = (int64_t)seq_lens[b] - 1;
    if (p < 0 || p >= (int64_t)max_pages * P) { rc = -1; break; }
    const uint16_t *kn = k_new + (size_t)b * Hkv * d;
    const uint16_t *vn = v_new + (size_t)b * Hkv * d;
    int64_t quant_pos = -1;           /* position quantized into INT2 this step */
    const uint16_t *qk = NULL, *qv = NULL;
    if (p >= S0 && W == 0) {
      quant_pos = p; qk = kn; qv = vn;
    } else if (p >= S0 && p - W >= S0) {
      int64_t slot = seg_slot(S0, W, p - W);
      for (int h = 0; h < Hkv; ++h) {
        memcpy(ko + (size_t)h * d, seg + seg_row(d, Hkv, S0, W, b, h, 0, slot), sizeof(uint16_t) * (size_t)d);
        memcpy(vo + (size_t)h * d, seg + seg_row(d, Hkv, S0, W, b, h, 1, slot), sizeof(uint16_t) * (size_t)d);
      }
      quant_pos = p - W; qk = ko; qv = vo;
    }
    if (quant_pos >= 0) {
      int32_t page = block_table[(size_t)b * max_pages + quant_pos / P];
      int64_t slot = (int64_t)page * P + quant_pos % P;
      int64_t r = oracle_kv_append(d, Hkv, P, G, meta, clip, num_pages, pages, qk, qv, &slot, 1, Rk, Rv,
                                   clip_k, clip_v, rph);
      if (r < 0) { rc = -1; break; }
      sat += r;
    }
    if (p < S0 || W > 0) {
      int32_t bb = b;
      if (oracle_seg_write(d, Hkv, S0, W, B, seg, kn, vn, &bb, &p, 1)) { rc = -1; break; }
    }
  }
  free(ko); free(vo);
  return rc ? -1 : sat;
}

/* Decode attention over the mixed cache (Alg. 1 DecodeStep: concatenate the bf16
 * sink, the dequantized and back-rotated INT2 history and the bf16 recent window,
 * then softmax(sm_scale * q K^T) V), fp64.  The history part is evaluated in the
 * rotated basis as in oracle_decode; the bf16 parts in the original basis:
 *   o = ( [sum_hist p_t Q(v~_t)] Rv^T + sum_bf16 p_t v_t ) / sum_t p_t.
 * Output layout as oracle_decode.  Returns 0 or -1. */
int oracle_decode_mixed(int d, int Hkv, int P, int G, int meta, int64_t num_pages,
                        const uint8_t *pages,
                        const uint16_t *seg, int S0, int W, const uint16_t *q, int B, int Hq,
                        const int32_t *block_table, int max_pages, const int32_t *seq_lens,
                        const float *Rk, const float *Rv, double sm_scale, const int32_t *pairs,
                        int n_pairs, double *out, int rph) {
  geo_t g = {d, Hkv, P, G, meta};
  if (Hq % Hkv || S0 < 0 || W < 0) return -1;
  int group = Hq / Hkv;
  int n = pairs ? n_pairs : B * Hq;
  int bad = 0;
#pragma omp parallel for reduction(+ : bad) schedule(dynamic, 1)
  for (int i = 0; i < n; ++i) {
    int b = pairs ? pairs[2 * i] : i / Hq;
    int h = pairs ? pairs[2 * i + 1] : i % Hq;
    int len = (b >= 0 && b < B) ? seq_lens[b] : 0;
    if (h < 0 || h >= Hq || len < 1 || len > max_pages * P) { bad += 1; continue; }
    int kvh = h / group;
    const float *Rkh = head_rot(Rk, rph, kvh, d), *Rvh = head_rot(Rv, rph, kvh, d);
    int lo = len < S0 ? len : S0;
    int hi = len - W > lo ? len - W : lo;
    const uint16_t *qr = q + ((size_t)b * Hq + h) * d;
    double *qd = (double *)malloc(sizeof(double) * (size_t)d);
    double *qt = (double *)calloc((size_t)d, sizeof(double));
    double *row = (double *)malloc(sizeof(double) * (size_t)d);
    double *ot = (double *)calloc((size_t)d, sizeof(double));
    double *op = (double *)calloc((size_t)d, sizeof(double));
    double *score = (double *)malloc(sizeof(double) * (size_t)len);
    for (int c = 0; c < d; ++c) qd[c] = (double)oracle_bf16_to_f32(qr[c]);
    for (int j = 0; j < d; ++j) {
      double acc = 0.0;
      if (!Rkh) acc = qd[j];
      else
        for (int c = 0; c < d; ++c) acc += qd[c] * (double)Rkh[(size_t)c * d + j];
      qt[j] = acc;
    }
    double m = -INFINITY;
    int ok = 1;
    for (int t = 0; t < len && ok; ++t) {
      double acc = 0.0;
      if (t < lo || t >= hi) {
        const uint16_t *kr = seg + seg_row(d, Hkv, S0, W, b, kvh, 0, seg_slot(S0, W, t));
        for (int c = 0; c < d; ++c) acc += qd[c] * (double)oracle_bf16_to_f32(kr[c]);
      } else {
        int32_t page = block_table[(size_t)b * max_pages + t / P];
        if (page < 0 || page >= num_pages) { ok = 0; break; }
        dequant_rotated(g, block_ptr(g, (uint8_t *)pages, page, kvh), 0, t % P, row);
        for (int c = 0; c < d; ++c) acc += qt[c] * row[c];
      }
      score[t] = sm_scale * acc;
      if (score[t] > m) m = score[t];
    }
    if (ok) {
      double l = 0.0;
      for (int t = 0; t < len; ++t) {
        double pt = exp(score[t] - m);
        l += pt;
        if (t < lo || t >= hi) {
          const uint16_t *vr = seg + seg_row(d, Hkv, S0, W, b, kvh, 1, seg_slot(S0, W, t));
          for (int c = 0; c < d; ++c) op[c] += pt * (double)oracle_bf16_to_f32(vr[c]);
        } else {
          int32_t page = block_table[(size_t)b * max_pages + t / P];
          dequant_rotated(g, block_ptr(g, (uint8_t *)pages, page, kvh), 1, t % P, row);
          for (int c = 0; c < d; ++c) ot[c] += pt * row[c];
        }
      }
      double *o = out + (size_t)i * d;
      for (int j = 0; j < d; ++j) {
        double acc = 0.0;
        if (!Rvh) acc = ot[j];
        else
          for (int c = 0; c < d; ++c) acc += ot[c] * (double)Rvh[(size_t)j * d + c];
        o[j] = (acc + op[j]) / l;
      }
    } else {
      bad += 1;
    }
    free(qd); free(qt); free(row); free(ot); free(op); free(score);
  }
  return bad ? -1 : 0;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Thread count of the parallel loops that follow (n >= 1); timing only. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------- */
/* Offline calibration (Sec. 3 "Algorithm Design: Offline Calibration and     */
/* Justification"; Alg. 1 Calibrate)                                          */
/* ------------------------------------------------------------------------- */

static double bf16d(uint16_t h) { return (double)oracle_bf16_to_f32(h); }

/* Query-aware key target covariance, GQA-averaged as in the appendix worked
 * example: C_Q = (1/Hkv) sum_h (1/(T g)) sum_{i in group h} sum_t q_{t,i}^T q_{t,i},
 * g = Hq/Hkv query heads per KV head, q: bf16 [T][Hq][d].  C: [d][d].  Returns
 * -1 on a bad shape. */
int oracle_query_cov(const uint16_t *q, int64_t T, int Hq, int Hkv, int d, double *C) {
  if (T < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv || d < 1) return -1;
  const int g = Hq / Hkv;
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < d; ++i) {
    double *outer = (double *)calloc((size_t)d, sizeof(double));
    double *grp = (double *)malloc(sizeof(double) * (size_t)d);
    for (int h = 0; h < Hkv; ++h) {
      for (int j = 0; j < d; ++j) grp[j] = 0.0;
      for (int qi = h * g; qi < (h + 1) * g; ++qi)
        for (int64_t t = 0; t < T; ++t) {
          const uint16_t *row = q + ((size_t)t * Hq + qi) * d;
          const double xi = bf16d(row[i]);
          for (int j = 0; j < d; ++j) grp[j] = grp[j] + xi * bf16d(row[j]);
        }
      for (int j = 0; j < d; ++j) outer[j] = outer[j] + grp[j] / ((double)T * (double)g);
    }
    for (int j = 0; j < d; ++j) C[(size_t)i * d + j] = outer[j] / (double)Hkv;
    free(outer); free(grp);
  }
  return 0;
}

/* Attention output rows of the calibration pass (Alg. 1 Calibrate):
 * S = softmax_row(Q_i K_h^T / sqrt(d) + M) for query head i and its KV head
 * h = i / g, M = 0 on keys j <= t and -inf on j > t when causal (no mask
 * otherwise), o_{t,i} = sum_j S[t][j] v_{j,h}.  fp64 throughout: scores summed
 * in ascending channel order, softmax with the row maximum subtracted.
 * q: bf16 [T][Hq][d], k, v: bf16 [T][Hkv][d].  pairs: (t, i) int32 pairs, or
 * NULL for every (t, i) in t-major order.  out: [n][d].  Returns -1 on a bad
 * shape or pair. */
int oracle_attn_rows(const uint16_t *q, const uint16_t *k, const uint16_t *v, int64_t T, int Hq,
                     int Hkv, int d, int causal, const int32_t *pairs, int64_t n_pairs,
                     double *out) {
  if (T < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv || d < 1) return -1;
  const int g = Hq / Hkv;
  const int64_t n = pairs ? n_pairs : T * Hq;
  int64_t bad = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(+ : bad)
  for (int64_t p = 0; p < n; ++p) {
    const int64_t t = pairs ? pairs[2 * p] : p / Hq;
    const int i = pairs ? pairs[2 * p + 1] : (int)(p % Hq);
    double *o = out + (size_t)p * d;
    if (t < 0 || t >= T || i < 0 || i >= Hq) { bad += 1; continue; }
    const int h = i / g;
    const int64_t nk = causal ? t + 1 : T;
    double *s = (double *)malloc(sizeof(double) * (size_t)nk);
    const uint16_t *qr = q + ((size_t)t * Hq + i) * d;
    double m = -INFINITY;
    for (int64_t j = 0; j < nk; ++j) {
      const uint16_t *kr = k + ((size_t)j * Hkv + h) * d;
      double dot = 0.0;
      for (int c = 0; c < d; ++c) dot = dot + bf16d(qr[c]) * bf16d(kr[c]);
      s[j] = dot / sqrt((double)d);
      if (s[j] > m) m = s[j];
    }
    double den = 0.0;
    for (int64_t j = 0; j < nk; ++j) { s[j] = exp(s[j] - m); den = den + s[j]; }
    for (int c = 0; c < d; ++c) o[c] = 0.0;
    for (int64_t j = 0; j < nk; ++j) {
      const uint16_t *vr = v + ((size_t)j * Hkv + h) * d;
      const double w = s[j] / den;
      for (int c = 0; c < d; ++c) o[c] = o[c] + w * bf16d(vr[c]);
    }
    free(s);
  }
  return bad ? -1 : 0;
}

/* Score-aware value target covariance (Sec. 3): C_S = (1/N) V^T S^T S V, i.e.
 * the second moment of the attention outputs o = S V, GQA-averaged like C_Q:
 * C_S = (1/Hkv) sum_h (1/(T g)) sum_{i in group h} sum_t o_{t,i}^T o_{t,i}. */
int oracle_score_cov(const uint16_t *q, const uint16_t *k, const uint16_t *v, int64_t T, int Hq,
                     int Hkv, int d, int causal, double *C) {
  if (T < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv || d < 1) return -1;
  const int g = Hq / Hkv;
  double *O = (double *)malloc(sizeof(double) * (size_t)T * Hq * d);
  if (!O) return -1;
  if (oracle_attn_rows(q, k, v, T, Hq, Hkv, d, causal, NULL, 0, O)) { free(O); return -1; }
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < d; ++i) {
    double *outer = (double *)calloc((size_t)d, sizeof(double));
    double *grp = (double *)malloc(sizeof(double) * (size_t)d);
    for (int h = 0; h < Hkv; ++h) {
      for (int j = 0; j < d; ++j) grp[j] = 0.0;
      for (int qi = h * g; qi < (h + 1) * g; ++qi)
        for (int64_t t = 0; t < T; ++t) {
          const double *row = O + ((size_t)t * Hq + qi) * d;
          for (int j = 0; j < d; ++j) grp[j] = grp[j] + row[i] * row[j];
        }
      for (int j = 0; j < d; ++j) outer[j] = outer[j] + grp[j] / ((double)T * (double)g);
    }
    for (int j = 0; j < d; ++j) C[(size_t)i * d + j] = outer[j] / (double)Hkv;
    free(outer); free(grp);
  }
  free(O);
  return 0;
}

/* Normalized Walsh-Hadamard matrix by the Sylvester recursion of the appendix
 * (App. "Hadamard transform"): H_1 = [1], H_2m = [[H_m, H_m], [H_m, -H_m]] / sqrt 2.
 * d must be a power of two.  H: [d][d]. */
int oracle_hadamard(int d, double *H) {
  if (d < 1 || (d & (d - 1))) return -1;
  H[0] = 1.0;
  for (int m = 1; m < d; m *= 2) {
    /* grow the leading m x m block in place, from the bottom-right corner */
    for (int i = m - 1; i >= 0; --i)
      for (int j = m - 1; j >= 0; --j) {
        const double x = H[(size_t)i * d + j] / sqrt(2.0);
        H[(size_t)i * d + j] = x;
        H[(size_t)i * d + j + m] = x;
        H[(size_t)(i + m) * d + j] = x;
        H[(size_t)(i + m) * d + j + m] = -x;
      }
  }
  return 0;
}

/* Bit reversal of k over log2(d) bits. */
static int bitrev(int k, int d) {
  int r = 0;
  for (int b = 1; b < d; b <<= 1) { r = (r << 1) | (k & 1); k >>= 1; }
  return r;
}

/* Permuted bit-reversal matrix P_br (App. "P_K"): the eigenvector of the k-th
 * largest eigenvalue goes to position bitrev(k), i.e. (x P)_{bitrev(k)} = x_k:
 * P[k][bitrev(k)] = 1.  P: [d][d]. */
int oracle_bit_reversal(int d, double *P) {
  if (d < 1 || (d & (d - 1))) return -1;
  for (size_t i = 0; i < (size_t)d * d; ++i) P[i] = 0.0;
  for (int kk = 0; kk < d; ++kk) P[(size_t)kk * d + bitrev(kk, d)] = 1.0;
  return 0;
}

/* Composed rotation (Eq. method_composed_rot): R = U H_Had P_br, fp64 matrix
 * products in ascending summation order.  U: [d][d], eigenvectors in columns
 * sorted by descending eigenvalue.  R: [d][d]. */
int oracle_compose(const double *U, int d, double *R) {
  if (d < 1 || (d & (d - 1))) return -1;
  double *H = (double *)malloc(sizeof(double) * (size_t)d * d);
  double *P = (double *)malloc(sizeof(double) * (size_t)d * d);
  double *UH = (double *)malloc(sizeof(double) * (size_t)d * d);
  oracle_hadamard(d, H);
  oracle_bit_reversal(d, P);
  for (int i = 0; i < d; ++i)
    for (int j = 0; j < d; ++j) {
      double acc = 0.0;
      for (int c = 0; c < d; ++c) acc = acc + U[(size_t)i * d + c] * H[(size_t)c * d + j];
      UH[(size_t)i * d + j] = acc;
    }
  for (int i = 0; i < d; ++i)
    for (int j = 0; j < d; ++j) {
      double acc = 0.0;
      for (int c = 0; c < d; ++c) acc = acc + UH[(size_t)i * d + c] * P[(size_t)c * d + j];
      R[(size_t)i * d + j] = acc;
    }
  free(H); free(P); free(UH);
  return 0;
}

/* Clip calibration (Alg. 1 CalibrateClip, whose procedure the paper leaves
 * open; read here as: pick the candidate ratio with the smallest quantization
 * error of the rotated calibration rows).  For each candidate ratio rho_n:
 *   err[n] = mean over rows r and channels c of (x~_{r,c} - s_g (code_{r,c} - z_g))^2
 * with x~ = x R rounded to fp32 (oracle_rotate_row) and (code, s, z) from
 * oracle_quantize_row with rho_n, s and z read back from their stored format.
 * x: bf16 [n_rows][d], row r of KV head r % Hkv (rotated by that head's matrix
 * when rph = 1).  Rows are summed in order (deterministic).  Returns -1 on a bad
 * shape. */
int oracle_clip_errors(const uint16_t *x, int64_t n_rows, int d, const float *R, int G, int meta,
                       int clip, const float *cands, int n_cands, double *err, int Hkv,
                       int rph) {
  if (n_rows < 1 || d < 1 || G < 1 || d % G || n_cands < 1 || Hkv < 1) return -1;
  double *per = (double *)malloc(sizeof(double) * (size_t)n_rows * n_cands);
  if (!per) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n_rows; ++r) {
    float *xr = (float *)malloc(sizeof(float) * (size_t)d);
    float *xt = (float *)malloc(sizeof(float) * (size_t)d);
    uint8_t *codes = (uint8_t *)malloc((size_t)d);
    uint16_t *s16 = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)(d / G));
    uint16_t *z16 = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)(d / G));
    for (int c = 0; c < d; ++c) xr[c] = oracle_bf16_to_f32(x[(size_t)r * d + c]);
    oracle_rotate_row(xr, head_rot(R, rph, (int)(r % Hkv), d), d, xt);
    for (int n = 0; n < n_cands; ++n) {
      oracle_quantize_row(xt, d, G, cands[n], meta, clip, codes, s16, z16);
      double e = 0.0;
      for (int c = 0; c < d; ++c) {
        const double s = (double)meta_load(meta, s16[c / G]);
        const double z = (double)meta_load(meta, z16[c / G]);
        const double diff = (double)xt[c] - s * ((double)codes[c] - z);
        e = e + diff * diff;
      }
      per[(size_t)r * n_cands + n] = e;
    }
    free(xr); free(xt); free(codes); free(s16); free(z16);
  }
  for (int n = 0; n < n_cands; ++n) {
    double acc = 0.0;
    for (int64_t r = 0; r < n_rows; ++r) acc = acc + per[(size_t)r * n_cands + n];
    err[n] = acc / ((double)n_rows * (double)d);
  }
  free(per);
  return 0;
}
