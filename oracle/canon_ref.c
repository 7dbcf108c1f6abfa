/*
 * canon_ref.c - CPU oracle of the canonical-order training step (CANON-v1).
 *
 * TEST INFRASTRUCTURE.  This library exists to check the GPU library; only the
 * tests, the smoke check and the CPU-baseline leg of the benchmark load it.  It
 * shares no source with the GPU path.
 *
 * Every floating-point operation below is spelled out.  Each one follows rule R0
 * (IEEE-754 binary32, round to nearest even; subnormal inputs read as zero of the
 * same sign; a result whose rounding to 24 significant bits with unbounded
 * exponent is below 2^-126 in magnitude becomes zero of the same sign).  This is
 * the paper's choice to flush subnormals everywhere (Section "Reproducible
 * Operations", paragraph on subnormals, and its Table of techniques), with the
 * tininess test that gfx950 applies in flush mode.
 *
 * Reductions follow rule R1: the terms of a sum, in the order of their logical
 * index, are cut into chunks of 32; each chunk is a left-to-right chain started
 * at +0 (fused multiply-add for bf16 x bf16 products, separate multiply and add
 * otherwise, the paper's fixed-order and single-convention rules); the chunk
 * partials are combined by the binary-carry fold of the paper's Algorithm 2
 * (TreeFold), pushed in ascending chunk order.
 *
 * Compiled with -ffp-contract=off and without fast-math, so the compiler neither
 * fuses nor reorders any of these operations.
 */
#include "canon_ref.h"

#include <math.h>
#include <stdio.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

#define CHUNK 32
#define TINY 0x1p-126f

/* ======================================================================== */
/* R0: primitives                                                            */
/* ======================================================================== */

static inline float f_from_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static inline uint32_t f_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* Subnormal input read as zero of the same sign. */
static inline float daz(float x) { return (x != 0.0f && fabsf(x) < TINY) ? copysignf(0.0f, x) : x; }

/* Round an exactly known real value x (held exactly in a double) to binary32 under R0. */
static float round_exact_double(double x) {
  if (x == 0.0 || isinf(x) || isnan(x)) return (float)x;
  double ax = fabs(x);
  if (ax < 0x1p-127) return x < 0 ? -0.0f : 0.0f;
  /* 24-bit rounding with unbounded exponent, moved into the normal float range by an exact scaling */
  float scaled = (float)(ax * 0x1p64);
  if (scaled < 0x1p-62f) return x < 0 ? -0.0f : 0.0f;
  /* not tiny: the ordinary rounding gives the same value */
  return (float)x;
}

/* Round the exact value s + e (a double-double with |e| <= ulp(s)/2, s = RN53(s+e)) under R0. */
static float round_double_double(double s, double e) {
  double as = fabs(s);
  if (as < 0x1p-140) return s < 0 ? -0.0f : 0.0f;       /* far below the normal range */
  double sc = (as < 0x1p-100) ? 0x1p150 : 1.0;          /* exact scaling into the float normal range */
  double S = s * sc, E = e * sc;
  float r = (float)S;                                   /* ties-to-even on S alone */
  double rd = (double)r;
  if (!isinf(r) && rd != S) {
    float lo, hi;
    if (rd < S) { lo = r; hi = nextafterf(r, INFINITY); }
    else { hi = r; lo = nextafterf(r, -INFINITY); }
    double mid = ((double)lo + (double)hi) * 0.5;       /* exact */
    if (S == mid) {                                     /* the tail e decides a tie on S */
      if (E > 0) r = hi;
      else if (E < 0) r = lo;
    }
  }
  if (isinf(r)) return r;
  double ar = fabs((double)r) / sc;
  if (ar < 0x1p-126) return s < 0 ? -0.0f : 0.0f;
  return (float)((double)r / sc);
}

float cref_add(float a, float b) {
  a = daz(a);
  b = daz(b);
  /* both operands are multiples of 2^-149, so a sum below 2^-126 is exact and therefore tiny */
  float r = a + b;
  if (r != 0.0f && fabsf(r) < TINY) r = copysignf(0.0f, r);
  return r;
}

float cref_sub(float a, float b) { return cref_add(a, -b); }

float cref_mul(float a, float b) {
  a = daz(a);
  b = daz(b);
  return round_exact_double((double)a * (double)b); /* 24 x 24 bits: the double product is exact */
}

float cref_fma(float a, float b, float c) {
  a = daz(a);
  b = daz(b);
  c = daz(c);
  float p = a * b;
  double pd = (double)a * (double)b; /* exact */
  if ((double)p == pd && (p == 0.0f || fabsf(p) >= TINY)) {
    /* the product is a normal float (always so for bf16 x bf16 away from underflow): the fused
       result is the R0 rounding of c + p, which is cref_add */
    return cref_add(c, p);
  }
  double cd = (double)c;
  double s = pd + cd; /* TwoSum: s + e == pd + cd exactly */
  double bv = s - pd;
  double e = (pd - (s - bv)) + (cd - bv);
  if (s == 0.0 && e == 0.0) return fmaf(a, b, c); /* exact zero: IEEE sign rule */
  return round_double_double(s, e);
}

float cref_div(float a, float b) {
  a = daz(a);
  b = daz(b);
  double q = (double)a / (double)b;
  if (q == 0.0 || isinf(q) || isnan(q)) return (float)q;
  /* RN24(RN53(x)) == RN24(x) for a quotient of binary32 numbers (53 >= 2*24+2) */
  double qs = ((double)a * 0x1p100) / (double)b;
  if (fabsf((float)qs) < 0x1p-26f) return q < 0 ? -0.0f : 0.0f;
  return (float)q;
}

float cref_sqrt(float a) {
  a = daz(a);
  return sqrtf(a); /* correctly rounded; a square root of a normal float is never tiny */
}

uint16_t cref_bf16(float x) {
  uint32_t u = f_bits(daz(x));
  u = u + 0x7FFFu + ((u >> 16) & 1u); /* round to nearest even on the 16 dropped bits */
  return (uint16_t)(u >> 16);
}

static inline float widen(uint16_t h) { return daz(f_from_bits((uint32_t)h << 16)); }

/* ======================================================================== */
/* R4: canonical functions                                                   */
/* ======================================================================== */

/* cexp: Cody-Waite reduction by ln 2 split in two parts, degree-7 Taylor polynomial
   by Horner in separate multiplies and adds, exact scaling by 2^k. */
static const uint32_t EXP_L2E = 0x3FB8AA3Bu;    /* RN32(1/ln 2) */
static const uint32_t EXP_LN2_HI = 0x3F317200u; /* ln 2 cut to 15 significant bits */
static const uint32_t EXP_LN2_LO = 0x35BFBE8Eu; /* RN32(ln 2 - LN2_HI) */
static const uint32_t EXP_C[8] = {               /* RN32(1/n!) for n = 0..7 */
    0x3F800000u, 0x3F800000u, 0x3F000000u, 0x3E2AAAABu,
    0x3D2AAAABu, 0x3C088889u, 0x3AB60B61u, 0x39500D01u};

float cref_exp(float x) {
  x = daz(x);
  float t = cref_mul(x, f_from_bits(EXP_L2E));
  float kf = nearbyintf(t); /* nearest integer, ties to even (default rounding mode); exact */
  if (kf > 127.0f) return INFINITY;
  if (kf < -125.0f) return 0.0f;
  float r = cref_sub(cref_sub(x, cref_mul(kf, f_from_bits(EXP_LN2_HI))), cref_mul(kf, f_from_bits(EXP_LN2_LO)));
  float p = f_from_bits(EXP_C[7]);
  for (int i = 6; i >= 0; --i) p = cref_add(cref_mul(p, r), f_from_bits(EXP_C[i]));
  int k = (int)kf;
  float scale = f_from_bits((uint32_t)(k + 127) << 23);
  return cref_mul(p, scale);
}

/* clog: x = 2^e f with f in (sqrt(1/2), sqrt(2)], s = (f-1)/(f+1), log f = 2 atanh(s) by the odd
   series up to s^11, then e ln 2 added in two parts. */
static const uint32_t LOG_SQRT2 = 0x3FB504F3u;            /* RN32(sqrt 2) */
static const uint32_t LOG_INV[5] = {0x3EAAAAABu, 0x3E4CCCCDu, 0x3E124925u, 0x3DE38E39u,
                                    0x3DBA2E8Cu}; /* RN32(1/3), 1/5, 1/7, 1/9, 1/11 */

float cref_log(float x) {
  x = daz(x);
  if (x == 0.0f) return -INFINITY;
  if (x < 0.0f || isnan(x)) return NAN;
  if (isinf(x)) return x;
  uint32_t u = f_bits(x);
  int e = (int)((u >> 23) & 0xFFu) - 127;
  float f = f_from_bits((u & 0x7FFFFFu) | 0x3F800000u);
  if (f > f_from_bits(LOG_SQRT2)) {
    f = cref_mul(f, 0.5f);
    e += 1;
  }
  float s = cref_div(cref_sub(f, 1.0f), cref_add(f, 1.0f));
  float z = cref_mul(s, s);
  float q = f_from_bits(LOG_INV[4]);
  for (int i = 3; i >= 0; --i) q = cref_add(cref_mul(q, z), f_from_bits(LOG_INV[i]));
  q = cref_add(cref_mul(q, z), 1.0f);
  float lf = cref_mul(cref_add(s, s), q);
  float ef = (float)e;
  return cref_add(cref_mul(ef, f_from_bits(EXP_LN2_HI)), cref_add(cref_mul(ef, f_from_bits(EXP_LN2_LO)), lf));
}

float cref_sigmoid(float x) {
  x = daz(x);
  return cref_div(1.0f, cref_add(1.0f, cref_exp(-x)));
}

float cref_silu(float x) { return cref_mul(x, cref_sigmoid(x)); }

int cref_prim(int32_t op, int64_t n, const float* a, const float* b, const float* c, float* out) {
  if (n < 0 || op < 0 || op > 10) return -1;
  for (int64_t i = 0; i < n; ++i) {
    switch (op) {
      case 0: out[i] = cref_add(a[i], b[i]); break;
      case 1: out[i] = cref_sub(a[i], b[i]); break;
      case 2: out[i] = cref_mul(a[i], b[i]); break;
      case 3: out[i] = cref_fma(a[i], b[i], c[i]); break;
      case 4: out[i] = cref_div(a[i], b[i]); break;
      case 5: out[i] = cref_sqrt(a[i]); break;
      case 6: out[i] = cref_exp(a[i]); break;
      case 7: out[i] = cref_log(a[i]); break;
      case 8: out[i] = cref_sigmoid(a[i]); break;
      case 9: out[i] = cref_silu(a[i]); break;
      case 10: out[i] = widen(cref_bf16(a[i])); break;
    }
  }
  return 0;
}

/* ======================================================================== */
/* R1: canonical reductions, Algorithm 2 (TreeFold)                          */
/* ======================================================================== */

typedef struct {
  int n;
  int level[64];
  float val[64];
} sfold;

/* Push: merge with the top entry while it has the same level; the earlier block stays on the left. */
static void sfold_push(sfold* f, float part) {
  int level = 0;
  while (f->n > 0 && f->level[f->n - 1] == level) {
    part = cref_add(f->val[f->n - 1], part);
    f->n--;
    level++;
  }
  f->level[f->n] = level;
  f->val[f->n] = part;
  f->n++;
}

/* Result: start from the lowest-level entry (top of the stack), then add the remaining entries in
   ascending level order. */
static float sfold_result(const sfold* f) {
  if (f->n == 0) return 0.0f;
  float acc = f->val[f->n - 1];
  for (int i = f->n - 2; i >= 0; --i) acc = cref_add(f->val[i], acc);
  return acc;
}

typedef struct {
  int n;
  int level[64];
  float* val[64];
  int64_t len;
} vfold;

static void vfold_push(vfold* f, float* part) { /* takes ownership of part */
  int level = 0;
  while (f->n > 0 && f->level[f->n - 1] == level) {
    float* lower = f->val[f->n - 1];
    for (int64_t j = 0; j < f->len; ++j) part[j] = cref_add(lower[j], part[j]);
    free(lower);
    f->n--;
    level++;
  }
  f->level[f->n] = level;
  f->val[f->n] = part;
  f->n++;
}

static void vfold_result(vfold* f, float* out) { /* frees the stack */
  if (f->n == 0) {
    for (int64_t j = 0; j < f->len; ++j) out[j] = 0.0f;
    return;
  }
  float* acc = f->val[f->n - 1];
  for (int i = f->n - 2; i >= 0; --i) {
    for (int64_t j = 0; j < f->len; ++j) acc[j] = cref_add(f->val[i][j], acc[j]);
    free(f->val[i]);
  }
  memcpy(out, acc, sizeof(float) * (size_t)f->len);
  free(acc);
  f->n = 0;
}

float cref_rsum(const float* t, int64_t n, int64_t stride, int32_t chunk) {
  sfold f = {0};
  for (int64_t c0 = 0; c0 < n; c0 += chunk) {
    int64_t c1 = c0 + chunk < n ? c0 + chunk : n;
    float s = 0.0f;
    for (int64_t k = c0; k < c1; ++k) s = cref_add(s, t[k * stride]);
    sfold_push(&f, s);
  }
  return sfold_result(&f);
}

float cref_rdot_bf16(const uint16_t* a, int64_t sa, const uint16_t* b, int64_t sb, int64_t n, int32_t chunk) {
  sfold f = {0};
  for (int64_t c0 = 0; c0 < n; c0 += chunk) {
    int64_t c1 = c0 + chunk < n ? c0 + chunk : n;
    float s = 0.0f;
    for (int64_t k = c0; k < c1; ++k) s = cref_fma(widen(a[k * sa]), widen(b[k * sb]), s);
    sfold_push(&f, s);
  }
  return sfold_result(&f);
}

float cref_rdot_f32(const float* a, int64_t sa, const float* b, int64_t sb, int64_t n, int32_t chunk) {
  sfold f = {0};
  for (int64_t c0 = 0; c0 < n; c0 += chunk) {
    int64_t c1 = c0 + chunk < n ? c0 + chunk : n;
    float s = 0.0f;
    for (int64_t k = c0; k < c1; ++k) s = cref_add(s, cref_mul(a[k * sa], b[k * sb]));
    sfold_push(&f, s);
  }
  return sfold_result(&f);
}

int cref_treefold(const float* parts, int64_t nparts, int64_t len, float* out, int32_t* max_entries) {
  if (nparts < 0 || len < 0) return -1;
  vfold f = {0};
  f.len = len;
  int deepest = 0;
  for (int64_t p = 0; p < nparts; ++p) {
    if (f.n + 1 > deepest) deepest = f.n + 1;
    float* part = (float*)malloc(sizeof(float) * (size_t)(len ? len : 1));
    memcpy(part, parts + p * len, sizeof(float) * (size_t)len);
    vfold_push(&f, part);
  }
  vfold_result(&f, out);
  if (max_entries) *max_entries = deepest;
  return 0;
}

/* ======================================================================== */
/* R2: GEMM                                                                   */
/* ======================================================================== */

int cref_gemm(int32_t trans_a, int32_t trans_b, int64_t m, int64_t n, int64_t k, const uint16_t* a, int64_t lda,
              const uint16_t* b, int64_t ldb, float* c, int64_t ldc) {
  if (m < 0 || n < 0 || k < 0 || ldc < n) return -1;
  if (m == 0 || n == 0) return 0;
  /* B widened once into a dense [k][n] fp32 copy (exact) */
  float* bw = (float*)malloc(sizeof(float) * (size_t)(k ? k : 1) * (size_t)n);
  for (int64_t kk = 0; kk < k; ++kk)
    for (int64_t j = 0; j < n; ++j) bw[kk * n + j] = widen(trans_b ? b[j * ldb + kk] : b[kk * ldb + j]);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < m; ++i) {
    vfold f = {0};
    f.len = n;
    for (int64_t c0 = 0; c0 < k; c0 += CHUNK) {
      int64_t c1 = c0 + CHUNK < k ? c0 + CHUNK : k;
      float* part = (float*)calloc((size_t)n, sizeof(float)); /* chain starts at +0 */
      for (int64_t kk = c0; kk < c1; ++kk) {
        float av = widen(trans_a ? a[kk * lda + i] : a[i * lda + kk]);
        const float* brow = bw + kk * n;
        for (int64_t j = 0; j < n; ++j) part[j] = cref_fma(av, brow[j], part[j]);
      }
      vfold_push(&f, part);
    }
    vfold_result(&f, c + i * ldc);
  }
  free(bw);
  return 0;
}

/* ======================================================================== */
/* R3: RMSNorm                                                                */
/* ======================================================================== */

static float inv_of(int64_t d) { return (float)(1.0 / (double)d); } /* RN32(1/d): correctly rounded */

int cref_rownorm_fwd(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps, uint16_t* y,
                     float* rstd) {
  if (rows < 0 || cols <= 0) return -1;
  const float inv_d = inv_of(cols);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < rows; ++t) {
    const float* xr = x + t * cols;
    sfold f = {0};
    for (int64_t c0 = 0; c0 < cols; c0 += CHUNK) {
      int64_t c1 = c0 + CHUNK < cols ? c0 + CHUNK : cols;
      float s = 0.0f;
      for (int64_t k = c0; k < c1; ++k) s = cref_add(s, cref_mul(xr[k], xr[k]));
      sfold_push(&f, s);
    }
    float ss = sfold_result(&f);
    float ms = cref_mul(ss, inv_d);
    float v = cref_add(ms, eps);
    float r = cref_div(1.0f, cref_sqrt(v));
    rstd[t] = r;
    for (int64_t k = 0; k < cols; ++k) y[t * cols + k] = cref_bf16(cref_mul(cref_mul(xr[k], r), widen(gain[k])));
  }
  return 0;
}

/* R3 forward with the output kept in fp32 (the embedding norm of R16, whose output is the residual stream) */
int cref_rownorm_fwd_f32(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps, float* y,
                         float* rstd) {
  if (rows < 0 || cols <= 0) return -1;
  const float inv_d = inv_of(cols);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < rows; ++t) {
    const float* xr = x + t * cols;
    float ss = cref_rdot_f32(xr, 1, xr, 1, cols, CHUNK);
    float r = cref_div(1.0f, cref_sqrt(cref_add(cref_mul(ss, inv_d), eps)));
    rstd[t] = r;
    for (int64_t k = 0; k < cols; ++k) y[t * cols + k] = cref_mul(cref_mul(xr[k], r), widen(gain[k]));
  }
  return 0;
}

int cref_rownorm_bwd(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, const float* rstd,
                     const float* dy, float* dx, float* dgain) {
  if (rows < 0 || cols <= 0) return -1;
  const float inv_d = inv_of(cols);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < rows; ++t) {
    const float* xr = x + t * cols;
    const float* dyr = dy + t * cols;
    float r = rstd[t];
    float* gy = (float*)malloc(sizeof(float) * (size_t)cols);
    for (int64_t k = 0; k < cols; ++k) gy[k] = cref_mul(dyr[k], widen(gain[k]));
    float dot = cref_rdot_f32(gy, 1, xr, 1, cols, CHUNK);
    float q = cref_mul(cref_mul(cref_mul(r, r), r), cref_mul(dot, inv_d));
    for (int64_t k = 0; k < cols; ++k) dx[t * cols + k] = cref_sub(cref_mul(r, gy[k]), cref_mul(xr[k], q));
    free(gy);
  }
  if (dgain) {
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < cols; ++k) {
      sfold f = {0};
      for (int64_t c0 = 0; c0 < rows; c0 += CHUNK) {
        int64_t c1 = c0 + CHUNK < rows ? c0 + CHUNK : rows;
        float s = 0.0f;
        for (int64_t t = c0; t < c1; ++t) s = cref_add(s, cref_mul(dy[t * cols + k], cref_mul(x[t * cols + k], rstd[t])));
        sfold_push(&f, s);
      }
      dgain[k] = sfold_result(&f);
    }
  }
  return 0;
}

/* ======================================================================== */
/* R5: causal softmax, R6: cross-entropy                                      */
/* ======================================================================== */

/* R5 with the hybrid attention window of R16: query i sees keys j with i - window < j <= i (window 0:
   every j <= i).  Keys outside enter the row sum as +0 terms at their own positions. */
int cref_softmax_window(int64_t batch, int64_t s, const float* raw, float scale, int64_t window, uint16_t* probs) {
  if (batch < 0 || s < 0 || window < 0) return -1;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t bi = 0; bi < batch * s; ++bi) {
    int64_t i = bi % s;
    int64_t j0 = (window > 0 && i - window + 1 > 0) ? i - window + 1 : 0; /* first key seen */
    const float* row = raw + bi * s;
    uint16_t* prow = probs + bi * s;
    float* e = (float*)malloc(sizeof(float) * (size_t)(s ? s : 1));
    float m = cref_mul(row[j0], scale);
    for (int64_t j = j0 + 1; j <= i; ++j) {
      float sc = cref_mul(row[j], scale);
      if (sc > m) m = sc;
    }
    for (int64_t j = 0; j < s; ++j) e[j] = (j >= j0 && j <= i) ? cref_exp(cref_sub(cref_mul(row[j], scale), m)) : 0.0f;
    float S = cref_rsum(e, s, 1, CHUNK); /* masked keys enter as +0 terms */
    float r = cref_div(1.0f, S);
    for (int64_t j = 0; j < s; ++j) prow[j] = (j >= j0 && j <= i) ? cref_bf16(cref_mul(e[j], r)) : (uint16_t)0;
    free(e);
  }
  return 0;
}

int cref_softmax_causal(int64_t batch, int64_t s, const float* raw, float scale, uint16_t* probs) {
  return cref_softmax_window(batch, s, raw, scale, 0, probs);
}

/* R6 with the z-loss of R16 (the architecture section: weight 1e-4, in the same pass as the cross-entropy).
   z = lse, the row's log-partition; row loss RN(CE + RN(z_loss * RN(z * z))); each probability is scaled
   by RN(1 + RN(RN(2 z_loss) * z)) before the target is subtracted.  z_loss = 0 is the plain R6. */
int cref_xent_z(int64_t rows, int64_t vocab, const uint16_t* logits, const int32_t* targets, float inv_tokens,
                float z_loss, uint16_t* dlogits, float* row_loss, float* mean_loss) {
  if (rows < 0 || vocab <= 0 || !(z_loss >= 0.0f)) return -1;
  for (int64_t t = 0; t < rows; ++t)
    if (targets[t] < 0 || targets[t] >= vocab) return -1;
  const float z2 = cref_mul(2.0f, z_loss);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < rows; ++t) {
    const uint16_t* lr = logits + t * vocab;
    float* e = (float*)malloc(sizeof(float) * (size_t)vocab);
    float m = widen(lr[0]);
    for (int64_t j = 1; j < vocab; ++j) {
      float l = widen(lr[j]);
      if (l > m) m = l;
    }
    for (int64_t j = 0; j < vocab; ++j) e[j] = cref_exp(cref_sub(widen(lr[j]), m));
    float S = cref_rsum(e, vocab, 1, CHUNK);
    float lse = cref_add(m, cref_log(S));
    int32_t y = targets[t];
    float ce = cref_sub(lse, widen(lr[y]));
    float pscale = 1.0f;
    if (z_loss != 0.0f) {
      ce = cref_add(ce, cref_mul(z_loss, cref_mul(lse, lse)));
      pscale = cref_add(1.0f, cref_mul(z2, lse));
    }
    row_loss[t] = ce;
    float r = cref_div(1.0f, S);
    if (dlogits) {
      for (int64_t j = 0; j < vocab; ++j) {
        float p = cref_mul(e[j], r);
        if (z_loss != 0.0f) p = cref_mul(p, pscale);
        dlogits[t * vocab + j] = cref_bf16(cref_mul(cref_sub(p, j == y ? 1.0f : 0.0f), inv_tokens));
      }
    }
    free(e);
  }
  if (mean_loss) *mean_loss = cref_mul(cref_rsum(row_loss, rows, 1, CHUNK), inv_tokens);
  return 0;
}

int cref_xent(int64_t rows, int64_t vocab, const uint16_t* logits, const int32_t* targets, float inv_tokens,
              uint16_t* dlogits, float* row_loss, float* mean_loss) {
  return cref_xent_z(rows, vocab, logits, targets, inv_tokens, 0.0f, dlogits, row_loss, mean_loss);
}

/* ======================================================================== */
/* R7: gradient plan (Algorithm 1, averages as reciprocal multiplies)        */
/* ======================================================================== */

typedef struct {
  cref_plan p;
  float inv_accum, inv_shard, inv_rep;
  int64_t n;
  float* g_r;   /* rank accumulator */
  float* inner; /* running ascending sum over shards */
  int have_inner;
  vfold fold;   /* TreeFold over replicas */
} plan_state;

static void plan_init(plan_state* s, const cref_plan* p, int64_t n) {
  memset(s, 0, sizeof(*s));
  s->p = *p;
  s->inv_accum = inv_of(p->accum);
  s->inv_shard = inv_of(p->dp_shard);
  s->inv_rep = inv_of(p->dp_replicate);
  s->n = n;
  s->g_r = (float*)malloc(sizeof(float) * (size_t)(n ? n : 1));
  s->inner = (float*)malloc(sizeof(float) * (size_t)(n ? n : 1));
  s->fold.len = n;
}

static void plan_rank_begin(plan_state* s) {
  for (int64_t i = 0; i < s->n; ++i) s->g_r[i] = 0.0f;
}

static void plan_add_microbatch(plan_state* s, const float* grad) {
  for (int64_t i = 0; i < s->n; ++i) s->g_r[i] = cref_add(s->g_r[i], cref_mul(grad[i], s->inv_accum));
}

static void plan_rank_end(plan_state* s, int r) {
  int shard = r % s->p.dp_shard;
  if (shard == 0) {
    memcpy(s->inner, s->g_r, sizeof(float) * (size_t)s->n);
  } else {
    for (int64_t i = 0; i < s->n; ++i) s->inner[i] = cref_add(s->inner[i], s->g_r[i]);
  }
  if (shard == s->p.dp_shard - 1) {
    float* part = (float*)malloc(sizeof(float) * (size_t)(s->n ? s->n : 1));
    for (int64_t i = 0; i < s->n; ++i) part[i] = cref_mul(s->inner[i], s->inv_shard);
    vfold_push(&s->fold, part);
  }
}

static void plan_finish(plan_state* s, float* out) {
  vfold_result(&s->fold, out);
  for (int64_t i = 0; i < s->n; ++i) out[i] = cref_mul(out[i], s->inv_rep);
  free(s->g_r);
  free(s->inner);
}

static int plan_valid(const cref_plan* p) {
  return p && p->accum >= 1 && p->dp_shard >= 1 && p->dp_replicate >= 1;
}

int cref_grad_accum(const cref_plan* plan, int64_t n, const float* const* grads, float* out) {
  if (!plan_valid(plan) || n < 0) return -1;
  plan_state s;
  plan_init(&s, plan, n);
  int N = plan->dp_shard * plan->dp_replicate;
  for (int r = 0; r < N; ++r) {
    plan_rank_begin(&s);
    for (int k = 0; k < plan->accum; ++k) plan_add_microbatch(&s, grads[r * plan->accum + k]);
    plan_rank_end(&s, r);
  }
  plan_finish(&s, out);
  return 0;
}

/* ======================================================================== */
/* R9: AdamW                                                                  */
/* ======================================================================== */

static void adamw_tensor(int64_t n, uint16_t* p16, float* m, float* v, const float* g, int decay,
                         const cref_adamw_consts* k) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    float p = widen(p16[i]);
    if (decay) p = cref_mul(p, k->decay_factor);
    float gi = g[i];
    float mi = cref_add(cref_mul(k->beta1, m[i]), cref_mul(k->one_minus_beta1, gi));
    float vi = cref_add(cref_mul(k->beta2, v[i]), cref_mul(k->one_minus_beta2, cref_mul(gi, gi)));
    float mh = cref_mul(mi, k->inv_bc1);
    float vh = cref_mul(vi, k->inv_bc2);
    float u = cref_div(mh, cref_add(cref_sqrt(vh), k->eps));
    p = cref_sub(p, cref_mul(k->lr, u));
    m[i] = mi;
    v[i] = vi;
    p16[i] = cref_bf16(p);
  }
}

int cref_adamw(int64_t n_tensors, const int64_t* sizes, uint16_t* const* params, float* const* m, float* const* v,
               const float* const* grads, const uint8_t* decay_mask, const cref_adamw_consts* k) {
  if (n_tensors < 0 || !k) return -1;
  for (int64_t t = 0; t < n_tensors; ++t) {
    if (sizes[t] < 0) return -1;
    adamw_tensor(sizes[t], params[t], m[t], v[t], grads[t], decay_mask[t] != 0, k);
  }
  return 0;
}

/* ======================================================================== */
/* R15: global gradient norm, clip and spike skip                             */
/* ======================================================================== */

/* The global l2 norm of the gradient (training-setup paragraph on the optimizer: clipping to a global
   norm of 1.0).  The gradient tensors, laid end to end in the declared tensor order, form one vector;
   its sum of squares is an R1 reduction over that vector's index (terms RN(g*g), chunks of 32 that may
   run across a tensor boundary, chunk partials folded by Algorithm 2), and the norm is its correctly
   rounded square root. */
float cref_global_norm(int64_t n_tensors, const int64_t* sizes, const float* const* grads) {
  sfold f = {0};
  float s = 0.0f;
  int in_chunk = 0;
  for (int64_t t = 0; t < n_tensors; ++t)
    for (int64_t i = 0; i < sizes[t]; ++i) {
      const float g = grads[t][i];
      s = cref_add(s, cref_mul(g, g));
      if (++in_chunk == CHUNK) {
        sfold_push(&f, s);
        s = 0.0f;
        in_chunk = 0;
      }
    }
  if (in_chunk) sfold_push(&f, s);
  return cref_sqrt(sfold_result(&f));
}

/* Clip coefficient and spike decision for one step (the optimizer paragraph's clip at 1.0; the section
   on gradient behaviour: a pre-clip norm above 5 skips five optimizer steps).
   coef = CRdiv(max_norm, RN(norm + RN32(1e-6))); the gradient is scaled by coef when coef < 1.
   A spike is a norm that is not <= spike_norm (NaN included); it sets the counter of updates still to
   skip to skip_steps, so that the spiking step and the skip_steps - 1 after it apply no update; a spike
   inside that window starts it again.  skip_steps = 0 turns the spike rule off. */
int cref_clip_decide(float norm, const cref_clip_cfg* k, int32_t* skip_state, float* coef, int32_t* skipped) {
  if (!k || !(k->max_norm > 0.0f) || k->skip_steps < 0 || (k->skip_steps > 0 && !skip_state)) return -1;
  *coef = cref_div(k->max_norm, cref_add(norm, 1e-6f));
  int32_t left = skip_state ? *skip_state : 0;
  if (k->skip_steps > 0 && !(norm <= k->spike_norm)) left = k->skip_steps;
  const int32_t skip = left > 0;
  if (skip) left -= 1;
  if (skip_state) *skip_state = left;
  *skipped = skip;
  return 0;
}

/* g <- RN(g * coef) for every element when coef < 1; otherwise the gradient is left as it is. */
int cref_clip_apply(int64_t n_tensors, const int64_t* sizes, float* const* grads, float coef) {
  if (n_tensors < 0) return -1;
  if (!(coef < 1.0f)) return 0;
  for (int64_t t = 0; t < n_tensors; ++t)
    for (int64_t i = 0; i < sizes[t]; ++i) grads[t][i] = cref_mul(grads[t][i], coef);
  return 0;
}

/* ======================================================================== */
/* Elementwise pieces of the decoder                                          */
/* ======================================================================== */

/* R8: half-split rotation of one head vector v[0..hd) at position s; output bf16. */
static void rope_fwd(const float* v, int hd, const float* cs, const float* sn, uint16_t* out) {
  int h = hd / 2;
  for (int i = 0; i < h; ++i) {
    float x1 = v[i], x2 = v[i + h];
    out[i] = cref_bf16(cref_sub(cref_mul(x1, cs[i]), cref_mul(x2, sn[i])));
    out[i + h] = cref_bf16(cref_add(cref_mul(x2, cs[i]), cref_mul(x1, sn[i])));
  }
}

/* transposed rotation of a gradient */
static void rope_bwd(const float* g, int hd, const float* cs, const float* sn, float* out) {
  int h = hd / 2;
  for (int i = 0; i < h; ++i) {
    float g1 = g[i], g2 = g[i + h];
    out[i] = cref_add(cref_mul(g1, cs[i]), cref_mul(g2, sn[i]));
    out[i + h] = cref_sub(cref_mul(g2, cs[i]), cref_mul(g1, sn[i]));
  }
}

/* ======================================================================== */
/* Decoder block                                                              */
/* ======================================================================== */

typedef struct {
  int64_t T, B, S, d, H, Hkv, hd, F, N; /* N = (H + 2 Hkv) hd: width of the fused q, k, v projection */
  int64_t window;                        /* 0: full causal; W: query i sees keys i - W + 1 .. i */
  int qk_norm;
  int pv_int8, dq_bits;                  /* R17 P.V, R18 dQ (0: off) */
  int int8;                              /* R19: the four projections in int8 */
  float sx[4];                           /* R19 activation steps (qkv, o, gate_up, down) */
  int8_t* qx[4];                         /* R19 activation codes [T][K] */
  int8_t* qw[4];                         /* R19 weight codes [N][K] */
  float* sw[4];                          /* R19 re-pinned weight steps [N] */
  float eps;
  float* x;      /* [T][d] input (residual) */
  uint16_t* xn;  /* [T][d] */
  float* rstd1;  /* [T] */
  float* qkv;    /* [T][N] projection output (kept for the QK-norm backward) */
  float* rq;     /* [T][H + Hkv]: QK-norm r of each q and k head row */
  uint16_t *q, *k, *v; /* q [B][H][S][hd], k and v [B][Hkv][S][hd] bf16, q and k after rotation */
  uint16_t* P;   /* [B][H][S][S] */
  uint16_t* O;   /* [T][d] */
  float* h;      /* [T][d] */
  uint16_t* hn;  /* [T][d] */
  float* rstd2;  /* [T] */
  float* gu;     /* [T][2F] */
  uint16_t* a;   /* [T][F] */
} block_saved;

static void* xmalloc(size_t n) {
  void* p = malloc(n ? n : 1);
  return p;
}

static int64_t kv_heads(const cref_model_cfg* c) { return c->n_kv_heads > 0 ? c->n_kv_heads : c->n_heads; }

static void block_saved_alloc(block_saved* s, const cref_model_cfg* c, int64_t B, int64_t window) {
  s->B = B; s->S = c->seq; s->T = B * c->seq; s->d = c->d_model; s->H = c->n_heads; s->Hkv = kv_heads(c);
  s->hd = c->head_dim; s->F = c->d_ffn; s->N = (s->H + 2 * s->Hkv) * s->hd;
  s->window = window; s->qk_norm = c->qk_norm; s->eps = c->rms_eps;
  s->pv_int8 = c->pv_int8; s->dq_bits = c->dq_fixed_bits;
  s->int8 = c->int8_linear;
  for (int i = 0; i < 4; ++i) { s->qx[i] = NULL; s->qw[i] = NULL; s->sw[i] = NULL; s->sx[i] = 0.0f; }
  const int64_t T = s->T, d = s->d, S = s->S, F = s->F, kvw = s->Hkv * s->hd;
  s->x = (float*)xmalloc(sizeof(float) * T * d);
  s->xn = (uint16_t*)xmalloc(2 * T * d);
  s->rstd1 = (float*)xmalloc(sizeof(float) * T);
  s->qkv = (float*)xmalloc(sizeof(float) * T * s->N);
  s->rq = (float*)xmalloc(sizeof(float) * T * (s->H + s->Hkv));
  s->q = (uint16_t*)xmalloc(2 * T * d);
  s->k = (uint16_t*)xmalloc(2 * T * kvw);
  s->v = (uint16_t*)xmalloc(2 * T * kvw);
  s->P = (uint16_t*)xmalloc(2 * B * s->H * S * S);
  s->O = (uint16_t*)xmalloc(2 * T * d);
  s->h = (float*)xmalloc(sizeof(float) * T * d);
  s->hn = (uint16_t*)xmalloc(2 * T * d);
  s->rstd2 = (float*)xmalloc(sizeof(float) * T);
  s->gu = (float*)xmalloc(sizeof(float) * T * 2 * F);
  s->a = (uint16_t*)xmalloc(2 * T * F);
}

static void block_saved_free(block_saved* s) {
  for (int i = 0; i < 4; ++i) { free(s->qx[i]); free(s->qw[i]); free(s->sw[i]); }
  free(s->x); free(s->xn); free(s->rstd1); free(s->qkv); free(s->rq); free(s->q); free(s->k); free(s->v);
  free(s->P); free(s->O); free(s->h); free(s->hn); free(s->rstd2); free(s->gu); free(s->a);
}

static const uint32_t ATTN_SCALE_128 = 0x3DB504F3u; /* RN32(1/sqrt(128)) */

/* Sign of (P 2^Q - 1/sqrt(n)) for an odd P < 2^27 and 1 <= n < 2^60: the sign of P^2 n - 2^(-2Q), exact in
   128-bit integers (every boundary used below has Q <= -24 and -2Q < 120). */
static int cmp_inv_sqrt(uint64_t P, int Q, uint64_t n) {
  unsigned __int128 lhs = (unsigned __int128)P * P * n;
  unsigned __int128 rhs = (unsigned __int128)1 << (-2 * Q);
  return lhs < rhs ? -1 : (lhs > rhs ? 1 : 0);
}

/* RN32(1/sqrt(n)) for an integer 1 <= n < 2^60, decided exactly.  A binary64 estimate gives a candidate y;
   y is the correctly rounded value iff 1/sqrt(n) lies strictly between the midpoints to its neighbours
   (1/sqrt(n) is never a midpoint: that would make n the square of a power of two over an odd square).
   Used for the attention scale RN32(1/sqrt(head_dim)) and LSQ's gradient scale RN32(1/sqrt(127 K)). */
float cref_inv_sqrt_int(int64_t n) {
  if (n < 1 || n >= ((int64_t)1 << 60)) return NAN;
  float y = (float)(1.0 / sqrt((double)n));
  for (int it = 0; it < 8; ++it) {
    int e;
    const float fr = frexpf(y, &e); /* y = fr 2^e, fr in [1/2, 1) */
    const uint64_t m = (uint64_t)ldexpf(fr, 24);
    e -= 24; /* y = m 2^e with 2^23 <= m < 2^24 */
    if (cmp_inv_sqrt(2 * m + 1, e - 1, (uint64_t)n) < 0) { y = nextafterf(y, INFINITY); continue; }
    const int pow2 = (m == ((uint64_t)1 << 23));
    if (cmp_inv_sqrt(pow2 ? 4 * m - 1 : 2 * m - 1, pow2 ? e - 2 : e - 1, (uint64_t)n) > 0) {
      y = nextafterf(y, 0.0f);
      continue;
    }
    return y;
  }
  return NAN; /* not reached: the binary64 estimate is within one unit of the answer */
}

static float attn_scale(int64_t hd) {
  if (hd == 128) return f_from_bits(ATTN_SCALE_128);
  return cref_inv_sqrt_int(hd);
}

/* SwiGLU forward of one element: a = bf16(RN(silu(g) u)) */
static uint16_t swiglu_fwd1(float g, float u) { return cref_bf16(cref_mul(cref_silu(g), u)); }

/* SwiGLU backward of one element from the fp32 gradient da of a: du = RN(da silu(g)) and
   dg = RN(RN(da u) dsg) with dsg = RN(sig RN(1 + RN(g RN(1 - sig)))), sig = sigmoid(g); both to bf16 */
static void swiglu_bwd1(float g, float u, float da, uint16_t* dg, uint16_t* du) {
  const float sig = cref_sigmoid(g);
  const float silu = cref_mul(g, sig);
  const float dsg = cref_mul(sig, cref_add(1.0f, cref_mul(g, cref_sub(1.0f, sig))));
  *du = cref_bf16(cref_mul(da, silu));
  *dg = cref_bf16(cref_mul(cref_mul(da, u), dsg));
}

int cref_swiglu(int64_t n, const float* g, const float* u, const float* da, uint16_t* a, uint16_t* dg,
                uint16_t* du) {
  if (n < 0 || (n > 0 && (!g || !u))) return -1;
  for (int64_t i = 0; i < n; ++i) {
    if (a) a[i] = swiglu_fwd1(g[i], u[i]);
    if (da && dg && du) swiglu_bwd1(g[i], u[i], da[i], &dg[i], &du[i]);
  }
  return 0;
}

/* R16 gain-free QK-norm of one head row (the architecture section: RMSNorm per head before RoPE, no
   gain): r as in R3, the normalised row kept in fp32 for the rotation. */
static float headnorm_r(const float* x, int64_t n, float eps) {
  const float ss = cref_rdot_f32(x, 1, x, 1, n, CHUNK);
  const float ms = cref_mul(ss, inv_of(n));
  return cref_div(1.0f, cref_sqrt(cref_add(ms, eps)));
}

/* R3's input gradient with the gain left out: gy is the gradient of the normalised row. */
static void headnorm_bwd(const float* x, float r, const float* gy, int64_t n, float* dx) {
  const float dot = cref_rdot_f32(gy, 1, x, 1, n, CHUNK);
  const float q = cref_mul(cref_mul(cref_mul(r, r), r), cref_mul(dot, inv_of(n)));
  for (int64_t k = 0; k < n; ++k) dx[k] = cref_sub(cref_mul(r, gy[k]), cref_mul(x[k], q));
}

/* q or k head row at projection column col0 of token t: optional QK-norm, then the rotation, bf16 out */
static void head_in(block_saved* s, int64_t t, int64_t col0, int64_t ridx, const float* rope_cos,
                    const float* rope_sin, uint16_t* out) {
  const int64_t hd = s->hd, pos = t % s->S;
  const float* x = s->qkv + t * s->N + col0;
  float* xn = (float*)xmalloc(sizeof(float) * hd);
  if (s->qk_norm) {
    const float r = headnorm_r(x, hd, s->eps);
    s->rq[t * (s->H + s->Hkv) + ridx] = r;
    for (int64_t j = 0; j < hd; ++j) xn[j] = cref_mul(x[j], r);
  } else {
    memcpy(xn, x, sizeof(float) * hd);
  }
  rope_fwd(xn, (int)hd, rope_cos + pos * (hd / 2), rope_sin + pos * (hd / 2), out);
  free(xn);
}

/* R19 forward of projection li (0 qkv, 1 o, 2 gate_up, 3 down): Y [T][N] = the int8 product of X (bf16
   [T][K]) with step s->sx[li] and W (bf16 [N][K]) with its re-pinned per-row steps; the codes and steps are
   kept for the backward. */
static void qlin_fwd(block_saved* s, int li, int64_t T, int64_t N, int64_t K, const uint16_t* X, const uint16_t* W,
                     float* Y) {
  s->sw[li] = (float*)xmalloc(sizeof(float) * N);
  s->qw[li] = (int8_t*)xmalloc((size_t)(N * K));
  s->qx[li] = (int8_t*)xmalloc((size_t)(T * K));
  cref_quant_scales(N, K, W, s->sw[li]);
  cref_quantize(N, K, 1, W, s->sw[li], 1, s->qw[li]);
  cref_quantize(T, K, 1, X, &s->sx[li], 0, s->qx[li]);
  cref_gemm_i8(T, N, K, s->qx[li], K, s->qw[li], K, NULL, Y, N, s->sx[li], s->sw[li]);
}

/* R19 backward of projection li: G16 is the bf16 gradient of its output [T][N] (the operand the canonical
   path would multiply), widened; dX [T][K] and dW [N][K] by R14; *dsx the LSQ gradient of the step. */
static void qlin_bwd(const block_saved* s, int li, int64_t T, int64_t N, int64_t K, const uint16_t* G16,
                     const uint16_t* X, float* dX, float* dW, float* dsx) {
  float* G = (float*)xmalloc(sizeof(float) * T * N);
  for (int64_t i = 0; i < T * N; ++i) G[i] = widen(G16[i]);
  cref_qlinear_bwd(T, N, K, G, s->qx[li], s->sx[li], s->qw[li], s->sw[li], dX, dW);
  free(G);
  *dsx = cref_lsq_step_grad(T, K, X, s->sx[li], dX);
}

/* forward of one block; w = {attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down}; y = block output.
   w_qkv rows: H query heads, then Hkv key heads, then Hkv value heads (hd rows each).  Query head h reads
   key/value head h / (H / Hkv). */
static void block_fwd(block_saved* s, const float* x, const uint16_t* const* w, const float* rope_cos,
                      const float* rope_sin, float* y) {
  const int64_t T = s->T, B = s->B, S = s->S, d = s->d, H = s->H, Hkv = s->Hkv, hd = s->hd, F = s->F, N = s->N;
  const int64_t G = H / Hkv;
  memcpy(s->x, x, sizeof(float) * T * d);
  cref_rownorm_fwd(T, d, x, w[0], s->eps, s->xn, s->rstd1);
  if (s->int8) for (int i = 0; i < 4; ++i) s->sx[i] = widen(w[6 + i][0]);
  if (s->int8) qlin_fwd(s, 0, T, N, d, s->xn, w[1], s->qkv);
  else cref_gemm(0, 1, T, N, d, s->xn, d, w[1], d, s->qkv, N);
  for (int64_t t = 0; t < T; ++t) {
    const int64_t b = t / S, pos = t % S;
    for (int64_t hh = 0; hh < H; ++hh) head_in(s, t, hh * hd, hh, rope_cos, rope_sin, s->q + ((b * H + hh) * S + pos) * hd);
    for (int64_t g = 0; g < Hkv; ++g) {
      const int64_t o = ((b * Hkv + g) * S + pos) * hd;
      head_in(s, t, (H + g) * hd, H + g, rope_cos, rope_sin, s->k + o);
      for (int64_t j = 0; j < hd; ++j) s->v[o + j] = cref_bf16(s->qkv[t * N + (H + Hkv + g) * hd + j]);
    }
  }
  float* raw = (float*)xmalloc(sizeof(float) * S * S);
  float* ob = (float*)xmalloc(sizeof(float) * S * hd);
  const float c = attn_scale(hd);
  for (int64_t bh = 0; bh < B * H; ++bh) {
    int64_t b = bh / H, hh = bh % H, g = hh / G;
    const uint16_t* Q = s->q + bh * S * hd;
    const uint16_t* K = s->k + (b * Hkv + g) * S * hd;
    const uint16_t* V = s->v + (b * Hkv + g) * S * hd;
    uint16_t* P = s->P + bh * S * S;
    cref_gemm(0, 1, S, S, hd, Q, hd, K, hd, raw, S);
    cref_softmax_window(1, S, raw, c, s->window, P);
    if (s->pv_int8) cref_attn_pv_i8(S, hd, P, V, ob);          /* R17 */
    else cref_gemm(0, 0, S, hd, S, P, S, V, hd, ob, hd);
    for (int64_t pos = 0; pos < S; ++pos)
      for (int64_t j = 0; j < hd; ++j) s->O[(b * S + pos) * d + hh * hd + j] = cref_bf16(ob[pos * hd + j]);
  }
  free(raw);
  free(ob);
  float* attn = (float*)xmalloc(sizeof(float) * T * d);
  if (s->int8) qlin_fwd(s, 1, T, d, d, s->O, w[2], attn);
  else cref_gemm(0, 1, T, d, d, s->O, d, w[2], d, attn, d);
  for (int64_t i = 0; i < T * d; ++i) s->h[i] = cref_add(x[i], attn[i]);
  free(attn);
  cref_rownorm_fwd(T, d, s->h, w[3], s->eps, s->hn, s->rstd2);
  if (s->int8) qlin_fwd(s, 2, T, 2 * F, d, s->hn, w[4], s->gu);
  else cref_gemm(0, 1, T, 2 * F, d, s->hn, d, w[4], d, s->gu, 2 * F);
  for (int64_t t = 0; t < T; ++t)
    for (int64_t j = 0; j < F; ++j) s->a[t * F + j] = swiglu_fwd1(s->gu[t * 2 * F + j], s->gu[t * 2 * F + F + j]);
  float* ffn = (float*)xmalloc(sizeof(float) * T * d);
  if (s->int8) qlin_fwd(s, 3, T, d, F, s->a, w[5], ffn);
  else cref_gemm(0, 1, T, d, F, s->a, F, w[5], F, ffn, d);
  for (int64_t i = 0; i < T * d; ++i) y[i] = cref_add(s->h[i], ffn[i]);
  free(ffn);
}

static uint16_t* to_bf16(const float* x, int64_t n) {
  uint16_t* o = (uint16_t*)xmalloc(2 * n);
  for (int64_t i = 0; i < n; ++i) o[i] = cref_bf16(x[i]);
  return o;
}

/* gradient of a rotated (and, with QK-norm, normalised) head row back to the projection output, bf16 */
static void head_out(const block_saved* s, int64_t t, int64_t col0, int64_t ridx, const float* g,
                     const float* rope_cos, const float* rope_sin, uint16_t* dqkv) {
  const int64_t hd = s->hd, pos = t % s->S;
  float* gn = (float*)xmalloc(sizeof(float) * hd);
  rope_bwd(g, (int)hd, rope_cos + pos * (hd / 2), rope_sin + pos * (hd / 2), gn);
  if (s->qk_norm) {
    float* gx = (float*)xmalloc(sizeof(float) * hd);
    headnorm_bwd(s->qkv + t * s->N + col0, s->rq[t * (s->H + s->Hkv) + ridx], gn, hd, gx);
    for (int64_t j = 0; j < hd; ++j) dqkv[t * s->N + col0 + j] = cref_bf16(gx[j]);
    free(gx);
  } else {
    for (int64_t j = 0; j < hd; ++j) dqkv[t * s->N + col0 + j] = cref_bf16(gn[j]);
  }
  free(gn);
}

/* backward of one block: dy = gradient of the block output; dx = gradient of the block input;
   dw = the six fp32 weight gradients.  With grouped heads, the gradient of a shared key (value) head is
   one contraction over every (query head of its group, query) pair, heads in ascending order and queries
   ascending within each (R16). */
static void block_bwd(const block_saved* s, const float* dy, const uint16_t* const* w, const float* rope_cos,
                      const float* rope_sin, float* dx, float* const* dw) {
  const int64_t T = s->T, B = s->B, S = s->S, d = s->d, H = s->H, Hkv = s->Hkv, hd = s->hd, F = s->F, N = s->N;
  const int64_t G = H / Hkv, W = s->window;
  /* MLP */
  uint16_t* dyb = to_bf16(dy, T * d);
  float* da = (float*)xmalloc(sizeof(float) * T * F);
  if (s->int8) {
    qlin_bwd(s, 3, T, d, F, dyb, s->a, da, dw[5], dw[9]);
  } else {
    cref_gemm(1, 0, d, F, T, dyb, d, s->a, F, dw[5], F);          /* dW_down = dy^T a */
    cref_gemm(0, 0, T, F, d, dyb, d, w[5], F, da, F);             /* da = dy W_down */
  }
  free(dyb);
  uint16_t* dgu = (uint16_t*)xmalloc(2 * T * 2 * F);
  for (int64_t t = 0; t < T; ++t) {
    for (int64_t j = 0; j < F; ++j) {
      swiglu_bwd1(s->gu[t * 2 * F + j], s->gu[t * 2 * F + F + j], da[t * F + j], &dgu[t * 2 * F + j],
                  &dgu[t * 2 * F + F + j]);
    }
  }
  free(da);
  float* dhn = (float*)xmalloc(sizeof(float) * T * d);
  if (s->int8) {
    qlin_bwd(s, 2, T, 2 * F, d, dgu, s->hn, dhn, dw[4], dw[8]);
  } else {
    cref_gemm(1, 0, 2 * F, d, T, dgu, 2 * F, s->hn, d, dw[4], d); /* dW_gate_up = dgu^T hn */
    cref_gemm(0, 0, T, d, 2 * F, dgu, 2 * F, w[4], d, dhn, d);    /* dhn = dgu W_gate_up */
  }
  free(dgu);
  float* dhnorm = (float*)xmalloc(sizeof(float) * T * d);
  cref_rownorm_bwd(T, d, s->h, w[3], s->rstd2, dhn, dhnorm, dw[3]);
  free(dhn);
  float* dh = (float*)xmalloc(sizeof(float) * T * d);
  for (int64_t i = 0; i < T * d; ++i) dh[i] = cref_add(dy[i], dhnorm[i]);
  free(dhnorm);
  /* attention output projection */
  uint16_t* dhb = to_bf16(dh, T * d);
  float* dO = (float*)xmalloc(sizeof(float) * T * d);
  if (s->int8) {
    qlin_bwd(s, 1, T, d, d, dhb, s->O, dO, dw[2], dw[7]);
  } else {
    cref_gemm(1, 0, d, d, T, dhb, d, s->O, d, dw[2], d);          /* dW_o = dh^T O */
    cref_gemm(0, 0, T, d, d, dhb, d, w[2], d, dO, d);             /* dO = dh W_o */
  }
  free(dhb);
  /* attention core, per (batch, key/value head group) */
  const float c = attn_scale(hd);
  uint16_t* dqkv = (uint16_t*)xmalloc(2 * T * N);
  uint16_t* dOs = (uint16_t*)xmalloc(2 * G * S * hd);  /* the group's dO, head after head */
  uint16_t* Qs = (uint16_t*)xmalloc(2 * G * S * hd);   /* the group's Q, head after head */
  uint16_t* Ps = (uint16_t*)xmalloc(2 * G * S * S);    /* the group's P, head after head */
  uint16_t* dSs = (uint16_t*)xmalloc(2 * G * S * S);   /* the group's dS, head after head */
  uint16_t* Ob = (uint16_t*)xmalloc(2 * S * hd);
  float* D = (float*)xmalloc(sizeof(float) * S);
  float* dP = (float*)xmalloc(sizeof(float) * S * S);
  float* gq = (float*)xmalloc(sizeof(float) * S * hd);
  float* gk = (float*)xmalloc(sizeof(float) * S * hd);
  float* gv = (float*)xmalloc(sizeof(float) * S * hd);
  for (int64_t b = 0; b < B; ++b) {
    for (int64_t g = 0; g < Hkv; ++g) {
      const uint16_t* K = s->k + (b * Hkv + g) * S * hd;
      const uint16_t* V = s->v + (b * Hkv + g) * S * hd;
      for (int64_t e = 0; e < G; ++e) {
        const int64_t hh = g * G + e, bh = b * H + hh;
        uint16_t* dOb = dOs + e * S * hd;
        uint16_t* dS = dSs + e * S * S;
        memcpy(Qs + e * S * hd, s->q + bh * S * hd, 2 * S * hd);
        memcpy(Ps + e * S * S, s->P + bh * S * S, 2 * S * S);
        const uint16_t* P = s->P + bh * S * S;
        for (int64_t pos = 0; pos < S; ++pos)
          for (int64_t j = 0; j < hd; ++j) {
            dOb[pos * hd + j] = cref_bf16(dO[(b * S + pos) * d + hh * hd + j]);
            Ob[pos * hd + j] = s->O[(b * S + pos) * d + hh * hd + j];
          }
        for (int64_t i = 0; i < S; ++i) D[i] = cref_rdot_bf16(dOb + i * hd, 1, Ob + i * hd, 1, hd, CHUNK);
        cref_gemm(0, 1, S, S, hd, dOb, hd, V, hd, dP, S);           /* dP = dO V^T */
        for (int64_t i = 0; i < S; ++i)
          for (int64_t j = 0; j < S; ++j) {
            const int seen = j <= i && (W == 0 || j > i - W);
            dS[i * S + j] = seen ? cref_bf16(cref_mul(cref_mul(widen(P[i * S + j]), cref_sub(dP[i * S + j], D[i])), c))
                                 : (uint16_t)0;
          }
        if (s->dq_bits) cref_attn_dq_fixed(S, hd, W, s->dq_bits, dS, K, gq); /* dQ = dS K by R18 */
        else cref_gemm(0, 0, S, hd, S, dS, S, K, hd, gq, hd);       /* dQ = dS K */
        for (int64_t pos = 0; pos < S; ++pos)
          head_out(s, b * S + pos, hh * hd, hh, gq + pos * hd, rope_cos, rope_sin, dqkv);
      }
      cref_gemm(1, 0, S, hd, G * S, dSs, S, Qs, hd, gk, hd);       /* dK = sum over the group of dS^T Q */
      cref_gemm(1, 0, S, hd, G * S, Ps, S, dOs, hd, gv, hd);       /* dV = sum over the group of P^T dO */
      for (int64_t pos = 0; pos < S; ++pos) {
        const int64_t t = b * S + pos;
        head_out(s, t, (H + g) * hd, H + g, gk + pos * hd, rope_cos, rope_sin, dqkv);
        for (int64_t j = 0; j < hd; ++j) dqkv[t * N + (H + Hkv + g) * hd + j] = cref_bf16(gv[pos * hd + j]);
      }
    }
  }
  free(dOs); free(Qs); free(Ps); free(dSs); free(Ob); free(D); free(dP); free(gq); free(gk); free(gv); free(dO);
  float* dxn = (float*)xmalloc(sizeof(float) * T * d);
  if (s->int8) {
    qlin_bwd(s, 0, T, N, d, dqkv, s->xn, dxn, dw[1], dw[6]);
  } else {
    cref_gemm(1, 0, N, d, T, dqkv, N, s->xn, d, dw[1], d);        /* dW_qkv = dqkv^T xn */
    cref_gemm(0, 0, T, d, N, dqkv, N, w[1], d, dxn, d);           /* dxn = dqkv W_qkv */
  }
  free(dqkv);
  float* dxnorm = (float*)xmalloc(sizeof(float) * T * d);
  cref_rownorm_bwd(T, d, s->x, w[0], s->rstd1, dxn, dxnorm, dw[0]);
  free(dxn);
  for (int64_t i = 0; i < T * d; ++i) dx[i] = cref_add(dh[i], dxnorm[i]);
  free(dxnorm);
  free(dh);
}

static int cfg_valid(const cref_model_cfg* c) {
  if (!c || c->n_layers < 1 || c->d_model <= 0 || c->n_heads <= 0 || c->head_dim <= 0 ||
      c->n_heads * c->head_dim != c->d_model || (c->head_dim % 2) != 0 || c->d_ffn <= 0 || c->vocab <= 0 ||
      c->seq <= 0 || c->micro_seqs <= 0)
    return 0;
  if (c->n_kv_heads < 0 || (c->n_kv_heads > 0 && c->n_heads % c->n_kv_heads != 0)) return 0;
  if ((c->qk_norm != 0 && c->qk_norm != 1) || (c->embed_norm != 0 && c->embed_norm != 1)) return 0;
  if (c->swa_window < 0 || c->swa_full_every < 0) return 0;
  if (!(c->z_loss >= 0.0f) || isinf(c->z_loss)) return 0;
  if ((c->pv_int8 != 0 && c->pv_int8 != 1) || c->dq_fixed_bits < 0 || c->dq_fixed_bits > 62) return 0;
  if (c->int8_linear != 0 && c->int8_linear != 1) return 0;
  return 1;
}

/* R16 hybrid attention: layer l (0-based) of L is windowed unless it is one of every swa_full_every-th
   layers (l + 1 a multiple of it) or the last layer. */
static int64_t layer_window(const cref_model_cfg* c, int64_t l) {
  if (c->swa_window == 0) return 0;
  if ((c->swa_full_every > 0 && (l + 1) % c->swa_full_every == 0) || l == c->n_layers - 1) return 0;
  return c->swa_window;
}

int cref_block_fwd_bwd(const cref_model_cfg* cfg, int32_t batch, const float* x, const float* dy,
                       const uint16_t* const* w, const float* rope_cos, const float* rope_sin, float* y, float* dx,
                       float* const* dw) {
  if (!cfg_valid(cfg) || batch <= 0) return -1;
  block_saved s;
  block_saved_alloc(&s, cfg, batch, cfg->swa_window);
  block_fwd(&s, x, w, rope_cos, rope_sin, y);
  block_bwd(&s, dy, w, rope_cos, rope_sin, dx, dw);
  block_saved_free(&s);
  return 0;
}

/* ======================================================================== */
/* Full step: forward + backward per microbatch, Algorithm 1, AdamW          */
/* ======================================================================== */

static int64_t per_layer(const cref_model_cfg* c) { return c->int8_linear ? 10 : 6; } /* tensors per layer */
static int64_t n_tensors_of(const cref_model_cfg* c) {
  return 3 + per_layer(c) * (int64_t)c->n_layers + (c->embed_norm ? 1 : 0);
}
static int64_t layer0_of(const cref_model_cfg* c) { return 1 + (c->embed_norm ? 1 : 0); } /* first layer tensor */

/* tensor sizes in the declared order: embed, [embed_norm], per layer attn_norm, w_qkv, w_o, ffn_norm,
   w_gate_up, w_down [, sx_qkv, sx_o, sx_gate_up, sx_down], then final_norm, head */
static void tensor_sizes(const cref_model_cfg* c, int64_t* sz, uint8_t* decay) {
  int64_t d = c->d_model, F = c->d_ffn, V = c->vocab;
  int64_t N = (c->n_heads + 2 * kv_heads(c)) * (int64_t)c->head_dim;
  int i = 0;
  sz[i] = V * d; decay[i++] = 0;                     /* embed */
  if (c->embed_norm) { sz[i] = d; decay[i++] = 0; }  /* embed_norm gain */
  for (int l = 0; l < c->n_layers; ++l) {
    sz[i] = d; decay[i++] = 0;                       /* attn_norm */
    sz[i] = N * d; decay[i++] = 1;                   /* w_qkv */
    sz[i] = d * d; decay[i++] = 1;                   /* w_o */
    sz[i] = d; decay[i++] = 0;                       /* ffn_norm */
    sz[i] = 2 * F * d; decay[i++] = 1;               /* w_gate_up */
    sz[i] = d * F; decay[i++] = 1;                   /* w_down */
    if (c->int8_linear)
      for (int q = 0; q < 4; ++q) { sz[i] = 1; decay[i++] = 0; } /* R19 activation steps */
  }
  sz[i] = d; decay[i++] = 0;                         /* final_norm */
  sz[i] = V * d; decay[i++] = 1;                     /* head */
}

/* R11 (the model section's list of bitwise-reproducible operators names the embedding backward):
   dE[v] = R1 sum over the ascending positions t with tok[t] == v of dx[t] (plain terms: chains of 32 from +0,
   then Algorithm 2 over the chain partials).  A vocabulary row that never occurs is +0; a token outside
   [0, V) contributes nothing. */
int cref_embed_bwd(int64_t T, int64_t V, int64_t d, const int32_t* tok, const float* dx, float* dE) {
  if (T < 0 || V <= 0 || d <= 0 || (T > 0 && (!tok || !dx)) || !dE) return -1;
  int64_t* cnt = (int64_t*)calloc((size_t)V + 1, sizeof(int64_t));
  for (int64_t t = 0; t < T; ++t)
    if (tok[t] >= 0 && tok[t] < V) cnt[tok[t] + 1]++;
  for (int64_t v = 0; v < V; ++v) cnt[v + 1] += cnt[v];
  int64_t* pos = (int64_t*)xmalloc(sizeof(int64_t) * (T > 0 ? T : 1));
  int64_t* fill = (int64_t*)xmalloc(sizeof(int64_t) * V);
  memcpy(fill, cnt, sizeof(int64_t) * V);
  for (int64_t t = 0; t < T; ++t) /* ascending t within each vocabulary row */
    if (tok[t] >= 0 && tok[t] < V) pos[fill[tok[t]]++] = t;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t v = 0; v < V; ++v) {
    int64_t n = cnt[v + 1] - cnt[v];
    for (int64_t j = 0; j < d; ++j) {
      sfold f = {0};
      for (int64_t c0 = 0; c0 < n; c0 += CHUNK) {
        int64_t c1 = c0 + CHUNK < n ? c0 + CHUNK : n;
        float s = 0.0f;
        for (int64_t q = c0; q < c1; ++q) s = cref_add(s, dx[pos[cnt[v] + q] * d + j]);
        sfold_push(&f, s);
      }
      dE[v * d + j] = sfold_result(&f);
    }
  }
  free(cnt); free(pos); free(fill);
  return 0;
}

/* Progress lines on stderr for long oracle runs (set CANON_REF_PROGRESS=1); no effect on any result. */
static void progress(const char* what, int64_t a, int64_t b) {
  static int on = -1;
  if (on < 0) {
    const char* e = getenv("CANON_REF_PROGRESS");
    on = (e && e[0] == '1') ? 1 : 0;
  }
  if (on) {
    fprintf(stderr, "oracle: %s %lld %lld\n", what, (long long)a, (long long)b);
    fflush(stderr);
  }
}

/* gradient of the mean loss of one microbatch; grad = flat fp32 buffer in tensor order */
static float microbatch_fwd_bwd(const cref_model_cfg* c, uint16_t* const* params, const int32_t* tok, int64_t B,
                                const float* rope_cos, const float* rope_sin, float* grad, const int64_t* off) {
  const int64_t S = c->seq, d = c->d_model, V = c->vocab, L = c->n_layers;
  const int64_t T = B * S;
  int32_t* inp = (int32_t*)xmalloc(sizeof(int32_t) * T);
  int32_t* lab = (int32_t*)xmalloc(sizeof(int32_t) * T);
  for (int64_t b = 0; b < B; ++b)
    for (int64_t s = 0; s < S; ++s) {
      inp[b * S + s] = tok[b * (S + 1) + s];
      lab[b * S + s] = tok[b * (S + 1) + s + 1];
    }
  /* embedding gather, then (R16) the embedding norm, whose fp32 output enters the first block */
  const int64_t l0 = layer0_of(c);
  float* x = (float*)xmalloc(sizeof(float) * T * d);
  for (int64_t t = 0; t < T; ++t)
    for (int64_t j = 0; j < d; ++j) x[t * d + j] = widen(params[0][(int64_t)inp[t] * d + j]);
  float* x_emb = NULL;   /* the gathered rows, kept for the embedding norm's backward */
  float* rstd_emb = NULL;
  if (c->embed_norm) {
    x_emb = x;
    rstd_emb = (float*)xmalloc(sizeof(float) * T);
    x = (float*)xmalloc(sizeof(float) * T * d);
    cref_rownorm_fwd_f32(T, d, x_emb, params[1], c->rms_eps, x, rstd_emb);
  }
  block_saved* saved = (block_saved*)xmalloc(sizeof(block_saved) * L);
  float* y = (float*)xmalloc(sizeof(float) * T * d);
  const int64_t PL = per_layer(c);
  for (int64_t l = 0; l < L; ++l) {
    const uint16_t* w[10];
    for (int i = 0; i < PL; ++i) w[i] = params[l0 + PL * l + i];
    block_saved_alloc(&saved[l], c, B, layer_window(c, l));
    block_fwd(&saved[l], x, w, rope_cos, rope_sin, y);
    progress("block forward done: layer, tokens", l, T);
    float* tmp = x; x = y; y = tmp;
  }
  /* final norm, head, loss */
  const int64_t i_fn = l0 + PL * L, i_head = i_fn + 1;
  uint16_t* xf = (uint16_t*)xmalloc(2 * T * d);
  float* rstdf = (float*)xmalloc(sizeof(float) * T);
  cref_rownorm_fwd(T, d, x, params[i_fn], c->rms_eps, xf, rstdf);
  float* logits_f = (float*)xmalloc(sizeof(float) * T * V);
  cref_gemm(0, 1, T, V, d, xf, d, params[i_head], d, logits_f, V);
  uint16_t* logits = to_bf16(logits_f, T * V);
  free(logits_f);
  uint16_t* dlogits = (uint16_t*)xmalloc(2 * T * V);
  float* row_loss = (float*)xmalloc(sizeof(float) * T);
  float loss = 0.0f;
  const float invT = inv_of(T);
  cref_xent_z(T, V, logits, lab, invT, c->z_loss, dlogits, row_loss, &loss);
  progress("head forward and cross-entropy done: tokens, vocab", T, V);
  free(logits);
  free(row_loss);
  /* backward */
  cref_gemm(1, 0, V, d, T, dlogits, V, xf, d, grad + off[i_head], d);     /* dHead = dlogits^T xf */
  float* dxf = (float*)xmalloc(sizeof(float) * T * d);
  cref_gemm(0, 0, T, d, V, dlogits, V, params[i_head], d, dxf, d);       /* dxf = dlogits Head */
  progress("head backward done: tokens, vocab", T, V);
  free(dlogits);
  free(xf);
  float* dx = (float*)xmalloc(sizeof(float) * T * d);
  cref_rownorm_bwd(T, d, x, params[i_fn], rstdf, dxf, dx, grad + off[i_fn]);
  free(dxf);
  free(rstdf);
  float* dxp = (float*)xmalloc(sizeof(float) * T * d);
  for (int64_t l = L - 1; l >= 0; --l) {
    const uint16_t* w[10];
    float* dw[10];
    for (int i = 0; i < PL; ++i) {
      w[i] = params[l0 + PL * l + i];
      dw[i] = grad + off[l0 + PL * l + i];
    }
    block_bwd(&saved[l], dx, w, rope_cos, rope_sin, dxp, dw);
    progress("block backward done: layer, tokens", l, T);
    block_saved_free(&saved[l]);
    float* tmp = dx; dx = dxp; dxp = tmp;
  }
  free(saved);
  if (c->embed_norm) {
    /* the embedding norm's backward: dx (gradient of its output) -> gradient of the gathered rows */
    cref_rownorm_bwd(T, d, x_emb, params[1], rstd_emb, dx, dxp, grad + off[1]);
    float* tmp = dx; dx = dxp; dxp = tmp;
    free(x_emb);
    free(rstd_emb);
  }
  cref_embed_bwd(T, V, d, inp, dx, grad + off[0]);
  free(dx); free(dxp); free(x); free(y); free(inp); free(lab);
  return loss;
}

int cref_step(const cref_model_cfg* c, const cref_plan* plan, uint16_t* const* params, float* const* m,
              float* const* v, const int32_t* windows, const float* rope_cos, const float* rope_sin,
              const cref_adamw_consts* k, const cref_clip_cfg* clip, float* loss_out, float* const* grads_out,
              float* norm_out, int32_t* skip_state, int32_t* skipped_out) {
  if (!cfg_valid(c) || !plan_valid(plan) || !k) return -1;
  if (clip && (!(clip->max_norm > 0.0f) || clip->skip_steps < 0 || (clip->skip_steps > 0 && !skip_state)))
    return -1;
  const int64_t nt = n_tensors_of(c);
  int64_t* sz = (int64_t*)xmalloc(sizeof(int64_t) * nt);
  uint8_t* decay = (uint8_t*)xmalloc(nt);
  tensor_sizes(c, sz, decay);
  int64_t* off = (int64_t*)xmalloc(sizeof(int64_t) * (nt + 1));
  off[0] = 0;
  for (int64_t i = 0; i < nt; ++i) off[i + 1] = off[i] + sz[i];
  const int64_t P = off[nt];
  const int64_t S1 = c->seq + 1, mb = c->micro_seqs;
  const int R = plan->dp_shard * plan->dp_replicate;
  const int64_t M = (int64_t)R * plan->accum * mb;
  for (int64_t i = 0; i < M * S1; ++i)
    if (windows[i] < 0 || windows[i] >= c->vocab) { free(sz); free(decay); free(off); return -1; }
  plan_state gs, ls;
  plan_init(&gs, plan, P);
  plan_init(&ls, plan, 1);
  float* grad = (float*)xmalloc(sizeof(float) * P);
  int32_t* tok = (int32_t*)xmalloc(sizeof(int32_t) * mb * S1);
  for (int r = 0; r < R; ++r) {           /* mesh order: r = rep * dp_shard + shard */
    plan_rank_begin(&gs);
    plan_rank_begin(&ls);
    for (int kk = 0; kk < plan->accum; ++kk) {
      /* R12: rank r owns windows m with m mod R == r, taken in ascending m, micro_seqs per microbatch */
      for (int64_t sidx = 0; sidx < mb; ++sidx) {
        int64_t mwin = r + (int64_t)R * (kk * mb + sidx);
        memcpy(tok + sidx * S1, windows + mwin * S1, sizeof(int32_t) * S1);
      }
      float loss = microbatch_fwd_bwd(c, params, tok, mb, rope_cos, rope_sin, grad, off);
      plan_add_microbatch(&gs, grad);
      plan_add_microbatch(&ls, &loss);
    }
    plan_rank_end(&gs, r);
    plan_rank_end(&ls, r);
  }
  plan_finish(&gs, grad);
  float loss = 0.0f;
  plan_finish(&ls, &loss);
  if (loss_out) *loss_out = loss;
  if (grads_out)
    for (int64_t i = 0; i < nt; ++i) memcpy(grads_out[i], grad + off[i], sizeof(float) * sz[i]);
  float** gp = (float**)xmalloc(sizeof(float*) * nt);
  for (int64_t i = 0; i < nt; ++i) gp[i] = grad + off[i];
  int32_t skipped = 0;
  if (clip) {
    /* R15: pre-clip norm of the reduced gradient, then the clip and the spike rule */
    const float norm = cref_global_norm(nt, sz, (const float* const*)gp);
    float coef;
    cref_clip_decide(norm, clip, skip_state, &coef, &skipped);
    cref_clip_apply(nt, sz, gp, coef);
    if (norm_out) *norm_out = norm;
  }
  if (skipped_out) *skipped_out = skipped;
  if (!skipped) cref_adamw(nt, sz, params, m, v, (const float* const*)gp, decay, k);
  free(gp); free(grad); free(tok); free(sz); free(decay); free(off);
  return 0;
}

/* ======================================================================== */
/* R13: int8 quantised linear (forward)                                      */
/* ======================================================================== */
/* The paper trains every attention and feed-forward projection with 8-bit weights and activations:
   per-output-channel weight step sizes re-pinned at each step to the LSQ initialisation value
   2 mean(|w|) / sqrt(q_max) (architecture section, int8 bullet; appendix on the quantisation-level
   collapse), a per-tensor activation step, exact int32 accumulation, then dequantisation.  The division
   by sqrt(q_max) is a multiply by the binary32 rounding of 1/sqrt(127). */
static const uint32_t INV_SQRT_QMAX = 0x3DB5BB09u; /* RN32(1/sqrt(127)) */

int cref_quant_scales(int64_t rows, int64_t cols, const uint16_t* w, float* scale) {
  if (rows < 0 || cols < 1 || (rows > 0 && (!w || !scale))) return -1;
  const float inv_k = inv_of(cols);
  const float c = f_from_bits(INV_SQRT_QMAX);
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    float* t = (float*)malloc(sizeof(float) * (size_t)cols);
    for (int64_t k = 0; k < cols; ++k) t[k] = fabsf(widen(w[r * cols + k]));
    const float a = cref_rsum(t, cols, 1, CHUNK);
    const float mean = cref_mul(a, inv_k);
    const float two = cref_mul(2.0f, mean);
    scale[r] = cref_mul(two, c);
    free(t);
  }
  return 0;
}

static int8_t quant1(float x, float s) {
  s = daz(s);
  if (!(s > 0.0f)) return 0;
  const float t = cref_div(x, s);
  if (isnan(t)) return 0;
  double r = rint((double)t); /* nearest integer, ties to even (default rounding mode) */
  if (r > 127.0) r = 127.0;
  if (r < -128.0) r = -128.0;
  return (int8_t)r;
}

int cref_quantize(int64_t rows, int64_t cols, int32_t dtype, const void* x, const float* scale, int32_t per_row,
                  int8_t* q) {
  if (rows < 0 || cols < 0 || (dtype != 0 && dtype != 1)) return -1;
  if (rows * cols > 0 && (!x || !scale || !q)) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const float s = scale[per_row ? r : 0];
    for (int64_t k = 0; k < cols; ++k) {
      const int64_t i = r * cols + k;
      const float v = dtype == 0 ? ((const float*)x)[i] : widen(((const uint16_t*)x)[i]);
      q[i] = quant1(v, s);
    }
  }
  return 0;
}

int cref_gemm_i8(int64_t m, int64_t n, int64_t k, const int8_t* a, int64_t lda, const int8_t* b, int64_t ldb,
                 int32_t* acc, float* y, int64_t ldc, float sa, const float* sb) {
  if (m < 0 || n < 0 || k < 0 || k > 65536 || lda < k || ldb < k || ldc < n) return -1;
  if (y && !sb) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < m; ++i)
    for (int64_t j = 0; j < n; ++j) {
      int64_t s = 0; /* exact */
      for (int64_t kk = 0; kk < k; ++kk) s += (int64_t)a[i * lda + kk] * (int64_t)b[j * ldb + kk];
      if (acc) acc[i * ldc + j] = (int32_t)s;
      if (y) y[i * ldc + j] = cref_mul(cref_mul((float)s, sa), sb[j]); /* (float) of an int: round to nearest even */
    }
  return 0;
}

/* ======================================================================== */
/* R14: int8 quantised linear, backward                                      */
/* ======================================================================== */
/* The paper's backward for the int8 linear layers passes the gradient through both quantisers unchanged
   (straight-through estimator) and runs the two gradient GEMMs in int8 after rotating the operands along
   the contraction dimension by a Walsh-Hadamard transform (training-details paragraph on int8
   computation).  Here: blocks of 256, the Sylvester matrix scaled by 1/16, evaluated as the fast transform
   with strides 1, 2, ..., 128; per-tensor absmax steps for the rotated operands. */
static const uint32_t INV_127 = 0x3C010204u; /* RN32(1/127) */

static void fwht_block(float* v) {
  for (int h = 1; h < 256; h <<= 1)
    for (int i = 0; i < 256; ++i)
      if (!(i & h)) {
        const float a = v[i], b = v[i + h];
        v[i] = cref_add(a, b);
        v[i + h] = cref_sub(a, b);
      }
  for (int i = 0; i < 256; ++i) v[i] = cref_mul(v[i], 0.0625f);
}

int cref_fwht256(int64_t n, float* v) {
  if (n < 0 || n % 256) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < n / 256; ++b) fwht_block(v + b * 256);
  return 0;
}

/* per-tensor step of a rotated operand: RN(amax * RN(1/127)); amax orders |x| by bit pattern, so a NaN is
   above every number and gives a NaN step (which quantises everything to 0) */
static float absmax_step(const float* x, int64_t n) {
  uint32_t m = 0;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t u = f_bits(daz(x[i])) & 0x7FFFFFFFu;
    if (u > m) m = u;
  }
  return cref_mul(f_from_bits(m), f_from_bits(INV_127));
}

/* rotated-and-quantised operand [rows][L] from src viewed as [rows][L] (row stride L) */
static void rot_quant(float* buf, int64_t rows, int64_t L, int8_t* q, float* step) {
  cref_fwht256(rows * L, buf);
  *step = absmax_step(buf, rows * L);
  cref_quantize(rows, L, 0, buf, step, 0, q);
}

int cref_qlinear_bwd(int64_t T, int64_t N, int64_t K, const float* dy, const int8_t* qx, float sx, const int8_t* qw,
                     const float* sw, float* dx, float* dw) {
  if (T < 1 || N < 1 || K < 1 || (dx && N % 256) || (dw && T % 256) || !dy || !qx || !qw || !sw) return -1;
  if (dx) { /* dx[t][k] = sum_n dy[t][n] W^[n][k]: contraction over N */
    float* g = (float*)xmalloc(sizeof(float) * (size_t)(T * N));
    memcpy(g, dy, sizeof(float) * (size_t)(T * N));
    float* wt = (float*)xmalloc(sizeof(float) * (size_t)(K * N)); /* W^ transposed: [K][N] */
    for (int64_t n = 0; n < N; ++n)
      for (int64_t k = 0; k < K; ++k) wt[k * N + n] = cref_mul(sw[n], (float)qw[n * K + k]);
    int8_t* qg = (int8_t*)xmalloc((size_t)(T * N));
    int8_t* qwt = (int8_t*)xmalloc((size_t)(K * N));
    float sg, swt;
    rot_quant(g, T, N, qg, &sg);
    rot_quant(wt, K, N, qwt, &swt);
    float* sb = (float*)xmalloc(sizeof(float) * (size_t)K);
    for (int64_t k = 0; k < K; ++k) sb[k] = swt;
    cref_gemm_i8(T, K, N, qg, N, qwt, N, NULL, dx, K, sg, sb);
    free(g); free(wt); free(qg); free(qwt); free(sb);
  }
  if (dw) { /* dw[n][k] = sum_t dy[t][n] X^[t][k]: contraction over T */
    float* gt = (float*)xmalloc(sizeof(float) * (size_t)(N * T)); /* dy transposed: [N][T] */
    for (int64_t t = 0; t < T; ++t)
      for (int64_t n = 0; n < N; ++n) gt[n * T + t] = dy[t * N + n];
    float* xt = (float*)xmalloc(sizeof(float) * (size_t)(K * T)); /* X^ transposed: [K][T] */
    for (int64_t t = 0; t < T; ++t)
      for (int64_t k = 0; k < K; ++k) xt[k * T + t] = cref_mul(sx, (float)qx[t * K + k]);
    int8_t* qgt = (int8_t*)xmalloc((size_t)(N * T));
    int8_t* qxt = (int8_t*)xmalloc((size_t)(K * T));
    float sgt, sxt;
    rot_quant(gt, N, T, qgt, &sgt);
    rot_quant(xt, K, T, qxt, &sxt);
    float* sb = (float*)xmalloc(sizeof(float) * (size_t)K);
    for (int64_t k = 0; k < K; ++k) sb[k] = sxt;
    cref_gemm_i8(N, K, T, qgt, T, qxt, T, NULL, dw, K, sgt, sb);
    free(gt); free(xt); free(qgt); free(qxt); free(sb);
  }
  return 0;
}

/* ======================================================================== */
/* R17: int8 P.V inside the attention forward                                */
/* ======================================================================== */
/* The paper's flash-attention forward quantises the attention weights and the values to int8 per block and
   multiplies them on the integer matrix cores, while the scores and the softmax stay in higher precision
   (training-details paragraph on int8 computation; architecture section, int8 bullet).  Here a block of P
   is 64 queries x 64 keys and a block of V is 64 keys x head_dim.  Each block's step is its absmax times
   RN(1/127) (the rule of R14's rotated operands), the codes come from R13's quantiser, the product of a P
   block and a V block is an exact integer sum, dequantised as RN(RN(RN32(acc) * sP) * sV) (left operand's
   step first, as in R13), and the per-block results are summed by R1 over the key blocks in ascending
   order. */
#define PV_BLOCK 64

/* step of a bf16 block [rows][cols] with row stride ld: RN(amax * RN(1/127)), amax by bit pattern */
static float block_absmax_step(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld) {
  uint32_t m = 0;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t c = 0; c < cols; ++c) {
      const uint32_t u = f_bits(widen(x[r * ld + c])) & 0x7FFFFFFFu;
      if (u > m) m = u;
    }
  return cref_mul(f_from_bits(m), f_from_bits(INV_127));
}

int cref_attn_pv_i8(int64_t S, int64_t hd, const uint16_t* P, const uint16_t* V, float* O) {
  if (S < 1 || hd < 1 || !P || !V || !O) return -1;
  const int64_t nb = (S + PV_BLOCK - 1) / PV_BLOCK;
  float* sv = (float*)xmalloc(sizeof(float) * (size_t)nb);
  int8_t* qv = (int8_t*)xmalloc((size_t)(S * hd));
  for (int64_t kb = 0; kb < nb; ++kb) {
    const int64_t k0 = kb * PV_BLOCK, nk = (S - k0) < PV_BLOCK ? (S - k0) : PV_BLOCK;
    sv[kb] = block_absmax_step(V + k0 * hd, nk, hd, hd);
    for (int64_t j = k0; j < k0 + nk; ++j)
      for (int64_t c = 0; c < hd; ++c) qv[j * hd + c] = quant1(widen(V[j * hd + c]), sv[kb]);
  }
#pragma omp parallel for schedule(static)
  for (int64_t qb = 0; qb < nb; ++qb) {
    const int64_t i0 = qb * PV_BLOCK, ni = (S - i0) < PV_BLOCK ? (S - i0) : PV_BLOCK;
    float* sp = (float*)xmalloc(sizeof(float) * (size_t)nb);
    int8_t* qp = (int8_t*)xmalloc((size_t)(ni * S)); /* the query block's codes, [ni][S] */
    float* terms = (float*)xmalloc(sizeof(float) * (size_t)nb);
    for (int64_t kb = 0; kb < nb; ++kb) {
      const int64_t k0 = kb * PV_BLOCK, nk = (S - k0) < PV_BLOCK ? (S - k0) : PV_BLOCK;
      sp[kb] = block_absmax_step(P + i0 * S + k0, ni, nk, S);
      for (int64_t i = 0; i < ni; ++i)
        for (int64_t j = k0; j < k0 + nk; ++j) qp[i * S + j] = quant1(widen(P[(i0 + i) * S + j]), sp[kb]);
    }
    for (int64_t i = 0; i < ni; ++i)
      for (int64_t c = 0; c < hd; ++c) {
        for (int64_t kb = 0; kb < nb; ++kb) {
          const int64_t k0 = kb * PV_BLOCK, k1 = (S - k0) < PV_BLOCK ? S : k0 + PV_BLOCK;
          int64_t acc = 0; /* exact: |acc| <= 64 * 128 * 128 */
          for (int64_t j = k0; j < k1; ++j) acc += (int64_t)qp[i * S + j] * (int64_t)qv[j * hd + c];
          terms[kb] = cref_mul(cref_mul((float)acc, sp[kb]), sv[kb]);
        }
        O[(i0 + i) * hd + c] = cref_rsum(terms, nb, 1, CHUNK);
      }
    free(sp); free(qp); free(terms);
  }
  free(sv); free(qv);
  return 0;
}

/* ======================================================================== */
/* R18: dQ accumulated in 64-bit fixed point                                 */
/* ======================================================================== */
/* The paper's deterministic flash backward accumulates the query gradient in 64-bit fixed point, which
   makes the sum independent of the order in which keys are visited (training-details paragraph on int8
   computation).  Here each product dS * K (exact: two bf16 significands) is scaled by 2^F and rounded to
   the nearest integer, ties to even; products and their sum are taken modulo 2^64 (two's complement), so
   every order of the keys gives the same 64 bits.  The sum times 2^-F is rounded once to binary32 under
   R0.  This implementation works in 80-bit long double, whose 64-bit significand holds every product
   times 2^F and every int64 exactly. */
uint64_t cref_fx_product(uint16_t a, uint16_t b, int32_t frac_bits) {
  const double p = (double)widen(a) * (double)widen(b); /* exact: 8 x 8 significant bits */
  if (p == 0.0) return 0;
  const long double x = ldexpl((long double)p, frac_bits);
  const long double r = nearbyintl(x); /* default rounding mode: ties to even */
  long double m = fabsl(r);
  const long double two64 = ldexpl(1.0L, 64);
  if (m >= two64) m = fmodl(m, two64); /* exact */
  const uint64_t u = (uint64_t)m;
  return r < 0 ? (uint64_t)0 - u : u;
}

float cref_fx_to_f32(uint64_t sum, int32_t frac_bits) {
  const int64_t s = (int64_t)sum;
  if (s == 0) return 0.0f;
  const float r = (float)(long double)s; /* one rounding to 24 significant bits, ties to even */
  /* r * 2^-F is exact unless it lies below 2^-126, where R0 gives a zero of its sign */
  if (fabsl(ldexpl((long double)r, -frac_bits)) < ldexpl(1.0L, -126)) return copysignf(0.0f, r);
  return ldexpf(r, -frac_bits);
}

int cref_attn_dq_fixed(int64_t S, int64_t hd, int64_t window, int32_t frac_bits, const uint16_t* dS,
                       const uint16_t* K, float* dQ) {
  if (S < 1 || hd < 1 || window < 0 || frac_bits < 1 || frac_bits > 62 || !dS || !K || !dQ) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < S; ++i) {
    const int64_t j0 = (window > 0 && i - window + 1 > 0) ? i - window + 1 : 0;
    for (int64_t c = 0; c < hd; ++c) {
      uint64_t sum = 0;
      for (int64_t j = j0; j <= i; ++j) sum += cref_fx_product(dS[i * S + j], K[j * hd + c], frac_bits);
      dQ[i * hd + c] = cref_fx_to_f32(sum, frac_bits);
    }
  }
  return 0;
}

/* ======================================================================== */
/* R19: int8 projections inside the block, LSQ gradient of activation steps  */
/* ======================================================================== */
/* The paper trains the four projections of every block with int8 weights (re-pinned per-channel steps, R13)
   and int8 activations with a learned per-tensor step (LSQ), and runs both gradient GEMMs in int8 (R14).
   The step's gradient is LSQ's: for each element the derivative of the dequantised value s q with respect
   to s, round(v) - v inside the integer range and the clamp bound outside it (v = x / s), times LSQ's
   gradient scale 1/sqrt(Q_P K) for K features. */
static float lsq_delta(float x, float s) {
  s = daz(s);
  if (!(s > 0.0f)) return 0.0f;
  const float v = cref_div(x, s);
  if (isnan(v)) return 0.0f;
  if (v < -128.0f) return -128.0f;
  if (v > 127.0f) return 127.0f;
  return cref_sub((float)rint((double)v), v); /* rint: nearest integer, ties to even */
}

float cref_lsq_step_grad(int64_t T, int64_t K, const uint16_t* x, float s, const float* dx) {
  if (T < 0 || K < 1) return 0.0f;
  const int64_t n = T * K;
  float* t = (float*)xmalloc(sizeof(float) * (size_t)n);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) t[i] = cref_mul(dx[i], lsq_delta(widen(x[i]), s));
  const float sum = cref_rsum(t, n, 1, CHUNK);
  free(t);
  const float gamma = cref_inv_sqrt_int(127 * K); /* RN32(1/sqrt(127 K)) */
  return cref_mul(sum, gamma);
}

int cref_num_threads(void) { return omp_get_max_threads(); }

void cref_set_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
}
