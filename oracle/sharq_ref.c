/*
 * sharq_ref.c -- plain C oracle of the SharQ sparse-dense FP4 linear layer
 * (MXFP4 and NVFP4), TEST INFRASTRUCTURE ONLY (see sharq_ref.h).  Built with -ffp-contract=off
 * and without fast-math, so every float operation below is one IEEE fp32
 * operation rounded to nearest even and every double one IEEE fp64 operation.
 *
 * Per row (SharQ Sec. 3.1, 3.3, 3.4; App. A.1):
 *   y      = RMSNorm(x) * gamma, or x (Sec. 3.4 "Fused sparse-residual
 *            preparation"; sum of squares as a balanced binary tree, R1)
 *   keep   = the n largest |y| of every m positions, ties to the lower index
 *            (Sec. 3.1 eq. "dynamic-mask"; Sec. 3.3 eq. "sharq-sparse-backbone")
 *   backbone: per 32 positions, E8M0 from the largest kept |y|, E2M1 codes of
 *            the kept values (Sec. 3.3 eq. "sharq-quantized-backbone")
 *   R      = y - dequant(backbone) (Sec. 3.3 eq. "sharq-residual"), then its
 *            own E8M0 and E2M1 codes per 32 positions
 *   Y      = dequant(backbone) W^T + dequant(R) W^T in fp64 (Sec. 3.3 eq.
 *            "sharq-output")
 * NVFP4 (App. A.1.2-A.1.3) replaces the E8M0 block scales by E4M3 ones, per
 * 32 positions for the backbone and 16 for the residual, under one fp32
 * per-tensor scale; see the NVFP4 section below.
 */
#include "sharq_ref.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

enum { REF_OK = 0, REF_EINVAL = 1, REF_EUNSUPPORTED = 2 };

static int g_threads = 0;

void sharq_ref_set_threads(int threads) { g_threads = threads; }

int sharq_ref_max_threads(void) {
#ifdef _OPENMP
  return g_threads > 0 ? g_threads : omp_get_max_threads();
#else
  return 1;
#endif
}

static float bf16_value(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

static int sign_bit(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return (int)(u >> 31);
}

/* The E2M1 magnitudes (App. A.1.2), indexed by the three low code bits. */
static const double kE2M1[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

/* Nearest E2M1 magnitude by exhaustive search over the eight, a tie going to
 * the even code; values beyond 6 take 6.  Bit 3 carries the sign of v, also
 * for zero (R5). */
static uint8_t e2m1_code(float v) {
  const double a = fabs((double)v);
  int best = 0;
  double best_d = a;
  for (int c = 1; c < 8; ++c) {
    const double d = fabs(a - kE2M1[c]);
    if (d < best_d || (d == best_d && c % 2 == 0)) {
      best = c;
      best_d = d;
    }
  }
  return (uint8_t)((sign_bit(v) << 3) | best);
}

static double e2m1_value(uint8_t code) { return (code & 8) ? -kE2M1[code & 7] : kE2M1[code & 7]; }

/* Shared exponent of a block with largest magnitude amax (R4, R13), clamped
 * to [-127, 127]; -127 for an all-zero block.
 *   floor: floor(log2 amax) - 2, the exponent of amax less that of 6's binade;
 *   ceil:  the smallest e with amax <= 6 * 2^e, found by stepping e. */
static int e8m0_exponent(float amax, int ceil_rule) {
  if (!(amax > 0.0f)) return -127;
  int ex;
  frexp((double)amax, &ex); /* amax = f 2^ex, f in [0.5, 1): floor(log2 amax) = ex - 1 */
  int e = ex - 1 - 2;
  if (ceil_rule) {
    while ((double)amax > 6.0 * ldexp(1.0, e)) ++e;
    while (e > -127 && (double)amax <= 6.0 * ldexp(1.0, e - 1)) --e;
  }
  if (e < -127) e = -127;
  if (e > 127) e = 127;
  return e;
}

/* Sum of squares of x[0..K) as the balanced binary tree over the row padded
 * with zeros to a power of two (R1): a recursion over aligned halves. */
static float tree_sum_sq(const float *x, int64_t lo, int64_t width, int64_t K) {
  if (width == 1) return lo < K ? x[lo] * x[lo] : 0.0f;
  const float a = tree_sum_sq(x, lo, width / 2, K);
  const float b = tree_sum_sq(x, lo + width / 2, width / 2, K);
  return a + b;
}

/* Keep mask of one row (Sec. 3.1 eq. "dynamic-mask"): the n largest |y| of
 * every m positions, a tie going to the lower index; pairs (App. A.1.4, R8):
 * the n/2 of the m/2 adjacent pairs with the largest max(|y_2i|, |y_2i+1|),
 * a tie going to the lower pair, each kept whole. */
static void keep_mask(const float *y, int64_t K, int n, int m, int pairs, uint8_t *keep) {
  for (int64_t g = 0; g < K / m; ++g) {
    const float *e = y + g * m;
    if (pairs) {
      for (int i = 0; i < m / 2; ++i) {
        const float si = fmaxf(fabsf(e[2 * i]), fabsf(e[2 * i + 1]));
        int rank = 0;
        for (int j = 0; j < m / 2; ++j) {
          if (j == i) continue;
          const float sj = fmaxf(fabsf(e[2 * j]), fabsf(e[2 * j + 1]));
          if (sj > si || (sj == si && j < i)) ++rank;
        }
        keep[g * m + 2 * i] = keep[g * m + 2 * i + 1] = (uint8_t)(rank < n / 2);
      }
      continue;
    }
    for (int p = 0; p < m; ++p) {
      const float ap = fabsf(e[p]);
      int rank = 0;
      for (int q = 0; q < m; ++q) {
        if (q == p) continue;
        const float aq = fabsf(e[q]);
        if (aq > ap || (aq == ap && q < p)) ++rank;
      }
      keep[g * m + p] = (uint8_t)(rank < n);
    }
  }
}

/* Backbone metadata of one row from its keep mask: 2:4, per group the two
 * kept positions i0 | i1 << 2, two groups per byte, even group low; 4:8, the
 * keep mask byte of every group. */
static void pack_meta(const uint8_t *keep, int64_t K, int m, uint8_t *spm) {
  memset(spm, 0, (size_t)(K / 8));
  for (int64_t g = 0; g < K / m; ++g) {
    if (m == 4) {
      int idx[2], c = 0;
      for (int p = 0; p < 4; ++p)
        if (keep[g * 4 + p]) idx[c++] = p;
      const uint8_t nib = (uint8_t)(idx[0] | (idx[1] << 2));
      spm[g / 2] |= (uint8_t)(nib << (4 * (g & 1)));
    } else {
      uint8_t mask = 0;
      for (int p = 0; p < 8; ++p) mask |= (uint8_t)(keep[g * 8 + p] << p);
      spm[g] = mask;
    }
  }
}

/* y of one row (Sec. 3.4): RMSNorm(x) * gamma with the tree sum of squares
 * (R1) and r = 1 / sqrt(ss / K + eps) in fp64 rounded to fp32 (R2), or x
 * itself without gamma (r = 1).  Returns r. */
static float norm_row(const uint16_t *xrow, const uint16_t *gamma, float eps, int64_t K, float *x, float *y) {
  for (int64_t k = 0; k < K; ++k) x[k] = bf16_value(xrow[k]);
  if (!gamma) {
    memcpy(y, x, sizeof(float) * (size_t)K);
    return 1.0f;
  }
  int64_t P = 1;
  while (P < K) P *= 2;
  const float ss = tree_sum_sq(x, 0, P, K);
  const float rt = (float)(1.0 / sqrt((double)ss / (double)K + (double)eps));
  for (int64_t k = 0; k < K; ++k) {
    const float xr = x[k] * rt;
    y[k] = xr * bf16_value(gamma[k]);
  }
  return rt;
}

/* One row: y in, packed buffers out (row pointers). */
static void prepare_row(const float *y, int64_t K, int n, int m, int ceil_rule, uint8_t *spc, uint8_t *spm,
                        uint8_t *sps, uint8_t *dnc, uint8_t *dns, uint8_t *keep_bits, float *R, uint8_t *keep) {
  keep_mask(y, K, n, m, 0, keep);
  int64_t kept_idx = 0;
  memset(spc, 0, (size_t)(K * n / m / 2));
  memset(dnc, 0, (size_t)(K / 2));
  for (int64_t b = 0; b < K / 32; ++b) {
    const float *yb = y + 32 * b;
    const uint8_t *kb = keep + 32 * b;
    float amax = 0.0f;
    for (int k = 0; k < 32; ++k)
      if (kb[k] && fabsf(yb[k]) > amax) amax = fabsf(yb[k]);
    const int e = e8m0_exponent(amax, ceil_rule);
    const float s = ldexpf(1.0f, e);
    sps[b] = (uint8_t)(e + 127);
    for (int k = 0; k < 32; ++k) {
      float d = 0.0f;
      if (kb[k]) {
        const uint8_t c = e2m1_code(yb[k] / s);
        d = (float)(e2m1_value(c) * (double)s);
        spc[kept_idx / 2] |= (uint8_t)(c << (4 * (kept_idx & 1)));
        ++kept_idx;
      }
      R[32 * b + k] = yb[k] - d;
    }
  }
  pack_meta(keep, K, m, spm);
  /* residual */
  for (int64_t b = 0; b < K / 32; ++b) {
    float amax = 0.0f;
    for (int k = 0; k < 32; ++k)
      if (fabsf(R[32 * b + k]) > amax) amax = fabsf(R[32 * b + k]);
    const int e = e8m0_exponent(amax, ceil_rule);
    const float s = ldexpf(1.0f, e);
    dns[b] = (uint8_t)(e + 127);
    for (int k = 0; k < 32; ++k) {
      const int64_t i = 32 * b + k;
      dnc[i / 2] |= (uint8_t)(e2m1_code(R[i] / s) << (4 * (i & 1)));
    }
  }
  if (keep_bits) {
    memset(keep_bits, 0, (size_t)(K / 8));
    for (int64_t i = 0; i < K; ++i) keep_bits[i / 8] |= (uint8_t)(keep[i] << (i & 7));
  }
}

int sharq_ref_prepare(const uint16_t *X, int64_t M, int64_t K, int64_t ldx, const uint16_t *gamma, float eps,
                      int n, int m, int scale_rule, uint8_t *sp_codes, uint8_t *sp_meta, uint8_t *sp_scale,
                      uint8_t *dn_codes, uint8_t *dn_scale, float *r, uint8_t *keep) {
  if (M < 0 || K <= 0 || K % 32 != 0 || ldx < K || m <= 0 || n < 0 || n > m || K % m != 0) return REF_EINVAL;
  if (scale_rule != 0 && scale_rule != 1) return REF_EINVAL;
  if (!(eps >= 0.0f)) return REF_EINVAL;
  if (!((n == 2 && m == 4) || (n == 4 && m == 8))) return REF_EUNSUPPORTED;
  if (M == 0) return REF_OK;
  if (!X || !sp_codes || !sp_meta || !sp_scale || !dn_codes || !dn_scale) return REF_EINVAL;
  int failed = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 4) num_threads(sharq_ref_max_threads())
#endif
  for (int64_t t = 0; t < M; ++t) {
    float *x = malloc(sizeof(float) * (size_t)K * 3);
    uint8_t *kp = malloc((size_t)K);
    if (!x || !kp) {
      failed = 1;
      free(x);
      free(kp);
      continue;
    }
    float *y = x + K, *R = x + 2 * K;
    const float rt = norm_row(X + t * ldx, gamma, eps, K, x, y);
    if (r) r[t] = rt;
    prepare_row(y, K, n, m, scale_rule, sp_codes + t * (K * n / m / 2), sp_meta + t * (K / 8),
                sp_scale + t * (K / 32), dn_codes + t * (K / 2), dn_scale + t * (K / 32),
                keep ? keep + t * (K / 8) : NULL, R, kp);
    free(x);
    free(kp);
  }
  return failed ? REF_EINVAL : REF_OK;
}

int sharq_ref_quantize_weight(const uint16_t *W, int64_t N, int64_t K, int64_t ldw, int scale_rule, uint8_t *codes,
                              uint8_t *scale) {
  if (N < 0 || K <= 0 || K % 32 != 0 || ldw < K) return REF_EINVAL;
  if (scale_rule != 0 && scale_rule != 1) return REF_EINVAL;
  if (N == 0) return REF_OK;
  if (!W || !codes || !scale) return REF_EINVAL;
#ifdef _OPENMP
#pragma omp parallel for schedule(static) num_threads(sharq_ref_max_threads())
#endif
  for (int64_t r = 0; r < N; ++r) {
    memset(codes + r * (K / 2), 0, (size_t)(K / 2));
    for (int64_t b = 0; b < K / 32; ++b) {
      float v[32], amax = 0.0f;
      for (int k = 0; k < 32; ++k) {
        v[k] = bf16_value(W[r * ldw + 32 * b + k]);
        if (fabsf(v[k]) > amax) amax = fabsf(v[k]);
      }
      const int e = e8m0_exponent(amax, scale_rule);
      const float s = ldexpf(1.0f, e);
      scale[r * (K / 32) + b] = (uint8_t)(e + 127);
      for (int k = 0; k < 32; ++k) {
        const int64_t i = 32 * b + k;
        codes[r * (K / 2) + i / 2] |= (uint8_t)(e2m1_code(v[k] / s) << (4 * (i & 1)));
      }
    }
  }
  return REF_OK;
}

/* fp64 values of one packed MXFP4 row (dense codes, all K positions). */
static void dequant_dense(const uint8_t *codes, const uint8_t *scale, int64_t K, double *out) {
  for (int64_t i = 0; i < K; ++i) {
    const uint8_t c = (uint8_t)((codes[i / 2] >> (4 * (i & 1))) & 0xF);
    out[i] = e2m1_value(c) * ldexp(1.0, (int)scale[i / 32] - 127);
  }
}

/* fp64 values of one compressed backbone row (zeros at the dropped positions). */
static void dequant_backbone(const uint8_t *spc, const uint8_t *spm, const uint8_t *sps, int64_t K, int n, int m,
                             double *out) {
  int64_t kept = 0;
  for (int64_t g = 0; g < K / m; ++g) {
    for (int p = 0; p < m; ++p) {
      int on;
      if (m == 4) {
        const uint8_t nib = (uint8_t)((spm[g / 2] >> (4 * (g & 1))) & 0xF);
        on = p == (nib & 3) || p == (nib >> 2);
      } else {
        on = (spm[g] >> p) & 1;
      }
      const int64_t i = g * m + p;
      if (on) {
        const uint8_t c = (uint8_t)((spc[kept / 2] >> (4 * (kept & 1))) & 0xF);
        out[i] = e2m1_value(c) * ldexp(1.0, (int)sps[i / 32] - 127);
        ++kept;
      } else {
        out[i] = 0.0;
      }
    }
  }
  (void)n;
}

int sharq_ref_linear(int64_t M, int64_t K, int n, int m, const uint8_t *sp_codes, const uint8_t *sp_meta,
                     const uint8_t *sp_scale, const uint8_t *dn_codes, const uint8_t *dn_scale, int64_t N,
                     const uint8_t *w_codes, const uint8_t *w_scale, double *Y, int64_t ldy) {
  if (M < 0 || N < 0 || K <= 0 || K % 32 != 0 || ldy < N || m <= 0 || n < 0 || n > m || K % m != 0)
    return REF_EINVAL;
  if (!((n == 2 && m == 4) || (n == 4 && m == 8))) return REF_EUNSUPPORTED;
  if (M == 0 || N == 0) return REF_OK;
  if (!sp_codes || !sp_meta || !sp_scale || !dn_codes || !dn_scale || !w_codes || !w_scale || !Y) return REF_EINVAL;
  double *w = malloc(sizeof(double) * (size_t)(N * K));
  if (!w) return REF_EINVAL;
  for (int64_t j = 0; j < N; ++j) dequant_dense(w_codes + j * (K / 2), w_scale + j * (K / 32), K, w + j * K);
  int failed = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(sharq_ref_max_threads())
#endif
  for (int64_t t = 0; t < M; ++t) {
    double *a = malloc(sizeof(double) * (size_t)K * 2);
    if (!a) {
      failed = 1;
      continue;
    }
    double *sp = a, *dn = a + K;
    dequant_backbone(sp_codes + t * (K * n / m / 2), sp_meta + t * (K / 8), sp_scale + t * (K / 32), K, n, m, sp);
    dequant_dense(dn_codes + t * (K / 2), dn_scale + t * (K / 32), K, dn);
    for (int64_t j = 0; j < N; ++j) {
      const double *wj = w + j * K;
      double acc_sp = 0.0, acc_dn = 0.0;
      for (int64_t k = 0; k < K; ++k) {
        acc_sp += sp[k] * wj[k];
        acc_dn += dn[k] * wj[k];
      }
      Y[t * ldy + j] = acc_sp + acc_dn;
    }
    free(a);
  }
  free(w);
  return failed ? REF_EINVAL : REF_OK;
}

/* ---------------------------------------------------------------------------
 * NVFP4 (App. A.1.2-A.1.3, reading R7).  One fp32 per-tensor scale S per call
 * and one E4M3 scale d per block of `len` positions (32 for the backbone and
 * the weight, 16 for the residual):
 *   S = fl32(amax / 2688) over every value of the call, or 1 if all are 0;
 *   d = E4M3(fl32(amax_block / fl32(6 S)));
 *   q = E2M1(fl32(v / fl32(d S))), a zero of v's sign when d = 0;
 *   value = fl32(fl32(q d) S).
 * ------------------------------------------------------------------------- */

/* Value of an E4M3 code (bias 7; exponent field 0: 2^-6 * M/8). */
static double e4m3_value(int code) {
  const int E = (code >> 3) & 15, M = code & 7;
  return E == 0 ? ldexp(M / 8.0, -6) : ldexp(1.0 + M / 8.0, E - 7);
}

uint8_t sharq_ref_e4m3_code(float a) {
  const double v = (double)a;
  if (!(v > 0.0)) return 0;
  int best = 0;
  double best_d = v;
  for (int c = 1; c <= 0x7E; ++c) { /* 0x7F is NaN */
    const double d = fabs(v - e4m3_value(c));
    if (d < best_d || (d == best_d && c % 2 == 0)) {
      best = c;
      best_d = d;
    }
  }
  return (uint8_t)best;
}

static float nv_tensor_scale(float amax) { return amax > 0.0f ? amax / 2688.0f : 1.0f; }

/* One block of len values; present == NULL: every position.  Codes go to
 * codes[k] (one per position, 0 where absent), values to deq[k]; returns the
 * block's E4M3 code. */
static uint8_t nv_block(const float *v, const uint8_t *present, int len, float S, uint8_t *codes, float *deq) {
  float amax = 0.0f;
  for (int k = 0; k < len; ++k)
    if ((!present || present[k]) && fabsf(v[k]) > amax) amax = fabsf(v[k]);
  const float six_s = 6.0f * S;
  const uint8_t dc = sharq_ref_e4m3_code(amax / six_s);
  const float d = (float)e4m3_value(dc);
  const float step = d * S;
  for (int k = 0; k < len; ++k) {
    if (present && !present[k]) {
      codes[k] = 0;
      deq[k] = 0.0f;
      continue;
    }
    uint8_t c;
    if (d > 0.0f)
      c = e2m1_code(step > 0.0f ? v[k] / step : v[k]);
    else
      c = (uint8_t)(sign_bit(v[k]) << 3);
    codes[k] = c;
    const float qd = (float)(e2m1_value(c) * (double)d); /* exact */
    deq[k] = qd * S;
  }
  return dc;
}

static void pack_codes(const uint8_t *codes, int64_t count, uint8_t *out) {
  memset(out, 0, (size_t)(count / 2));
  for (int64_t i = 0; i < count; ++i) out[i / 2] |= (uint8_t)(codes[i] << (4 * (i & 1)));
}

int sharq_ref_prepare_nv(const uint16_t *X, int64_t M, int64_t K, int64_t ldx, const uint16_t *gamma, float eps,
                         int n, int m, int pairs, const float *tensor_scale_in, float *tensor_scale_out,
                         uint8_t *sp_codes, uint8_t *sp_meta, uint8_t *sp_scale, uint8_t *dn_codes,
                         uint8_t *dn_scale) {
  if (M < 0 || K <= 0 || K % 32 != 0 || ldx < K || m <= 0 || n < 0 || n > m || K % m != 0) return REF_EINVAL;
  if (!(eps >= 0.0f) || (pairs != 0 && pairs != 1)) return REF_EINVAL;
  if (!((n == 2 && m == 4) || (n == 4 && m == 8))) return REF_EUNSUPPORTED;
  if (pairs && m != 8) return REF_EUNSUPPORTED;
  if (M == 0) return REF_OK;
  if (!X || !sp_codes || !sp_meta || !sp_scale || !dn_codes || !dn_scale || !tensor_scale_out) return REF_EINVAL;
  /* pass 1: y of every row, and S */
  float *Y = malloc(sizeof(float) * (size_t)(M * K));
  if (!Y) return REF_EINVAL;
  int failed = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 4) num_threads(sharq_ref_max_threads())
#endif
  for (int64_t t = 0; t < M; ++t) {
    float *x = malloc(sizeof(float) * (size_t)K);
    if (!x) {
      failed = 1;
      continue;
    }
    norm_row(X + t * ldx, gamma, eps, K, x, Y + t * K);
    free(x);
  }
  if (failed) {
    free(Y);
    return REF_EINVAL;
  }
  float S;
  if (tensor_scale_in) {
    S = *tensor_scale_in;
  } else {
    float amax = 0.0f;
    for (int64_t i = 0; i < M * K; ++i)
      if (fabsf(Y[i]) > amax) amax = fabsf(Y[i]);
    S = nv_tensor_scale(amax);
  }
  *tensor_scale_out = S;
  /* pass 2: every row */
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 4) num_threads(sharq_ref_max_threads())
#endif
  for (int64_t t = 0; t < M; ++t) {
    float *R = malloc(sizeof(float) * (size_t)K * 2);
    uint8_t *buf = malloc((size_t)K * 3);
    if (!R || !buf) {
      failed = 1;
      free(R);
      free(buf);
      continue;
    }
    const float *y = Y + t * K;
    float *deq = R + K;
    uint8_t *keep = buf, *c = buf + K, *kept = buf + 2 * K;
    keep_mask(y, K, n, m, pairs, keep);
    int64_t nk = 0;
    for (int64_t b = 0; b < K / 32; ++b) {
      sp_scale[t * (K / 32) + b] = nv_block(y + 32 * b, keep + 32 * b, 32, S, c + 32 * b, deq + 32 * b);
      for (int k = 0; k < 32; ++k) {
        const int64_t i = 32 * b + k;
        R[i] = y[i] - deq[i];
        if (keep[i]) kept[nk++] = c[i];
      }
    }
    pack_codes(kept, nk, sp_codes + t * (K * n / m / 2));
    pack_meta(keep, K, m, sp_meta + t * (K / 8));
    for (int64_t b = 0; b < K / 16; ++b)
      dn_scale[t * (K / 16) + b] = nv_block(R + 16 * b, NULL, 16, S, c + 16 * b, deq + 16 * b);
    pack_codes(c, K, dn_codes + t * (K / 2));
    free(R);
    free(buf);
  }
  free(Y);
  return failed ? REF_EINVAL : REF_OK;
}

int sharq_ref_quantize_weight_nv(const uint16_t *W, int64_t N, int64_t K, int64_t ldw, uint8_t *codes,
                                 uint8_t *scale, float *tensor_scale) {
  if (N < 0 || K <= 0 || K % 32 != 0 || ldw < K) return REF_EINVAL;
  if (N == 0) return REF_OK;
  if (!W || !codes || !scale || !tensor_scale) return REF_EINVAL;
  float amax = 0.0f;
  for (int64_t r = 0; r < N; ++r)
    for (int64_t k = 0; k < K; ++k)
      if (fabsf(bf16_value(W[r * ldw + k])) > amax) amax = fabsf(bf16_value(W[r * ldw + k]));
  const float S = nv_tensor_scale(amax);
  *tensor_scale = S;
  int failed = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(static) num_threads(sharq_ref_max_threads())
#endif
  for (int64_t r = 0; r < N; ++r) {
    float *v = malloc(sizeof(float) * (size_t)K * 2);
    uint8_t *c = malloc((size_t)K);
    if (!v || !c) {
      failed = 1;
      free(v);
      free(c);
      continue;
    }
    for (int64_t k = 0; k < K; ++k) v[k] = bf16_value(W[r * ldw + k]);
    for (int64_t b = 0; b < K / 32; ++b)
      scale[r * (K / 32) + b] = nv_block(v + 32 * b, NULL, 32, S, c + 32 * b, v + K + 32 * b);
    pack_codes(c, K, codes + r * (K / 2));
    free(v);
    free(c);
  }
  return failed ? REF_EINVAL : REF_OK;
}

/* fp64 values of one NVFP4 row of dense codes under E4M3 scales per `block`
 * positions and the per-tensor scale S. */
static void dequant_dense_nv(const uint8_t *codes, const uint8_t *scale, int block, float S, int64_t K, double *out) {
  for (int64_t i = 0; i < K; ++i) {
    const uint8_t c = (uint8_t)((codes[i / 2] >> (4 * (i & 1))) & 0xF);
    out[i] = e2m1_value(c) * e4m3_value(scale[i / block]) * (double)S;
  }
}

int sharq_ref_linear_nv(int64_t M, int64_t K, int n, int m, const uint8_t *sp_codes, const uint8_t *sp_meta,
                        const uint8_t *sp_scale, const uint8_t *dn_codes, const uint8_t *dn_scale,
                        float tensor_scale_x, int64_t N, const uint8_t *w_codes, const uint8_t *w_scale,
                        float tensor_scale_w, double *Y, int64_t ldy) {
  if (M < 0 || N < 0 || K <= 0 || K % 32 != 0 || ldy < N || m <= 0 || n < 0 || n > m || K % m != 0)
    return REF_EINVAL;
  if (!((n == 2 && m == 4) || (n == 4 && m == 8))) return REF_EUNSUPPORTED;
  if (M == 0 || N == 0) return REF_OK;
  if (!sp_codes || !sp_meta || !sp_scale || !dn_codes || !dn_scale || !w_codes || !w_scale || !Y) return REF_EINVAL;
  /* the weight's one scale per 32 positions serves both paths (its dense view
   * repeats it over the two 16-position halves) */
  double *w = malloc(sizeof(double) * (size_t)(N * K));
  if (!w) return REF_EINVAL;
  for (int64_t j = 0; j < N; ++j)
    dequant_dense_nv(w_codes + j * (K / 2), w_scale + j * (K / 32), 32, tensor_scale_w, K, w + j * K);
  int failed = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(sharq_ref_max_threads())
#endif
  for (int64_t t = 0; t < M; ++t) {
    double *a = malloc(sizeof(double) * (size_t)K * 2);
    if (!a) {
      failed = 1;
      continue;
    }
    double *sp = a, *dn = a + K;
    /* backbone: the compressed codes at their kept positions, zeros elsewhere */
    const uint8_t *spm = sp_meta + t * (K / 8), *spc = sp_codes + t * (K * n / m / 2);
    int64_t kept = 0;
    for (int64_t g = 0; g < K / m; ++g) {
      for (int p = 0; p < m; ++p) {
        int on;
        if (m == 4) {
          const uint8_t nib = (uint8_t)((spm[g / 2] >> (4 * (g & 1))) & 0xF);
          on = p == (nib & 3) || p == (nib >> 2);
        } else {
          on = (spm[g] >> p) & 1;
        }
        const int64_t i = g * m + p;
        if (on) {
          const uint8_t c = (uint8_t)((spc[kept / 2] >> (4 * (kept & 1))) & 0xF);
          sp[i] = e2m1_value(c) * e4m3_value(sp_scale[t * (K / 32) + i / 32]) * (double)tensor_scale_x;
          ++kept;
        } else {
          sp[i] = 0.0;
        }
      }
    }
    dequant_dense_nv(dn_codes + t * (K / 2), dn_scale + t * (K / 16), 16, tensor_scale_x, K, dn);
    for (int64_t j = 0; j < N; ++j) {
      const double *wj = w + j * K;
      double acc_sp = 0.0, acc_dn = 0.0;
      for (int64_t k = 0; k < K; ++k) {
        acc_sp += sp[k] * wj[k];
        acc_dn += dn[k] * wj[k];
      }
      Y[t * ldy + j] = acc_sp + acc_dn;
    }
    free(a);
  }
  free(w);
  return failed ? REF_EINVAL : REF_OK;
}
