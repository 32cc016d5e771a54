/*
 * fxpq_oracle.c -- plain, slow, exact CPU oracle of the DFX calibration hot path.
 *
 * TEST INFRASTRUCTURE ONLY (see fxpq_oracle.h).  Built with gcc, no -ffast-math.
 *
 * Method: FxP-QNet (Shawahna et al., IEEE Access 2022).
 *   - format and ranges: Sec. "Dynamic Fixed-Point Representation", Eq. 1, Eq. 12;
 *   - quantizer: Sec. "Quantization Methodology", Eq. 10-11 (round half to even),
 *     Eq. 13 (1-bit binary case);
 *   - sign strategy: Eq. 6;
 *   - data-structure error: Eq. 14;
 *   - integer C-Block: Fig. "FxP-QNet hardware" and the text below it (bias
 *     aligned by a shift, Scale multiply, ReLU, FxP-QLayer requantization);
 *   - FxP-QLayer placement and pooling: Sec. "FxP-QLayer".
 *
 * Every value the quantizer sees is handled as a dyadic rational m * 2^e.
 */
#include "fxpq_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

typedef __int128 i128;
typedef unsigned __int128 u128;

/* ------------------------------------------------------------------------- */
/* Wide fixed-point accumulator for exact sums of non-negative dyadic values.  */
/* Bit 0 of limb 0 weighs 2^KA_LSB.                                           */
/* ------------------------------------------------------------------------- */
#define KA_LIMBS 40
#define KA_LSB (-1280)

typedef struct {
  uint64_t w[KA_LIMBS];
} kacc;

static void ka_zero(kacc* a) { memset(a, 0, sizeof(*a)); }

/* a += m * 2^e, m >= 0.  Returns 0, or ORC_ERANGE if outside the window. */
static int ka_add(kacc* a, u128 m, int e) {
  if (m == 0) return ORC_OK;
  int p = e - KA_LSB;
  if (p < 0 || p + 192 > 64 * KA_LIMBS) return ORC_ERANGE;
  int limb = p / 64, off = p % 64;
  uint64_t part[3];
  part[0] = (uint64_t)(m << off);
  part[1] = off ? (uint64_t)(m >> (64 - off)) : (uint64_t)(m >> 64);
  part[2] = off ? (uint64_t)(m >> (128 - off)) : 0;
  unsigned carry = 0;
  for (int i = 0; i < 3 || carry; ++i) {
    int j = limb + i;
    if (j >= KA_LIMBS) return ORC_ERANGE;
    uint64_t add = (i < 3) ? part[i] : 0;
    u128 s = (u128)a->w[j] + add + carry;
    a->w[j] = (uint64_t)s;
    carry = (unsigned)(s >> 64);
  }
  return ORC_OK;
}

static void ka_merge(kacc* a, const kacc* b) {
  unsigned carry = 0;
  for (int j = 0; j < KA_LIMBS; ++j) {
    u128 s = (u128)a->w[j] + b->w[j] + carry;
    a->w[j] = (uint64_t)s;
    carry = (unsigned)(s >> 64);
  }
}

/* -1, 0, +1 as a < b, a == b, a > b. */
static int ka_cmp(const kacc* a, const kacc* b) {
  for (int j = KA_LIMBS - 1; j >= 0; --j) {
    if (a->w[j] != b->w[j]) return a->w[j] < b->w[j] ? -1 : 1;
  }
  return 0;
}

static double ka_to_double(const kacc* a) {
  long double r = 0.0L;
  for (int j = KA_LIMBS - 1; j >= 0; --j) {
    if (a->w[j]) r += ldexpl((long double)a->w[j], KA_LSB + 64 * j);
  }
  return (double)r;
}

/* ------------------------------------------------------------------------- */
/* Format, sign strategy, quantizer.                                          */
/* ------------------------------------------------------------------------- */
int orc_qrange(int k, int sign, int64_t* qmin, int64_t* qmax) {
  if (k < 1 || k > 32 || (sign != 0 && sign != 1)) return ORC_EINVAL;
  /* Eq. 12 with alpha + beta = k: Qmin = -S / 2^(S-k), Qmax = 2^(k-S) - 1. */
  *qmax = ((int64_t)1 << (k - sign)) - 1;
  *qmin = sign ? -((int64_t)1 << (k - sign)) : 0;
  return ORC_OK;
}

int orc_sign_f32(const float* x, int64_t n) {
  for (int64_t i = 0; i < n; ++i)
    if (x[i] < 0.0f) return 1;
  return 0;
}

int orc_sign_i64(const int64_t* v, int64_t n) {
  for (int64_t i = 0; i < n; ++i)
    if (v[i] < 0) return 1;
  return 0;
}

/* fp32 -> exact dyadic m * 2^e (finite input). */
static int f32_to_dyadic(float x, int64_t* m, int* e) {
  if (!isfinite(x)) return ORC_EINVAL;
  if (x == 0.0f) {
    *m = 0;
    *e = 0;
    return ORC_OK;
  }
  int ex;
  float fr = frexpf(x, &ex);          /* x = fr * 2^ex, 0.5 <= |fr| < 1 */
  *m = (int64_t)ldexpf(fr, 24);       /* exact: fr has at most 24 significant bits */
  *e = ex - 24;
  return ORC_OK;
}

/* Round m / 2^d to the nearest integer, ties to even (d >= 1). */
static i128 rne_shift(i128 m, int d) {
  if (d >= 126) return 0; /* |m| < 2^63 <= 2^(d-1): below one half */
  i128 one = 1;
  i128 q = m >> d; /* floor */
  i128 r = m - (q << d);
  i128 half = one << (d - 1);
  if (r > half || (r == half && (q & 1))) q += 1;
  return q;
}

/* Eq. 10-13 for the dyadic value m * 2^e: returns the code.  *dec gets the
 * integer the code decodes to (the code itself, except +1 for the binary 0). */
static int64_t quant_dyadic(int64_t m, int e, int k, int fl, int sign, int64_t qmin, int64_t qmax,
                            int64_t* dec) {
  if (k == 1 && sign == 1) { /* Eq. 13 */
    int64_t q = (m < 0) ? -1 : 0;
    *dec = (q == 0) ? 1 : -1;
    return q;
  }
  int sh = e + fl; /* x * 2^fl = m * 2^sh */
  int64_t q;
  if (sh >= 0) {
    if (m == 0) {
      q = 0;
    } else if (sh >= 64) {
      q = (m > 0) ? qmax : qmin;
    } else {
      i128 t = (i128)m << sh; /* |m| < 2^63, sh < 64: fits */
      q = (t > qmax) ? qmax : (t < qmin) ? qmin : (int64_t)t;
    }
  } else {
    i128 t = rne_shift((i128)m, -sh);
    q = (t > qmax) ? qmax : (t < qmin) ? qmin : (int64_t)t;
  }
  *dec = q;
  return q;
}

static int bitlen_abs(i128 v) {
  if (v < 0) v = -v;
  int b = 0;
  while (v) {
    ++b;
    v >>= 1;
  }
  return b;
}

/* Exact (x - dec * 2^-fl)^2 added to acc, x = m * 2^e. */
static int add_sq_error(kacc* acc, int64_t m, int e, int64_t dec, int fl) {
  int E = (e < -fl) ? e : -fl;
  int sx = e - E, sq = -fl - E; /* both >= 0 */
  if ((m != 0 && bitlen_abs(m) + sx > 120) || (dec != 0 && bitlen_abs(dec) + sq > 120))
    return ORC_ERANGE;
  i128 a = (i128)m << sx;
  i128 b = (i128)dec << sq;
  i128 d = a - b;
  if (d < 0) d = -d;
  if (d >> 63) return ORC_ERANGE; /* the square must fit 126 bits */
  u128 d2 = (u128)d * (u128)d;
  return ka_add(acc, d2, 2 * E);
}

static int check_fmt(int k, int sign) {
  if (k < 1 || k > 32) return ORC_EINVAL;
  if (sign != 0 && sign != 1) return ORC_EINVAL;
  return ORC_OK;
}

int orc_quantize_f32(const float* x, int64_t n, int k, int fl, int sign, int32_t* codes) {
  if (check_fmt(k, sign) || n < 0) return ORC_EINVAL;
  int64_t qmin, qmax, dec;
  orc_qrange(k, sign, &qmin, &qmax);
  for (int64_t i = 0; i < n; ++i) {
    int64_t m;
    int e;
    if (f32_to_dyadic(x[i], &m, &e)) return ORC_EINVAL;
    codes[i] = (int32_t)quant_dyadic(m, e, k, fl, sign, qmin, qmax, &dec);
  }
  return ORC_OK;
}

int orc_quantize_i64(const int64_t* v, int64_t n, int s, int k, int fl, int sign, int32_t* codes) {
  if (check_fmt(k, sign) || n < 0) return ORC_EINVAL;
  int64_t qmin, qmax, dec;
  orc_qrange(k, sign, &qmin, &qmax);
  for (int64_t i = 0; i < n; ++i) codes[i] = (int32_t)quant_dyadic(v[i], -s, k, fl, sign, qmin, qmax, &dec);
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Eq. 14 and the exhaustive FL search.                                       */
/* ------------------------------------------------------------------------- */
typedef int (*dyadic_at)(const void* src, int64_t i, int64_t* m, int* e);

typedef struct {
  const float* x;
} f32_src;
typedef struct {
  const int64_t* v;
  int s;
} i64_src;

static int f32_at(const void* src, int64_t i, int64_t* m, int* e) {
  return f32_to_dyadic(((const f32_src*)src)->x[i], m, e);
}
static int i64_at(const void* src, int64_t i, int64_t* m, int* e) {
  const i64_src* p = (const i64_src*)src;
  *m = p->v[i];
  *e = -p->s;
  return ORC_OK;
}

/* Exact Eq. 14 for every fl in [fl_lo, fl_hi] into acc[0..nfl). */
static int sse_all(const void* src, dyadic_at at, int64_t n, int k, int sign, int fl_lo, int fl_hi,
                   kacc* acc) {
  int nfl = fl_hi - fl_lo + 1;
  int64_t qmin, qmax;
  orc_qrange(k, sign, &qmin, &qmax);
  for (int j = 0; j < nfl; ++j) ka_zero(&acc[j]);
  int status = ORC_OK;
#pragma omp parallel
  {
    kacc* local = (kacc*)calloc((size_t)nfl, sizeof(kacc));
    int st = local ? ORC_OK : ORC_EINVAL;
#pragma omp for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
      if (st) continue;
      int64_t m;
      int e;
      if (at(src, i, &m, &e)) {
        st = ORC_EINVAL;
        continue;
      }
      for (int j = 0; j < nfl && !st; ++j) {
        int fl = fl_lo + j;
        int64_t dec;
        quant_dyadic(m, e, k, fl, sign, qmin, qmax, &dec);
        st = add_sq_error(&local[j], m, e, dec, fl);
      }
    }
#pragma omp critical
    {
      if (st && !status) status = st;
      if (local)
        for (int j = 0; j < nfl; ++j) ka_merge(&acc[j], &local[j]);
    }
    free(local);
  }
  return status;
}

int orc_sse_f32(const float* x, int64_t n, int k, int fl, int sign, double* sse) {
  if (check_fmt(k, sign) || n < 0) return ORC_EINVAL;
  f32_src s = {x};
  kacc acc;
  int st = sse_all(&s, f32_at, n, k, sign, fl, fl, &acc);
  if (st) return st;
  *sse = ka_to_double(&acc);
  return ORC_OK;
}

int orc_sse_i64(const int64_t* v, int64_t n, int s, int k, int fl, int sign, double* sse) {
  if (check_fmt(k, sign) || n < 0) return ORC_EINVAL;
  i64_src src = {v, s};
  kacc acc;
  int st = sse_all(&src, i64_at, n, k, sign, fl, fl, &acc);
  if (st) return st;
  *sse = ka_to_double(&acc);
  return ORC_OK;
}

static int fl_search(const void* src, dyadic_at at, int64_t n, int k, int sign, int fl_lo, int fl_hi,
                     int* fl_best, double* sse) {
  int nfl = fl_hi - fl_lo + 1;
  kacc* acc = (kacc*)malloc(sizeof(kacc) * (size_t)nfl);
  if (!acc) return ORC_EINVAL;
  int st = sse_all(src, at, n, k, sign, fl_lo, fl_hi, acc);
  if (!st) {
    int best = 0;
    for (int j = 1; j < nfl; ++j)
      if (ka_cmp(&acc[j], &acc[best]) <= 0) best = j; /* ties -> larger fl */
    *fl_best = fl_lo + best;
    if (sse)
      for (int j = 0; j < nfl; ++j) sse[j] = ka_to_double(&acc[j]);
  }
  free(acc);
  return st;
}

int orc_fl_search_f32(const float* x, int64_t n, int k, int sign, int fl_lo, int fl_hi,
                      int* fl_best, int* sign_used, double* sse) {
  if (n < 1 || fl_lo > fl_hi || k < 1 || k > 32) return ORC_EINVAL;
  for (int64_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) return ORC_EINVAL;
  if (sign == ORC_SIGN_AUTO) sign = orc_sign_f32(x, n);
  if (check_fmt(k, sign)) return ORC_EINVAL;
  if (sign_used) *sign_used = sign;
  f32_src s = {x};
  return fl_search(&s, f32_at, n, k, sign, fl_lo, fl_hi, fl_best, sse);
}

int orc_fl_search_i64(const int64_t* v, int64_t n, int s, int k, int sign, int fl_lo, int fl_hi,
                      int* fl_best, int* sign_used, double* sse) {
  if (n < 1 || fl_lo > fl_hi || k < 1 || k > 32) return ORC_EINVAL;
  if (sign == ORC_SIGN_AUTO) sign = orc_sign_i64(v, n);
  if (check_fmt(k, sign)) return ORC_EINVAL;
  if (sign_used) *sign_used = sign;
  i64_src src = {v, s};
  return fl_search(&src, i64_at, n, k, sign, fl_lo, fl_hi, fl_best, sse);
}

/* ------------------------------------------------------------------------- */
/* Integer contraction and convolution.                                       */
/* ------------------------------------------------------------------------- */
/* The sum s as int64, or ORC_ERANGE. */
static int fit_i64(i128 s, int64_t* out) {
  if (s > (i128)INT64_MAX || s < (i128)INT64_MIN) return ORC_ERANGE;
  *out = (int64_t)s;
  return ORC_OK;
}

int orc_gemm(const int64_t* A, const int64_t* B, int64_t M, int64_t N, int64_t K, int64_t* C) {
  if (M < 0 || N < 0 || K < 0) return ORC_EINVAL;
  int status = ORC_OK;
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m)
    for (int64_t n = 0; n < N; ++n) {
      i128 s = 0;
      for (int64_t k = 0; k < K; ++k) s += (i128)A[m * K + k] * (i128)B[n * K + k];
      if (fit_i64(s, &C[m * N + n])) {
#pragma omp atomic write
        status = ORC_ERANGE;
      }
    }
  return status;
}

int orc_conv2d_point(const int64_t* x, int N, int C, int H, int W, const int64_t* w, int K,
                     int R, int S, int stride, int pad, int n, int k, int oh, int ow, int64_t* y) {
  (void)N;
  (void)K;
  i128 s = 0;
  for (int c = 0; c < C; ++c)
    for (int r = 0; r < R; ++r) {
      int ih = oh * stride - pad + r;
      if (ih < 0 || ih >= H) continue;
      for (int q = 0; q < S; ++q) {
        int iw = ow * stride - pad + q;
        if (iw < 0 || iw >= W) continue;
        s += (i128)x[(((int64_t)n * C + c) * H + ih) * W + iw] *
             (i128)w[(((int64_t)k * C + c) * R + r) * S + q];
      }
    }
  return fit_i64(s, y);
}

int orc_conv2d(const int64_t* x, int N, int C, int H, int W, const int64_t* w, int K, int R,
               int S, int stride, int pad, int64_t* y) {
  if (stride < 1 || pad < 0) return ORC_EINVAL;
  int Ho = (H + 2 * pad - R) / stride + 1, Wo = (W + 2 * pad - S) / stride + 1;
  if (Ho < 1 || Wo < 1) return ORC_EINVAL;
  int status = ORC_OK;
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int k = 0; k < K; ++k)
      for (int oh = 0; oh < Ho; ++oh)
        for (int ow = 0; ow < Wo; ++ow)
          if (orc_conv2d_point(x, N, C, H, W, w, K, R, S, stride, pad, n, k, oh, ow,
                               &y[(((int64_t)n * K + k) * Ho + oh) * Wo + ow])) {
#pragma omp atomic write
            status = ORC_ERANGE;
          }
  return status;
}

/* ------------------------------------------------------------------------- */
/* C-Block epilogue, pools, eltwise.                                          */
/* ------------------------------------------------------------------------- */
static int fits62(i128 v) { return v < ((i128)1 << 62) && v > -((i128)1 << 62); }

/* (a at scale sa) + (b at scale sb), both aligned to max(sa, sb) by exact left shifts. */
static int align_add(i128 a, int sa, i128 b, int sb, i128* out, int* s_out) {
  int s = sa > sb ? sa : sb;
  if (s - sa > 62 || s - sb > 62) return ORC_ERANGE;
  i128 x = a * ((i128)1 << (s - sa));
  i128 y = b * ((i128)1 << (s - sb));
  if (!fits62(x) || !fits62(y)) return ORC_ERANGE;
  *out = x + y;
  *s_out = s;
  return ORC_OK;
}

int orc_epilogue(const int64_t* acc, int n_img, int channels, int64_t hw, int s_acc,
                 const int64_t* bias, int fl_b, const int64_t* a1, int fl_a1,
                 const int64_t* a2, int fl_a2, int relu, int64_t* v, int* s_out) {
  if (n_img < 0 || channels < 1 || hw < 0) return ORC_EINVAL;
  int s_final = s_acc;
  int st = ORC_OK;
  for (int64_t img = 0; img < n_img; ++img)
    for (int c = 0; c < channels; ++c)
      for (int64_t p = 0; p < hw; ++p) {
        int64_t idx = (img * channels + c) * hw + p;
        i128 x = acc[idx];
        int s = s_acc;
        if (bias) {
          st = align_add(x, s, bias[c], fl_b, &x, &s);
          if (st) return st;
        }
        if (a1) {
          x = x * (i128)a1[c];
          s = s + fl_a1;
          if (!fits62(x)) return ORC_ERANGE;
        }
        if (a2) {
          st = align_add(x, s, a2[c], fl_a2, &x, &s);
          if (st) return st;
        }
        if (relu && x < 0) x = 0;
        if (!fits62(x)) return ORC_ERANGE;
        v[idx] = (int64_t)x;
        s_final = s;
      }
  *s_out = s_final;
  if (n_img == 0 || hw == 0) { /* scale still defined by the parameters */
    int s = s_acc;
    if (bias) s = s > fl_b ? s : fl_b;
    if (a1) s += fl_a1;
    if (a2) s = s > fl_a2 ? s : fl_a2;
    *s_out = s;
  }
  return ORC_OK;
}

int orc_maxpool(const int32_t* x, int N, int C, int H, int W, int k, int stride, int pad,
                int32_t* y) {
  if (k < 1 || stride < 1 || pad < 0) return ORC_EINVAL;
  int Ho = (H + 2 * pad - k) / stride + 1, Wo = (W + 2 * pad - k) / stride + 1;
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int oh = 0; oh < Ho; ++oh)
        for (int ow = 0; ow < Wo; ++ow) {
          int have = 0;
          int32_t best = 0;
          for (int r = 0; r < k; ++r)
            for (int q = 0; q < k; ++q) {
              int ih = oh * stride - pad + r, iw = ow * stride - pad + q;
              if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
              int32_t val = x[(((int64_t)n * C + c) * H + ih) * W + iw];
              if (!have || val > best) best = val;
              have = 1;
            }
          y[(((int64_t)n * C + c) * Ho + oh) * Wo + ow] = best;
        }
  return ORC_OK;
}

int orc_avgpool_global(const int32_t* x, int N, int C, int HW, int64_t recip, int64_t* y) {
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c) {
      int64_t s = 0;
      for (int p = 0; p < HW; ++p) s += x[((int64_t)n * C + c) * HW + p];
      i128 t = (i128)s * recip;
      if (!fits62(t)) return ORC_ERANGE;
      y[(int64_t)n * C + c] = (int64_t)t;
    }
  return ORC_OK;
}

int orc_eltwise_add(const int32_t* a, int fa, const int32_t* b, int fb, int64_t n, int relu,
                    int64_t* v, int* s_out) {
  int s = fa > fb ? fa : fb;
  for (int64_t i = 0; i < n; ++i) {
    i128 x;
    int st = align_add(a[i], fa, b[i], fb, &x, &s);
    if (st) return st;
    if (relu && x < 0) x = 0;
    v[i] = (int64_t)x;
  }
  *s_out = s;
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Layer error.                                                               */
/* ------------------------------------------------------------------------- */
int orc_layer_error(const float* ref, const int32_t* codes, int64_t n, int k, int fl, int sign,
                    double out[4]) {
  if (n < 1 || check_fmt(k, sign)) return ORC_EINVAL;
  kacc acc;
  ka_zero(&acc);
  double mn = INFINITY, mx = -INFINITY, sum = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    int64_t m;
    int e;
    if (f32_to_dyadic(ref[i], &m, &e)) return ORC_EINVAL;
    int64_t dec = codes[i];
    if (k == 1 && sign == 1) dec = (codes[i] == 0) ? 1 : -1; /* Eq. 13 decoding */
    int st = add_sq_error(&acc, m, e, dec, fl);
    if (st) return st;
    double r = ref[i];
    if (r < mn) mn = r;
    if (r > mx) mx = r;
    sum += r;
  }
  double mean = sum / (double)n, var = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    double d = (double)ref[i] - mean;
    var += d * d;
  }
  out[0] = ka_to_double(&acc);
  out[1] = mn;
  out[2] = mx;
  out[3] = sqrt(var / (double)n);
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* FP32 teacher (reference activations of the sensitivity sweep).            */
/* ------------------------------------------------------------------------- */
int orc_teacher_conv2d(const float* x, int N, int C, int H, int W, const float* w, int K, int R,
                       int S, int stride, int pad, float* y) {
  if (stride < 1 || pad < 0) return ORC_EINVAL;
  int Ho = (H + 2 * pad - R) / stride + 1, Wo = (W + 2 * pad - S) / stride + 1;
  if (Ho < 1 || Wo < 1) return ORC_EINVAL;
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int k = 0; k < K; ++k)
      for (int oh = 0; oh < Ho; ++oh)
        for (int ow = 0; ow < Wo; ++ow) {
          double acc = 0.0;
          for (int r = 0; r < R; ++r) {
            int ih = oh * stride - pad + r;
            if (ih < 0 || ih >= H) continue;
            for (int q = 0; q < S; ++q) {
              int iw = ow * stride - pad + q;
              if (iw < 0 || iw >= W) continue;
              for (int c = 0; c < C; ++c) {
                double prod = (double)x[(((int64_t)n * C + c) * H + ih) * W + iw] *
                              (double)w[(((int64_t)k * C + c) * R + r) * S + q];
                acc = acc + prod;
              }
            }
          }
          y[(((int64_t)n * K + k) * Ho + oh) * Wo + ow] = (float)acc;
        }
  return ORC_OK;
}

int orc_teacher_affine(const float* t, int N, int C, int64_t hw, const float* a1,
                       const float* a2, const float* bias, int relu, float* y) {
  if (N < 0 || C < 1 || hw < 0 || (a1 && !a2)) return ORC_EINVAL;
  for (int64_t n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int64_t p = 0; p < hw; ++p) {
        int64_t i = ((int64_t)n * C + c) * hw + p;
        float v = t[i];
        if (a1) v = fmaf(v, a1[c], a2[c]);
        else if (bias) v = v + bias[c];
        if (relu) v = v > 0.0f ? v : 0.0f;
        y[i] = v;
      }
  return ORC_OK;
}

int orc_teacher_avgpool(const float* x, int N, int C, int64_t hw, float* y) {
  if (N < 0 || C < 1 || hw < 1) return ORC_EINVAL;
  for (int64_t n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c) {
      double acc = 0.0;
      for (int64_t p = 0; p < hw; ++p) acc = acc + (double)x[((int64_t)n * C + c) * hw + p];
      y[(int64_t)n * C + c] = (float)(acc / (double)hw);
    }
  return ORC_OK;
}
