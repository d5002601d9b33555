/*
 * SpecQuant CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct fp64 implementation of what the SpecQuant
 * hot path computes.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark may load this library; the product path never does.
 * It shares no source, header, table or helper with the HIP library.
 *
 * Paper: "SpecQuant -- Speculative Decoding with Multi-Parent Quantization for
 * Adaptive LLM Inference" (arXiv 2609.21704).
 *
 *   sqo_quantize_int4_g128  -- Q4 = f(W16, 4), SS III-A.1.  The paper gives no
 *                              formula; reading: asymmetric round-to-nearest
 *                              with one fp16 scale and one integer zero per 128
 *                              consecutive K elements of a row, range widened
 *                              to include 0, scale rounded up to fp16.
 *   sqo_quantize_fp8_e4m3   -- Q8 = f(W16, 8), SS III-A.2.  Reading: OCP E4M3
 *                              (bias 7, max 448, no infinities), one fp32 scale
 *                              per output row = amax/448, RNE, saturating.
 *   sqo_qgemv_w4a16 / sqo_qgemv_w8a16 / sqo_gemm_f16
 *                           -- draft pass (SS III-D.2) on the quantized parents
 *                              and the parent verification pass (SS III-D.3) on
 *                              Q16 = W16 (SS III-A.3): y = x . W'^T in fp64.
 *   sqo_softmax             -- LM-head distribution softmax(l / T).
 *   sqo_spec_accept         -- token acceptance or correction (SS III-D.4 and
 *                              the guess-set rule of SS III-A): the standard
 *                              speculative-sampling rule accept iff
 *                              u * q(x) < p(x), residual max(0, p - q)
 *                              renormalised at the first rejection, a bonus
 *                              draw from p when every draft is accepted; the
 *                              greedy "parent agrees" rule at T = 0.  The
 *                              distributions are computed in fp64 and held in
 *                              fp32, the precision the call hands back; the
 *                              decisions and draws use those fp32 values.
 *   sqo_accept_probs        -- the same decisions and draws taken directly from
 *                              given fp32 distributions.
 *
 * Every floating-point step is fp64 with IEEE division and round-to-nearest-
 * even, compiled without contraction (-ffp-contract=off).  Parallelism is an
 * OpenMP loop over independent output rows only; the order of every sum is the
 * plain ascending index order of its definition.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { SQO_OK = 0, SQO_ERR_NULL = 1, SQO_ERR_SHAPE = 2, SQO_ERR_NONFINITE = 5, SQO_ERR_VALUE = 6 };

int sqo_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the following calls (OpenMP over output rows); n >= 1.  Only
   the timing of the oracle changes: every output is one thread's fp64 sum in
   a fixed order whatever the count. */
void sqo_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ---------------------------------------------------------------- fp16 ---- */

/* IEEE binary16 bit pattern -> exact double. */
double sqo_f16_to_f64(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1F;
  int m = h & 0x3FF;
  double v;
  if (e == 0)
    v = ldexp((double)m, -24);
  else if (e == 31)
    v = (m == 0) ? INFINITY : NAN;
  else
    v = ldexp((double)(1024 + m), e - 25);
  return sign ? -v : v;
}

/* Bit pattern of a positive finite double that is exactly representable in
 * binary16 (normal or subnormal).  Returns 0xFFFF if it is not. */
static uint16_t f64_exact_to_f16(double v) {
  if (!(v > 0.0) || v > 65504.0) return 0xFFFF;
  if (v < ldexp(1.0, -14)) {              /* subnormal: v = m * 2^-24 */
    double m = ldexp(v, 24);
    if (m != floor(m)) return 0xFFFF;
    return (uint16_t)m;
  }
  int ex;
  double f = frexp(v, &ex);               /* v = f * 2^ex, f in [0.5, 1) */
  int e = ex - 1;                         /* v = (2f) * 2^e, 2f in [1, 2) */
  double mant = ldexp(2.0 * f - 1.0, 10); /* fraction field */
  if (mant != floor(mant)) return 0xFFFF;
  return (uint16_t)(((e + 15) << 10) | (int)mant);
}

/* Smallest binary16 value >= s, for finite s > 0.  Uses the binary16 grid
 * spacing 2^(e-10) (normal, e >= -14) or 2^-24 (subnormal); s / spacing is an
 * exact power-of-two scaling, so ceil() lands exactly on the grid. */
double sqo_f16_round_up(double s) {
  int ex;
  frexp(s, &ex);
  int e = ex - 1;                         /* 2^e <= s < 2^(e+1) */
  double spacing = (e < -14) ? ldexp(1.0, -24) : ldexp(1.0, e - 10);
  return ceil(s / spacing) * spacing;
}

/* ------------------------------------------------------------ INT4 g128 --- */

/* Q4 = f(W16, 4) (SS III-A.1).  w: [n][k] binary16 bits, k % 128 == 0.
 * codes: [n][k/2], element 2j in the low nibble of byte j, 2j+1 in the high.
 * scales, zeros: [n][k/128] binary16 bits.  Dequantized value: (q - z) * s. */
int sqo_quantize_int4_g128(const uint16_t* w, int64_t n, int64_t k, uint8_t* codes,
                           uint16_t* scales, uint16_t* zeros) {
  if (!w || !codes || !scales || !zeros) return SQO_ERR_NULL;
  if (n < 1 || k < 128 || k % 128 != 0) return SQO_ERR_SHAPE;
  const int64_t groups = k / 128;
  int status = SQO_OK;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t g = 0; g < groups; ++g) {
      const uint16_t* src = w + row * k + g * 128;
      double v[128];
      int bad = 0;
      for (int i = 0; i < 128; ++i) {
        v[i] = sqo_f16_to_f64(src[i]);
        if (!isfinite(v[i])) bad = 1;
      }
      uint8_t* dst = codes + row * (k / 2) + g * 64;
      if (bad) {                          /* defined output: codes 0, scale NaN */
        memset(dst, 0, 64);
        scales[row * groups + g] = 0x7E00;
        zeros[row * groups + g] = 0;
#pragma omp atomic write
        status = SQO_ERR_NONFINITE;
        continue;
      }
      double lo = 0.0, hi = 0.0;          /* range always contains zero */
      for (int i = 0; i < 128; ++i) {
        if (v[i] < lo) lo = v[i];
        if (v[i] > hi) hi = v[i];
      }
      double s16 = 1.0;
      double z = 0.0;
      int q[128];
      if (hi == lo) {                     /* all-zero group */
        for (int i = 0; i < 128; ++i) q[i] = 0;
      } else {
        double s = (hi - lo) / 15.0;
        s16 = sqo_f16_round_up(s);
        z = nearbyint(-lo / s16);
        if (z < 0.0) z = 0.0;
        if (z > 15.0) z = 15.0;
        for (int i = 0; i < 128; ++i) {
          double c = nearbyint(v[i] / s16) + z;
          if (c < 0.0) c = 0.0;
          if (c > 15.0) c = 15.0;
          q[i] = (int)c;
        }
      }
      for (int j = 0; j < 64; ++j) dst[j] = (uint8_t)(q[2 * j] | (q[2 * j + 1] << 4));
      scales[row * groups + g] = f64_exact_to_f16(s16);
      zeros[row * groups + g] = (z == 0.0) ? 0 : f64_exact_to_f16(z);
    }
  }
  return status;
}

/* Dequantized INT4 weight w'[row][col] = (q - z) * s (exact in fp64). */
static double int4_weight(const uint8_t* codes, const uint16_t* scales, const uint16_t* zeros,
                          int64_t k, int64_t row, int64_t col) {
  uint8_t byte = codes[row * (k / 2) + col / 2];
  int q = (col & 1) ? (byte >> 4) : (byte & 15);
  int64_t gi = row * (k / 128) + col / 128;
  return ((double)q - sqo_f16_to_f64(zeros[gi])) * sqo_f16_to_f64(scales[gi]);
}

int sqo_dequant_int4(const uint8_t* codes, const uint16_t* scales, const uint16_t* zeros,
                     int64_t n, int64_t k, double* out) {
  if (!codes || !scales || !zeros || !out) return SQO_ERR_NULL;
  if (n < 1 || k < 128 || k % 128 != 0) return SQO_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < n; ++row)
    for (int64_t col = 0; col < k; ++col) out[row * k + col] = int4_weight(codes, scales, zeros, k, row, col);
  return SQO_OK;
}

/* ------------------------------------------------------------- FP8 E4M3 --- */

/* OCP E4M3 code -> value: S.EEEE.MMM, bias 7; E = 0 subnormal; S.1111.111 NaN. */
double sqo_fp8_e4m3_decode(uint8_t c) {
  int sign = (c >> 7) & 1;
  int e = (c >> 3) & 15;
  int m = c & 7;
  double v;
  if (e == 15 && m == 7)
    return NAN;
  if (e == 0)
    v = ldexp((double)m / 8.0, -6);
  else
    v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return sign ? -v : v;
}

/* Round-to-nearest-even encode into OCP E4M3, saturating to +-448; the sign
 * of zero is kept. */
uint8_t sqo_fp8_e4m3_encode(double v) {
  uint8_t sign = signbit(v) ? 0x80 : 0x00;
  double a = fabs(v);
  int code;
  if (a > 448.0) {
    code = 0x7E;
  } else if (a < ldexp(1.0, -6)) {         /* subnormal grid: multiples of 2^-9 */
    code = (int)nearbyint(ldexp(a, 9));     /* 8 here is the smallest normal */
  } else {
    int ex;
    frexp(a, &ex);
    int e = ex - 1;                         /* 2^e <= a < 2^(e+1), e in [-6, 8] */
    double frac = ldexp(a, -e) - 1.0;       /* [0, 1), exact */
    int mant = (int)nearbyint(frac * 8.0);  /* 8 carries into the exponent */
    code = ((e + 7) << 3) + mant;
  }
  if (code > 0x7E) code = 0x7E;
  return (uint8_t)(sign | code);
}

/* Q8 = f(W16, 8) (SS III-A.2).  w: [n][k] binary16 bits.  codes: [n][k];
 * scales: [n] fp32 = amax/448 rounded once to fp32 (1.0 for an all-zero row).
 * Dequantized value: decode(c) * s. */
int sqo_quantize_fp8_e4m3(const uint16_t* w, int64_t n, int64_t k, uint8_t* codes, float* scales) {
  if (!w || !codes || !scales) return SQO_ERR_NULL;
  if (n < 1 || k < 1) return SQO_ERR_SHAPE;
  int status = SQO_OK;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < n; ++row) {
    const uint16_t* src = w + row * k;
    double amax = 0.0;
    int bad = 0;
    for (int64_t i = 0; i < k; ++i) {
      double v = sqo_f16_to_f64(src[i]);
      if (!isfinite(v)) bad = 1;
      else if (fabs(v) > amax) amax = fabs(v);
    }
    if (bad) {                            /* defined output: codes 0, scale NaN */
      memset(codes + row * k, 0, (size_t)k);
      scales[row] = NAN;
#pragma omp atomic write
      status = SQO_ERR_NONFINITE;
      continue;
    }
    float s = (amax == 0.0) ? 1.0f : (float)(amax / 448.0);
    scales[row] = s;
    for (int64_t i = 0; i < k; ++i) codes[row * k + i] = sqo_fp8_e4m3_encode(sqo_f16_to_f64(src[i]) / (double)s);
  }
  return status;
}

int sqo_dequant_fp8(const uint8_t* codes, const float* scales, int64_t n, int64_t k, double* out) {
  if (!codes || !scales || !out) return SQO_ERR_NULL;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < n; ++row)
    for (int64_t col = 0; col < k; ++col)
      out[row * k + col] = sqo_fp8_e4m3_decode(codes[row * k + col]) * (double)scales[row];
  return SQO_OK;
}

/* ---------------------------------------------------- GEMV and GEMM ------ */
/* y[i][j] = sum_c x[i][c] * W'[j][c] (ascending c), and the normaliser
 * d[i][j] = sum_c |x[i][c] * W'[j][c]|.  x: [m][k] binary16 bits.  Every
 * product below is exact in fp64. */

int sqo_qgemv_w4a16(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes,
                    const uint16_t* scales, const uint16_t* zeros, int64_t n, double* y, double* d) {
  if (!x || !codes || !scales || !zeros || !y) return SQO_ERR_NULL;
  if (m < 1 || n < 1 || k < 128 || k % 128 != 0) return SQO_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    for (int64_t i = 0; i < m; ++i) {
      double acc = 0.0, mag = 0.0;
      for (int64_t c = 0; c < k; ++c) {
        double t = sqo_f16_to_f64(x[i * k + c]) * int4_weight(codes, scales, zeros, k, j, c);
        acc += t;
        mag += fabs(t);
      }
      y[i * n + j] = acc;
      if (d) d[i * n + j] = mag;
    }
  }
  return SQO_OK;
}

int sqo_qgemv_w8a16(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes, const float* scales,
                    int64_t n, double* y, double* d) {
  if (!x || !codes || !scales || !y) return SQO_ERR_NULL;
  if (m < 1 || n < 1 || k < 1) return SQO_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    for (int64_t i = 0; i < m; ++i) {
      double acc = 0.0, mag = 0.0;
      for (int64_t c = 0; c < k; ++c) {
        double wv = sqo_fp8_e4m3_decode(codes[j * k + c]) * (double)scales[j];
        double t = sqo_f16_to_f64(x[i * k + c]) * wv;
        acc += t;
        mag += fabs(t);
      }
      y[i * n + j] = acc;
      if (d) d[i * n + j] = mag;
    }
  }
  return SQO_OK;
}

int sqo_gemm_f16(const uint16_t* x, int64_t m, int64_t k, const uint16_t* w, int64_t n, double* y, double* d) {
  if (!x || !w || !y) return SQO_ERR_NULL;
  if (m < 1 || n < 1 || k < 1) return SQO_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    for (int64_t i = 0; i < m; ++i) {
      double acc = 0.0, mag = 0.0;
      for (int64_t c = 0; c < k; ++c) {
        double t = sqo_f16_to_f64(x[i * k + c]) * sqo_f16_to_f64(w[j * k + c]);
        acc += t;
        mag += fabs(t);
      }
      y[i * n + j] = acc;
      if (d) d[i * n + j] = mag;
    }
  }
  return SQO_OK;
}

/* ------------------------------------------------------------- softmax --- */

/* One row: p_j = exp(z_j - L) / sum_i exp(z_i - L), z = l / T, L = max z.
 * A logit of -inf is a masked token: z = -inf, p = 0.  A row that holds a NaN
 * or +inf logit, or no finite logit at all, has no distribution: the function
 * returns 0 and sets every p_j to NaN.  Returns 1 for a valid row.  (For a
 * finite fp32 logit and a finite fp32 T > 0, |z| < 2^280, so z is finite.) */
static int softmax_row(const float* l, int64_t v, double temp, double* p) {
  int finite = 0;
  for (int64_t j = 0; j < v; ++j) {
    if (isnan(l[j]) || l[j] == INFINITY) finite = -1;
    if (finite == 0 && isfinite(l[j])) finite = 1;
  }
  if (finite != 1) {
    for (int64_t j = 0; j < v; ++j) p[j] = NAN;
    return 0;
  }
  double L = -INFINITY;
  for (int64_t j = 0; j < v; ++j) {
    double z = (double)l[j] / temp;
    if (z > L) L = z;
  }
  double sum = 0.0;
  for (int64_t j = 0; j < v; ++j) sum += exp((double)l[j] / temp - L);
  for (int64_t j = 0; j < v; ++j) p[j] = exp((double)l[j] / temp - L) / sum;
  return 1;
}

int sqo_softmax(const float* logits, int64_t rows, int64_t v, double temperature, double* p) {
  if (!logits || !p) return SQO_ERR_NULL;
  if (rows < 1 || v < 1) return SQO_ERR_SHAPE;
  if (!(temperature > 0.0) || !isfinite(temperature)) return SQO_ERR_VALUE;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) softmax_row(logits + r * v, v, temperature, p + r * v);
  return SQO_OK;
}

/* ------------------------------------------------------ accept / resample --- */

/* Greedy target of a row: the index of its largest logit, the smallest index
 * on ties.  A row holding a NaN or +inf logit, or no finite logit, has none:
 * returns -1. */
static int64_t argmax_row(const float* l, int64_t v) {
  int64_t best = -1;
  for (int64_t j = 0; j < v; ++j) {
    if (isnan(l[j]) || l[j] == INFINITY) return -1;
    if (isfinite(l[j]) && (best < 0 || l[j] > l[best])) best = j; /* strict: ties keep the smallest */
  }
  return best;
}

/* Inverse-CDF draw from weights r[0..v) >= 0 with the 24-bit uniform u24.
 * Each weight is put on the fixed-point grid R = rint(r * 2^60); the draw is
 * the smallest j whose running sum exceeds t = floor(u24 * Z / 2^24),
 * Z = sum R.  Returns -1 when Z == 0. */
static int64_t draw_fixed_point(const double* r, int64_t v, uint32_t u24) {
  int64_t* R = (int64_t*)malloc((size_t)v * sizeof(int64_t));
  int64_t Z = 0;
  for (int64_t j = 0; j < v; ++j) {
    R[j] = llrint(ldexp(r[j], 60));
    Z += R[j];
  }
  int64_t tok = -1;
  if (Z > 0) {
    unsigned __int128 prod = (unsigned __int128)(uint64_t)(u24 & 0xFFFFFFu) * (unsigned __int128)(uint64_t)Z;
    int64_t t = (int64_t)(prod >> 24);
    int64_t run = 0;
    for (int64_t j = 0; j < v; ++j) {
      run += R[j];
      if (run > t) {
        tok = j;
        break;
      }
    }
  }
  free(R);
  return tok;
}

/* Acceptance or correction of one sequence from its distributions held in
 * fp32 (SS III-D.4; the standard speculative-sampling rule):
 *   p[i] (i = 0..kd) the parent's rows, q[i] (i < kd) the draft's rows, each
 *   v probabilities; x[i * xs] the drafted token of position i; u[i] the
 *   24-bit uniforms, u[kd] driving the final draw.
 * Position i is accepted iff u_i * q_i(x_i) < p_i(x_i) with u_i = u[i] / 2^24,
 * formed in fp64 from the fp32 values (a 24-bit u times a 24-bit q is exact);
 * a token outside [0, v) is rejected.  n = the first rejection (kd if none).
 * At a rejection the token is drawn from max(0, p_n - q_n), each difference
 * formed in fp64 from the fp32 values, and from p_n itself when that mass is
 * zero on the grid; when all kd are accepted the bonus token is drawn from
 * p_kd.  A row holding a NaN makes the sequence invalid: n = token = -1. */
static void accept_from_rows(const float* const* p, const float* const* q, const int32_t* x, int64_t xs,
                             const uint32_t* u, int32_t kd, int64_t v, int32_t* n_out, int32_t* tok_out) {
  for (int32_t i = 0; i <= kd; ++i)
    for (int64_t j = 0; j < v; ++j)
      if (isnan(p[i][j]) || (i < kd && isnan(q[i][j]))) {
        *n_out = -1;
        *tok_out = -1;
        return;
      }
  int32_t n = kd;
  for (int32_t i = 0; i < kd; ++i) {
    int32_t xi = x[(int64_t)i * xs];
    double ui = ldexp((double)(u[i] & 0xFFFFFFu), -24);
    int accept = 0;
    if (xi >= 0 && xi < v) accept = (ui * (double)q[i][xi] < (double)p[i][xi]);
    if (!accept) {
      n = i;
      break;
    }
  }
  double* r = (double*)calloc((size_t)v, sizeof(double));
  int64_t tok;
  if (n < kd) {
    for (int64_t j = 0; j < v; ++j) {
      double diff = (double)p[n][j] - (double)q[n][j];
      r[j] = diff > 0.0 ? diff : 0.0;
    }
    tok = draw_fixed_point(r, v, u[kd]);
    if (tok < 0) { /* no residual mass on the grid: draw from p_n */
      for (int64_t j = 0; j < v; ++j) r[j] = (double)p[n][j];
      tok = draw_fixed_point(r, v, u[kd]);
    }
  } else {
    for (int64_t j = 0; j < v; ++j) r[j] = (double)p[kd][j];
    tok = draw_fixed_point(r, v, u[kd]);
  }
  free(r);
  *n_out = n;
  *tok_out = (int32_t)tok;
}

/* The decisions and draws of sqo_spec_accept (T > 0) taken directly from fp32
 * distributions in the call's own layouts: p [b][kd+1][v], q [kd][b][v],
 * draft_tokens [kd][b], u24 [b][kd+1].  Each row is a distribution (its
 * values sum to at most 1 + 2^-20). */
int sqo_accept_probs(const float* p, const float* q, const int32_t* draft_tokens, const uint32_t* u24, int32_t b,
                     int32_t kd, int32_t v, int32_t* n_accepted, int32_t* next_token) {
  if (!p || !u24 || !n_accepted || !next_token) return SQO_ERR_NULL;
  if (kd > 0 && (!q || !draft_tokens)) return SQO_ERR_NULL;
  if (b < 1 || kd < 0 || v < 1) return SQO_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int32_t s = 0; s < b; ++s) {
    const float** prow = (const float**)malloc((size_t)(kd + 1) * sizeof(float*));
    const float** qrow = (const float**)malloc((size_t)(kd > 0 ? kd : 1) * sizeof(float*));
    for (int32_t i = 0; i <= kd; ++i) prow[i] = p + ((int64_t)s * (kd + 1) + i) * v;
    for (int32_t i = 0; i < kd; ++i) qrow[i] = q + ((int64_t)i * b + s) * v;
    accept_from_rows(prow, qrow, draft_tokens ? draft_tokens + s : NULL, b, u24 + (int64_t)s * (kd + 1), kd, v,
                     n_accepted + s, next_token + s);
    free(prow);
    free(qrow);
  }
  return SQO_OK;
}

/* Speculative acceptance for b sequences with kd drafted tokens each.
 *   draft_logits  [kd][b][v]    (position-major: one draft step for all b)
 *   target_logits [b][kd+1][v]  (sequence-major: the parent's verify rows)
 *   draft_tokens  [kd][b] (position-major), u24 [b][kd+1] (low 24 bits used)
 * T > 0: p_i = softmax(target_i / T) and q_i = softmax(draft_i / T) in fp64,
 * each rounded once to fp32; then the rule of accept_from_rows on those fp32
 * values.  A row with no distribution (softmax_row) makes its sequence
 * invalid: n = token = -1.
 * T = 0: accept iff x_i == argmax p_i (smallest index on ties); the emitted
 * token is argmax of the first disagreeing row, or of row kd; a target row
 * without a greedy target (argmax_row) makes the sequence invalid.
 * q_out [kd][b][v] and p_out [b][kd+1][v] (optional, T > 0 only) receive the
 * fp64 distributions (NaN rows for rows without one). */
int sqo_spec_accept(const float* draft_logits, const float* target_logits, const int32_t* draft_tokens,
                    const uint32_t* u24, int32_t b, int32_t kd, int32_t v, double temperature,
                    int32_t* n_accepted, int32_t* next_token, double* q_out, double* p_out) {
  if (!target_logits || !n_accepted || !next_token) return SQO_ERR_NULL;
  if (kd > 0 && (!draft_logits || !draft_tokens)) return SQO_ERR_NULL;
  if (b < 1 || kd < 0 || v < 1) return SQO_ERR_SHAPE;
  if (!(temperature >= 0.0) || !isfinite(temperature)) return SQO_ERR_VALUE;
  if (temperature == 0.0 && (q_out || p_out)) return SQO_ERR_VALUE;
  if (temperature > 0.0 && !u24) return SQO_ERR_NULL;

#pragma omp parallel for schedule(static)
  for (int32_t s = 0; s < b; ++s) {
    const float* tgt = target_logits + (int64_t)s * (kd + 1) * v;
    if (temperature == 0.0) {
      int valid = 1;
      for (int32_t i = 0; i <= kd; ++i)
        if (argmax_row(tgt + (int64_t)i * v, v) < 0) valid = 0;
      if (!valid) {
        n_accepted[s] = -1;
        next_token[s] = -1;
        continue;
      }
      int32_t n = kd;
      for (int32_t i = 0; i < kd; ++i) {
        int32_t x = draft_tokens[(int64_t)i * b + s];
        if (x < 0 || x >= v || (int64_t)x != argmax_row(tgt + (int64_t)i * v, v)) {
          n = i;
          break;
        }
      }
      n_accepted[s] = n;
      next_token[s] = (int32_t)argmax_row(tgt + (int64_t)n * v, v);
      continue;
    }
    const int64_t nq = kd > 0 ? kd : 1;
    double* p = (double*)malloc((size_t)(kd + 1) * v * sizeof(double));
    double* q = (double*)malloc((size_t)nq * v * sizeof(double));
    float* p32 = (float*)malloc((size_t)(kd + 1) * v * sizeof(float));
    float* q32 = (float*)malloc((size_t)nq * v * sizeof(float));
    const float** prow = (const float**)malloc((size_t)(kd + 1) * sizeof(float*));
    const float** qrow = (const float**)malloc((size_t)nq * sizeof(float*));
    for (int32_t i = 0; i <= kd; ++i) softmax_row(tgt + (int64_t)i * v, v, temperature, p + (int64_t)i * v);
    for (int32_t i = 0; i < kd; ++i)
      softmax_row(draft_logits + ((int64_t)i * b + s) * v, v, temperature, q + (int64_t)i * v);
    for (int64_t j = 0; j < (kd + 1) * (int64_t)v; ++j) p32[j] = (float)p[j];
    for (int64_t j = 0; j < kd * (int64_t)v; ++j) q32[j] = (float)q[j];
    for (int32_t i = 0; i <= kd; ++i) prow[i] = p32 + (int64_t)i * v;
    for (int32_t i = 0; i < kd; ++i) qrow[i] = q32 + (int64_t)i * v;
    accept_from_rows(prow, qrow, kd > 0 ? draft_tokens + s : NULL, b, u24 + (int64_t)s * (kd + 1), kd, v,
                     n_accepted + s, next_token + s);
    if (p_out) memcpy(p_out + (int64_t)s * (kd + 1) * v, p, (size_t)(kd + 1) * v * sizeof(double));
    if (q_out)
      for (int32_t i = 0; i < kd; ++i)
        memcpy(q_out + ((int64_t)i * b + s) * v, q + (int64_t)i * v, (size_t)v * sizeof(double));
    free(p);
    free(q);
    free(p32);
    free(q32);
    free(prow);
    free(qrow);
  }
  return SQO_OK;
}
