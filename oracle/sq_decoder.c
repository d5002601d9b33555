/*
 * SpecQuant CPU oracle, decoder-step operations -- TEST INFRASTRUCTURE ONLY.
 *
 * The transformer layer that surrounds the projections of a draft pass
 * (SS III-D.2) and of the verification pass (SS III-D.3).  The paper evaluates
 * Qwen2.5 models (SS IV) and describes neither the layer nor the cache; these
 * functions are the plain textbook definitions of the operations of that model
 * family (RMS normalisation, rotary position embedding with the half-split
 * pairing, causal grouped-query attention over a key/value cache, the
 * SiLU-gated product), written out in fp64 in the order of their definitions.
 * The restart after a rejection (SS III-D.4) keeps only the cache positions of
 * accepted tokens; that bookkeeping lives in the Python side of the oracle.
 *
 * Same rules as sq_oracle.c: fp64, IEEE division, no contraction, ascending
 * summation order, OpenMP only across independent output rows.  Shares no
 * code with the HIP library.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

enum { SQD_OK = 0, SQD_ERR_NULL = 1, SQD_ERR_SHAPE = 2, SQD_ERR_VALUE = 6 };

/* RMS normalisation of each row:
 *   y[i][j] = h[i][j] / sqrt(mean_j(h[i][j]^2) + eps) * w[j]
 * h [m][d], w [d] (already widened to fp64), y [m][d]. */
int sqo_rmsnorm(const double* h, int64_t m, int64_t d, const double* w, double eps, double* y) {
  if (!h || !w || !y) return SQD_ERR_NULL;
  if (m < 1 || d < 1 || !(eps >= 0.0)) return SQD_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < m; ++i) {
    double ss = 0.0;
    for (int64_t j = 0; j < d; ++j) ss += h[i * d + j] * h[i * d + j];
    const double rms = sqrt(ss / (double)d + eps);
    for (int64_t j = 0; j < d; ++j) y[i * d + j] = h[i * d + j] / rms * w[j];
  }
  return SQD_OK;
}

/* Rotary position embedding, in place, of x [n][heads][hd] (hd even), row i at
 * position pos[i] >= 0.  Element j < hd/2 of a head pairs with element
 * j + hd/2 and the pair turns by the angle a = pos * theta^(-2j/hd):
 *   (x_j, x_{j+hd/2}) <- (x_j cos a - x_{j+hd/2} sin a, x_{j+hd/2} cos a + x_j sin a) */
int sqo_rope(double* x, int64_t n, int64_t heads, int64_t hd, const int64_t* pos, double theta) {
  if (!x || !pos) return SQD_ERR_NULL;
  if (n < 1 || heads < 1 || hd < 2 || hd % 2 != 0 || !(theta > 1.0)) return SQD_ERR_SHAPE;
  const int64_t half = hd / 2;
  for (int64_t i = 0; i < n; ++i)
    if (pos[i] < 0) return SQD_ERR_VALUE;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    for (int64_t h = 0; h < heads; ++h) {
      double* v = x + (i * heads + h) * hd;
      for (int64_t j = 0; j < half; ++j) {
        const double a = (double)pos[i] * pow(theta, -2.0 * (double)j / (double)hd);
        const double c = cos(a), s = sin(a);
        const double x1 = v[j], x2 = v[j + half];
        v[j] = x1 * c - x2 * s;
        v[j + half] = x2 * c + x1 * s;
      }
    }
  }
  return SQD_OK;
}

/* Causal grouped-query attention of one sequence.
 * q [n][hq][hd]; kc, vc [hkv][len][hd] hold the keys and values of cache
 * positions 0 .. len-1; hq is a multiple of hkv and query head h reads kv head
 * h / (hq / hkv).  Row i sits at position pos[i] (0 <= pos[i] < len) and
 * attends to positions 0 .. pos[i]:
 *   s_t = (q . k_t) / sqrt(hd),  out = sum_t exp(s_t - max s) v_t / sum_t exp(s_t - max s). */
int sqo_attention(const double* q, int64_t n, int64_t hq, int64_t hkv, int64_t hd, const double* kc,
                  const double* vc, int64_t len, const int64_t* pos, double* out) {
  if (!q || !kc || !vc || !pos || !out) return SQD_ERR_NULL;
  if (n < 1 || hq < 1 || hkv < 1 || hq % hkv != 0 || hd < 1 || len < 1) return SQD_ERR_SHAPE;
  for (int64_t i = 0; i < n; ++i)
    if (pos[i] < 0 || pos[i] >= len) return SQD_ERR_VALUE;
  const int64_t group = hq / hkv;
  const double scale = 1.0 / sqrt((double)hd);
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t ih = 0; ih < n * hq; ++ih) {
    const int64_t i = ih / hq, h = ih % hq, g = h / group;
    const int64_t last = pos[i];
    double* s = (double*)malloc((size_t)(last + 1) * sizeof(double));
    if (!s) {
      bad |= 1;
      continue;
    }
    const double* qv = q + (i * hq + h) * hd;
    double mx = -INFINITY;
    for (int64_t t = 0; t <= last; ++t) {
      const double* kv = kc + (g * len + t) * hd;
      double dot = 0.0;
      for (int64_t c = 0; c < hd; ++c) dot += qv[c] * kv[c];
      s[t] = dot * scale;
      if (s[t] > mx) mx = s[t];
    }
    double z = 0.0;
    for (int64_t t = 0; t <= last; ++t) {
      s[t] = exp(s[t] - mx);
      z += s[t];
    }
    double* o = out + (i * hq + h) * hd;
    for (int64_t c = 0; c < hd; ++c) {
      double acc = 0.0;
      for (int64_t t = 0; t <= last; ++t) acc += s[t] * vc[(g * len + t) * hd + c];
      o[c] = acc / z;
    }
    free(s);
  }
  return bad ? SQD_ERR_VALUE : SQD_OK;
}

/* SiLU-gated product of the fused gate|up output gu [m][2 inter] (gate in
 * columns 0 .. inter-1, up in inter .. 2 inter - 1):
 *   out[i][j] = g / (1 + exp(-g)) * u,  g = gu[i][j], u = gu[i][inter + j]. */
int sqo_silu_mul(const double* gu, int64_t m, int64_t inter, double* out) {
  if (!gu || !out) return SQD_ERR_NULL;
  if (m < 1 || inter < 1) return SQD_ERR_SHAPE;
  for (int64_t i = 0; i < m; ++i)
    for (int64_t j = 0; j < inter; ++j) {
      const double g = gu[i * 2 * inter + j], u = gu[i * 2 * inter + inter + j];
      out[i * inter + j] = g / (1.0 + exp(-g)) * u;
    }
  return SQD_OK;
}
