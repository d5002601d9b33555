/* Drives every function of the CPU oracle (oracle/sq_oracle.c, test
 * infrastructure) on small inputs, edge cases included, under
 * AddressSanitizer and UndefinedBehaviorSanitizer: quantizers with zero,
 * one-hot, subnormal, extreme and non-finite groups; the GEMV/GEMM forms; the
 * softmax and the accept step with masked and invalid rows, kd = 0, v = 1,
 * greedy mode, and the decision core on given fp32 distributions. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int sqo_quantize_int4_g128(const uint16_t*, int64_t, int64_t, uint8_t*, uint16_t*, uint16_t*);
int sqo_dequant_int4(const uint8_t*, const uint16_t*, const uint16_t*, int64_t, int64_t, double*);
int sqo_quantize_fp8_e4m3(const uint16_t*, int64_t, int64_t, uint8_t*, float*);
int sqo_dequant_fp8(const uint8_t*, const float*, int64_t, int64_t, double*);
int sqo_qgemv_w4a16(const uint16_t*, int64_t, int64_t, const uint8_t*, const uint16_t*, const uint16_t*, int64_t,
                    double*, double*);
int sqo_qgemv_w8a16(const uint16_t*, int64_t, int64_t, const uint8_t*, const float*, int64_t, double*, double*);
int sqo_gemm_f16(const uint16_t*, int64_t, int64_t, const uint16_t*, int64_t, double*, double*);
int sqo_softmax(const float*, int64_t, int64_t, double, double*);
int sqo_spec_accept(const float*, const float*, const int32_t*, const uint32_t*, int32_t, int32_t, int32_t, double,
                    int32_t*, int32_t*, double*, double*);
int sqo_accept_probs(const float*, const float*, const int32_t*, const uint32_t*, int32_t, int32_t, int32_t, int32_t*,
                     int32_t*);
uint8_t sqo_fp8_e4m3_encode(double);
double sqo_fp8_e4m3_decode(uint8_t);
double sqo_f16_round_up(double);

static uint32_t rng = 12345u;
static uint32_t next(void) {
  rng = rng * 1664525u + 1013904223u;
  return rng >> 8;
}

int main(void) {
  int fails = 0;
  const int64_t n = 7, k = 384;
  uint16_t* w = malloc(n * k * 2);
  for (int64_t i = 0; i < n * k; ++i) w[i] = (uint16_t)(next() & 0x3FFF);  /* positive, finite, some subnormal */
  for (int64_t i = 0; i < k; ++i) w[i] = 0;                               /* zero row */
  w[k + 5] = 0x3C00;                                                      /* one-hot row */
  for (int64_t i = 2 * k; i < 3 * k; ++i) w[i] = (i & 1) ? 0x7BFF : 0xFBFF; /* +-65504 */
  uint8_t* c4 = malloc(n * k / 2);
  uint16_t* s4 = malloc(n * k / 128 * 2);
  uint16_t* z4 = malloc(n * k / 128 * 2);
  double* dq = malloc(n * k * 8);
  fails += sqo_quantize_int4_g128(w, n, k, c4, s4, z4) != 0;
  fails += sqo_dequant_int4(c4, s4, z4, n, k, dq) != 0;
  uint8_t* c8 = malloc(n * k);
  float* s8 = malloc(n * 4);
  fails += sqo_quantize_fp8_e4m3(w, n, k, c8, s8) != 0;
  fails += sqo_dequant_fp8(c8, s8, n, k, dq) != 0;
  w[3 * k + 7] = 0x7E00;  /* NaN: a non-finite group and row, reported */
  fails += sqo_quantize_int4_g128(w, n, k, c4, s4, z4) != 5;
  fails += sqo_quantize_fp8_e4m3(w, n, k, c8, s8) != 5;
  for (int c = 0; c < 256; ++c) (void)sqo_fp8_e4m3_decode((uint8_t)c);
  (void)sqo_fp8_e4m3_encode(-0.0);
  (void)sqo_fp8_e4m3_encode(1e30);
  (void)sqo_f16_round_up(1e-9);
  const int64_t m = 3;
  uint16_t* x = malloc(m * k * 2);
  for (int64_t i = 0; i < m * k; ++i) x[i] = (uint16_t)(0x3000 + (next() & 0xFFF));
  double* y = malloc(m * n * 8);
  double* d = malloc(m * n * 8);
  fails += sqo_qgemv_w4a16(x, m, k, c4, s4, z4, n, y, d) != 0;
  fails += sqo_qgemv_w8a16(x, m, k, c8, s8, n, y, NULL) != 0;
  fails += sqo_gemm_f16(x, m, k, w, n, y, d) != 0;
  /* accept: b = 4 sequences, kd = 3, v = 70; masked and invalid rows */
  const int b = 4, kd = 3, v = 70;
  float* dl = malloc((size_t)kd * b * v * 4);
  float* tl = malloc((size_t)b * (kd + 1) * v * 4);
  for (int i = 0; i < kd * b * v; ++i) dl[i] = (float)((int)(next() % 2000) - 1000) / 300.0f;
  for (int i = 0; i < b * (kd + 1) * v; ++i) tl[i] = (float)((int)(next() % 2000) - 1000) / 300.0f;
  for (int j = 0; j < v; ++j) tl[(1 * (kd + 1) + 2) * v + j] = -INFINITY; /* sequence 1: a fully masked row */
  tl[(2 * (kd + 1) + 0) * v + 9] = NAN;                                   /* sequence 2: a NaN */
  for (int j = 10; j < 40; ++j) tl[(3 * (kd + 1) + 1) * v + j] = -INFINITY;
  int32_t tok[3 * 4];
  uint32_t u24[4 * 4];
  for (int i = 0; i < kd * b; ++i) tok[i] = (int32_t)(next() % v);
  tok[0] = -1;
  tok[5] = v;
  for (int i = 0; i < b * (kd + 1); ++i) u24[i] = next() & 0xFFFFFF;
  int32_t na[4], nt[4];
  double* q = malloc((size_t)kd * b * v * 8);
  double* p = malloc((size_t)b * (kd + 1) * v * 8);
  fails += sqo_spec_accept(dl, tl, tok, u24, b, kd, v, 1.0, na, nt, q, p) != 0;
  fails += !(na[1] == -1 && nt[1] == -1 && na[2] == -1 && nt[2] == -1);
  float* q32 = malloc((size_t)kd * b * v * 4);
  float* p32 = malloc((size_t)b * (kd + 1) * v * 4);
  for (int i = 0; i < kd * b * v; ++i) q32[i] = (float)q[i];
  for (int i = 0; i < b * (kd + 1) * v; ++i) p32[i] = (float)p[i];
  int32_t na2[4], nt2[4];
  fails += sqo_accept_probs(p32, q32, tok, u24, b, kd, v, na2, nt2) != 0;
  fails += memcmp(na, na2, sizeof na) != 0 || memcmp(nt, nt2, sizeof nt) != 0;
  fails += sqo_spec_accept(dl, tl, tok, NULL, b, kd, v, 0.0, na, nt, NULL, NULL) != 0;  /* greedy */
  fails += sqo_spec_accept(NULL, tl, NULL, u24, b, 0, v, 0.7, na, nt, NULL, p) != 0;    /* kd = 0 */
  fails += sqo_spec_accept(dl, tl, tok, u24, b, kd, 1, 1.0, na, nt, NULL, NULL) != 0;   /* v = 1 */
  fails += sqo_softmax(tl, b * (kd + 1), v, 1.3, p) != 0;
  fails += sqo_spec_accept(dl, tl, tok, u24, b, kd, v, -1.0, na, nt, NULL, NULL) == 0;  /* rejected */
  free(w); free(c4); free(s4); free(z4); free(dq); free(c8); free(s8); free(x); free(y); free(d);
  free(dl); free(tl); free(q); free(p); free(q32); free(p32);
  printf(fails ? "FAILED %d\n" : "ORACLE OK\n", fails);
  return fails ? 1 : 0;
}
