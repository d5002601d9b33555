/*
 * SpecQuant CPU oracle, multi-candidate drafting -- TEST INFRASTRUCTURE ONLY.
 *
 * SS III-D.2 lets a draft variant produce many candidate tokens in one step
 * to parallelise drafting; the paper gives no verification rule for them.
 * Reading: each sequence drafts c independent chains of kd tokens with the
 * quantized parent (every chain samples its own tokens, so the candidates at
 * any node of the chains' common prefix tree are independent draws from the
 * draft distribution at that node), the FP16 parent verifies all chains in one
 * pass, and acceptance walks the tree with recursive rejection sampling, the
 * multi-candidate form of the standard speculative-sampling rule:
 *
 *   at a node with draft distribution q and parent distribution p, the alive
 *   chains' candidates x_1, x_2, ... (ascending chain index) are tested in
 *   turn against a residual r (r = p at first):
 *     accept x_m iff u_m * q(x_m) < r(x_m);
 *     on rejection r <- max(0, r - q) renormalised;
 *   an accepted x continues with the chains whose token here is x; when
 *   every alive candidate is rejected the emitted token is drawn from r;
 *   after kd accepted tokens the bonus token is drawn from p of the last node.
 * With one chain this is exactly the single-candidate rule of sq_oracle.c.
 *
 * Arithmetic (every step integer or exact, so that results are reproducible
 * bit for bit from the fp32 distributions): the first test is
 * u * q(x) < p(x) in fp64 (a 24-bit u times a 24-bit q is exact); the first
 * residual is R = rint(max(0, p - q) * 2^60) (the difference formed in fp64)
 * with total Z = sum R, or rint(p * 2^60) when that total is 0; later tests
 * are u * q(x) * Z < R(x), compared exactly in 128-bit integers; later
 * residuals are R(y) <- max(0, R(y) - floor(q(y) * Z)) (the product exact),
 * with the same fallback to p when the total reaches 0; draws are the
 * inverse-CDF on the integer weights, t = floor(u24 * Z / 2^24), the smallest
 * y whose running sum exceeds t.
 *
 * Shares no code with the HIP library.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { SQM_OK = 0, SQM_ERR_NULL = 1, SQM_ERR_SHAPE = 2, SQM_ERR_VALUE = 6 };

/* q = M * 2^E exactly, M an integer below 2^24 (q finite, >= 0). */
static void split_f32(float q, uint64_t* m, int* e) {
  if (q == 0.0f) {
    *m = 0;
    *e = 0;
    return;
  }
  int ex;
  double f = frexp((double)q, &ex); /* q = f 2^ex, f in [0.5, 1) */
  *m = (uint64_t)ldexp(f, 24);      /* exact: q has at most 24 significant bits */
  *e = ex - 24;
}

/* floor(q * Z) for fp32 q in [0, 1] and 0 <= Z < 2^62, exactly. */
static int64_t floor_qz(float q, int64_t z) {
  uint64_t m;
  int e;
  split_f32(q, &m, &e);
  if (m == 0 || z == 0) return 0;
  unsigned __int128 prod = (unsigned __int128)m * (unsigned __int128)(uint64_t)z;
  if (e >= 0) return (int64_t)(prod << e); /* q <= 1, so this is at most Z */
  int sh = -e;
  if (sh >= 128) return 0;
  return (int64_t)(prod >> sh);
}

/* u24 / 2^24 * q * Z < R, exactly. */
static int test_grid(uint32_t u24, float q, int64_t z, int64_t r) {
  uint64_t m;
  int e;
  split_f32(q, &m, &e);
  unsigned __int128 lhs = (unsigned __int128)((uint64_t)(u24 & 0xFFFFFFu) * m) * (unsigned __int128)(uint64_t)z;
  if (r <= 0) return 0;
  /* compare lhs * 2^e with r * 2^24, i.e. lhs with r * 2^(24 - e) */
  int sh = 24 - e;
  if (sh < 0) return lhs < ((unsigned __int128)(uint64_t)r >> (-sh)) ? 1 : 0; /* not reached for q <= 1 */
  int bits = 0;
  for (uint64_t t = (uint64_t)r; t; t >>= 1) ++bits;
  if (bits + sh >= 127) return 1; /* r * 2^sh >= 2^126 > lhs (lhs < 2^24 * 2^24 * 2^62) */
  unsigned __int128 rhs = (unsigned __int128)(uint64_t)r << sh;
  return lhs < rhs ? 1 : 0;
}

static int64_t draw_grid(const int64_t* R, int64_t v, int64_t z, uint32_t u24) {
  if (z <= 0) return -1;
  unsigned __int128 prod = (unsigned __int128)(uint64_t)(u24 & 0xFFFFFFu) * (unsigned __int128)(uint64_t)z;
  int64_t t = (int64_t)(prod >> 24);
  int64_t run = 0;
  for (int64_t y = 0; y < v; ++y) {
    run += R[y];
    if (run > t) return y;
  }
  return -1;
}

static int64_t grid_of_p(const float* p, int64_t v, int64_t* R) {
  int64_t z = 0;
  for (int64_t y = 0; y < v; ++y) {
    R[y] = llrint(ldexp((double)p[y], 60));
    z += R[y];
  }
  return z;
}

/* One sequence.  prow(j, d): parent row of chain j at depth d (d = 0..kd);
 * qrow(j, d): draft row of chain j at step d (d < kd); tok(j, d): chain j's
 * token at depth d; u[d * c + j] the test uniform of chain j at depth d,
 * u[kd * c] the final draw. */
typedef struct {
  const float* p;
  const float* q;
  const int32_t* drafts;
  int32_t b, c, kd, s;
  int64_t v;
} MultiSeq;

static const float* mprow(const MultiSeq* m, int j, int d) {
  return m->p + (((int64_t)m->s * m->c + j) * (m->kd + 1) + d) * m->v;
}
static const float* mqrow(const MultiSeq* m, int j, int d) {
  return m->q + (((int64_t)d * m->b + m->s) * m->c + j) * m->v;
}
static int32_t mtok(const MultiSeq* m, int j, int d) {
  return m->drafts[((int64_t)d * m->b + m->s) * m->c + j];
}

static void multi_accept_seq(const MultiSeq* m, const uint32_t* u, int32_t* n_out, int32_t* tok_out,
                             int32_t* chain_out) {
  const int64_t v = m->v;
  const int c = m->c, kd = m->kd;
  /* a NaN in any row of the sequence: no distribution */
  for (int j = 0; j < c; ++j)
    for (int d = 0; d <= kd; ++d) {
      const float* pr = mprow(m, j, d);
      const float* qr = d < kd ? mqrow(m, j, d) : NULL;
      for (int64_t y = 0; y < v; ++y)
        if (isnan(pr[y]) || (qr && isnan(qr[y]))) {
          *n_out = *tok_out = *chain_out = -1;
          return;
        }
    }
  int64_t* R = (int64_t*)malloc((size_t)v * sizeof(int64_t));
  int alive[64];
  int nalive = c;
  for (int j = 0; j < c; ++j) alive[j] = j;
  int32_t n = kd, tok = -1;
  for (int d = 0; d < kd; ++d) {
    const float* p = mprow(m, alive[0], d);
    const float* q = mqrow(m, alive[0], d);
    int64_t z = 0;
    int accepted = -1;
    for (int a = 0; a < nalive; ++a) {
      const int j = alive[a];
      const int32_t x = mtok(m, j, d);
      const uint32_t uj = u[d * c + j];
      int acc = 0;
      if (x >= 0 && x < v) {
        if (a == 0)
          acc = ldexp((double)(uj & 0xFFFFFFu), -24) * (double)q[x] < (double)p[x];
        else
          acc = test_grid(uj, q[x], z, R[x]);
      }
      if (acc) {
        accepted = x;
        break;
      }
      if (a == 0) { /* first residual: max(0, p - q) on the grid */
        z = 0;
        for (int64_t y = 0; y < v; ++y) {
          const double diff = (double)p[y] - (double)q[y];
          R[y] = llrint(ldexp(diff > 0.0 ? diff : 0.0, 60));
          z += R[y];
        }
      } else {
        const int64_t z0 = z;
        z = 0;
        for (int64_t y = 0; y < v; ++y) {
          const int64_t t = R[y] - floor_qz(q[y], z0);
          R[y] = t > 0 ? t : 0;
          z += R[y];
        }
      }
      if (z == 0) z = grid_of_p(p, v, R); /* no residual mass on the grid: back to p */
    }
    if (accepted < 0) {
      n = d;
      tok = (int32_t)draw_grid(R, v, z, u[kd * c]);
      break;
    }
    int keep = 0;
    for (int a = 0; a < nalive; ++a)
      if (mtok(m, alive[a], d) == accepted) alive[keep++] = alive[a];
    nalive = keep;
  }
  if (n == kd) {
    const int64_t z = grid_of_p(mprow(m, alive[0], kd), v, R);
    tok = (int32_t)draw_grid(R, v, z, u[kd * c]);
  }
  free(R);
  *n_out = n;
  *tok_out = tok;
  *chain_out = alive[0];
}

/* Multi-candidate acceptance from fp32 distributions:
 *   p [b][c][kd+1][v] (chain j's verify rows), q [kd][b][c][v] (draft step d
 *   for all chains), drafts [kd][b][c], u24 [b][c kd + 1];
 *   out: n_accepted [b], next_token [b], chain [b] (the lowest chain whose
 *   first n tokens are the accepted ones).  1 <= c <= 64. */
int sqo_multi_accept_probs(const float* p, const float* q, const int32_t* drafts, const uint32_t* u24, int32_t b,
                           int32_t c, int32_t kd, int32_t v, int32_t* n_accepted, int32_t* next_token,
                           int32_t* chain) {
  if (!p || !u24 || !n_accepted || !next_token || !chain) return SQM_ERR_NULL;
  if (kd > 0 && (!q || !drafts)) return SQM_ERR_NULL;
  if (b < 1 || c < 1 || c > 64 || kd < 0 || v < 1) return SQM_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int32_t s = 0; s < b; ++s) {
    MultiSeq m = {p, q, drafts, b, c, kd, s, v};
    multi_accept_seq(&m, u24 + (int64_t)s * (c * kd + 1), n_accepted + s, next_token + s, chain + s);
  }
  return SQM_OK;
}

/* Greedy multi-candidate acceptance (T = 0) from the parent's logits
 * target [b][c][kd+1][v]: at each depth the argmax of the node's row (the
 * lowest alive chain's; smallest index on ties) is accepted when an alive
 * chain drafted it, and those chains continue; else it is the emitted token.
 * After kd accepted tokens the emitted token is the argmax of the last node.
 * A target row of the sequence (any chain, any depth) holding a NaN or +inf,
 * or no finite logit, makes the sequence invalid (n = token = chain = -1). */
int sqo_multi_accept_greedy(const float* target, const int32_t* drafts, int32_t b, int32_t c, int32_t kd,
                            int32_t v, int32_t* n_accepted, int32_t* next_token, int32_t* chain) {
  if (!target || !n_accepted || !next_token || !chain || (kd > 0 && !drafts)) return SQM_ERR_NULL;
  if (b < 1 || c < 1 || c > 64 || kd < 0 || v < 1) return SQM_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int32_t s = 0; s < b; ++s) {
    int alive[64], nalive = c, bad = 0;
    for (int j = 0; j < c; ++j) alive[j] = j;
    /* every target row of the sequence needs a greedy target */
    for (int64_t r = 0; r < (int64_t)c * (kd + 1) && !bad; ++r) {
      const float* row = target + ((int64_t)s * c * (kd + 1) + r) * v;
      int finite = 0;
      for (int64_t y = 0; y < v; ++y) {
        if (isnan(row[y]) || row[y] == INFINITY) bad = 1;
        if (isfinite(row[y])) finite = 1;
      }
      if (!finite) bad = 1;
    }
    int32_t n = kd, tok = -1;
    for (int d = 0; d <= kd && !bad; ++d) {
      const float* row = target + (((int64_t)s * c + alive[0]) * (kd + 1) + d) * v;
      int64_t best = -1;
      for (int64_t y = 0; y < v; ++y)
        if (isfinite(row[y]) && (best < 0 || row[y] > row[best])) best = y; /* strict: ties keep the smallest */
      if (d == kd) {
        tok = (int32_t)best;
        break;
      }
      int keep = 0;
      for (int a = 0; a < nalive; ++a)
        if (drafts[((int64_t)d * b + s) * c + alive[a]] == best) alive[keep++] = alive[a];
      if (keep == 0) {
        n = d;
        tok = (int32_t)best;
        break;
      }
      nalive = keep;
    }
    n_accepted[s] = bad ? -1 : n;
    next_token[s] = bad ? -1 : tok;
    chain[s] = bad ? -1 : alive[0];
  }
  return SQM_OK;
}
