/*
 * CPU oracle for the distribution-aware fused-MoE path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline of the benchmark load this library.  It shares no code with the
 * HIP path: plain loops, fp64 for floating point, no blocking, no fusion.
 *
 * Paper: "Decoding the Skew: Distribution-Aware MoE Inference with Adaptive
 * Kernel Dispatch" (DA-MoE).  Each function names the passage it follows.
 *
 * Integer results (histogram, Effective Experts numerator/denominator and
 * bucket, permutation, tile list, dispatch choice) are plain definitions.
 * The layer output is the plain definition of a top-k MoE layer with SwiGLU
 * experts, evaluated expert by expert in fp64 from the bf16 (or fp8 + scale)
 * inputs.  Alg. 1 and the exemplar construction follow the paper's steps.
 * The router (linear gate, top-k, softmax over the chosen logits) is the plain
 * definition of a top-k gate (Sec. II-A), evaluated in fp64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Routing statistics                                                         */
/* ------------------------------------------------------------------------- */

/* Per-expert token counts t_e = #{(t, j) : ids[t*k + j] == e}, the t_i of
 * Eq. (2) in Sec. III-A and the histogram of Sec. IV-B.  Ids outside [0, E)
 * are not counted; the return value is how many there were. */
int64_t oracle_histogram(const int32_t* ids, int64_t A, int32_t E, int64_t* counts) {
  int64_t bad = 0;
  for (int32_t e = 0; e < E; ++e) counts[e] = 0;
  for (int64_t a = 0; a < A; ++a) {
    if (ids[a] < 0 || ids[a] >= E) { ++bad; continue; }
    counts[ids[a]] += 1;
  }
  return bad;
}

/* Effective Experts, Eq. (2) of Sec. III-A:
 *   eff_exp = (sum_e t_e)^2 / sum_e t_e^2
 * returned as the exact integer pair (num, den) plus its fp64 value.
 * With no tokens num = den = 0 and eff = 0. */
void oracle_effexp(const int64_t* counts, int32_t E, uint64_t* num, uint64_t* den, double* eff) {
  uint64_t s = 0, s2 = 0;
  for (int32_t e = 0; e < E; ++e) {
    s += (uint64_t)counts[e];
    s2 += (uint64_t)counts[e] * (uint64_t)counts[e];
  }
  *num = s * s;
  *den = s2;
  *eff = s2 ? (double)(*num) / (double)(*den) : 0.0;
}

/* Skew multipliers X of the ddist:X parameterisation (Sec. III-A), as exact
 * fractions: the paper's tuning grid of Sec. V-A {1.1, 1.3, 1.5, 1.7, 2.0,
 * 2.5, 4.0} extended by {6, 8, 12, 16, 24, 32} to reach alpha near 0.03. */
static const uint64_t XN[13] = {11, 13, 3, 17, 2, 5, 4, 6, 8, 12, 16, 24, 32};
static const uint64_t XD[13] = {10, 10, 2, 10, 1, 2, 1, 1, 1, 1, 1, 1, 1};

/* Effective Experts bucket: the number of grid points X whose ddist:X target
 * E/X is at least eff_exp, i.e. #{j : eff_exp <= E / X_j}, decided exactly
 * as num * XN_j <= E * XD_j * den.  0 = near-uniform ... 13 = most skewed;
 * -1 when there are no tokens. */
int32_t oracle_effexp_bucket(uint64_t num, uint64_t den, int32_t E) {
  if (den == 0) return -1;
  int32_t b = 0;
  for (int j = 0; j < 13; ++j)
    if (num * XN[j] <= (uint64_t)E * XD[j] * den) ++b;
  return b;
}

/* Routing metadata: assignments grouped by expert.  offsets[e] is the first
 * position of expert e; perm[p] is the flat assignment index a = t*k + j at
 * position p, experts in increasing order and, within one expert, a in
 * increasing order; inv_perm[perm[p]] = p.  Ids outside [0, E) get
 * inv_perm = -1 and no position.  (Routing-metadata construction, Sec. V-C.) */
void oracle_permute(const int32_t* ids, int64_t A, int32_t E, int64_t* offsets, int64_t* perm,
                    int64_t* inv_perm) {
  int64_t p = 0;
  for (int64_t a = 0; a < A; ++a) inv_perm[a] = -1;
  for (int32_t e = 0; e < E; ++e) {
    offsets[e] = p;
    for (int64_t a = 0; a < A; ++a) {
      if (ids[a] == e) {
        perm[p] = a;
        inv_perm[a] = p;
        ++p;
      }
    }
  }
  offsets[E] = p;
}

/* ------------------------------------------------------------------------- */
/* Online dispatch (Sec. IV, IV-B)                                            */
/* ------------------------------------------------------------------------- */

/* Token-count bucket: the smallest tuned bucket size that is >= T, or the
 * last one when T exceeds them all (Sec. IV: the bucket for the current
 * token count is chosen first).  bucket_T is ascending. */
int32_t oracle_select_bucket(const int32_t* bucket_T, int32_t nb, int32_t T) {
  for (int32_t b = 0; b < nb; ++b)
    if (T <= bucket_T[b]) return b;
  return nb - 1;
}

static int cmp_desc_i64(const void* x, const void* y) {
  const int64_t a = *(const int64_t*)x, b = *(const int64_t*)y;
  return (a < b) - (a > b);
}

/* Exemplar match of Sec. IV-B: the histogram sorted in descending order is
 * scored against every exemplar of the bucket by a dot product (the cosine
 * similarity up to the query's norm, which does not change the argmax).
 * Exemplars are unit vectors quantised as Q = round(u * 2^15), so the score
 * is the exact integer sum_r sorted[r] * Q[i][r].  Returns the first index
 * with the highest score; scores[] receives every score. */
int32_t oracle_match(const int64_t* counts, int32_t E, const int32_t* Q, int32_t n_ex,
                     int64_t* scores) {
  int64_t* s = (int64_t*)malloc(sizeof(int64_t) * (size_t)(E > 0 ? E : 1));
  memcpy(s, counts, sizeof(int64_t) * (size_t)E);
  qsort(s, (size_t)E, sizeof(int64_t), cmp_desc_i64);
  int32_t best = -1;
  int64_t best_score = 0;
  for (int32_t i = 0; i < n_ex; ++i) {
    int64_t acc = 0;
    for (int32_t r = 0; r < E; ++r) acc += s[r] * (int64_t)Q[(int64_t)i * E + r];
    scores[i] = acc;
    if (best < 0 || acc > best_score) {
      best = i;
      best_score = acc;
    }
  }
  free(s);
  return best;
}

/* Token tiles of one tile size BM (the Tile-N of Sec. II-C): for every expert
 * e in increasing order, ceil(t_e / BM) tiles; tile j of expert e starts at
 * position offsets[e] + j*BM and has min(BM, t_e - j*BM) rows.  Writes
 * (start, expert, rows) triples and returns the number of tiles. */
int64_t oracle_tiles(const int64_t* counts, int32_t E, int32_t BM, int64_t* out) {
  int64_t n = 0, p = 0;
  for (int32_t e = 0; e < E; ++e) {
    for (int64_t r = 0; r < counts[e]; r += BM) {
      out[3 * n + 0] = p + r;
      out[3 * n + 1] = e;
      out[3 * n + 2] = (counts[e] - r < BM) ? counts[e] - r : BM;
      ++n;
    }
    p += counts[e];
  }
  return n;
}

/* ------------------------------------------------------------------------- */
/* The MoE layer (Sec. II-A, fused over experts as in Sec. II-C)              */
/* ------------------------------------------------------------------------- */

static double bf16_value(uint16_t h) {
  union { uint32_t u; float f; } v;
  v.u = (uint32_t)h << 16;
  return (double)v.f;
}

/* OCP e4m3fn: 1 sign, 4 exponent (bias 7), 3 mantissa bits; exponent 0 is
 * subnormal (mant * 2^-9); 0x7F / 0xFF are NaN. */
static double e4m3_value(uint8_t q) {
  const int sign = q >> 7, ex = (q >> 3) & 15, man = q & 7;
  double v;
  if (ex == 15 && man == 7) return NAN;
  if (ex == 0) v = man * ldexp(1.0, -9);
  else v = (1.0 + man / 8.0) * ldexp(1.0, ex - 7);
  return sign ? -v : v;
}

/* OCP MX FP4 (e2m1): 1 sign, 2 exponent (bias 1), 1 mantissa bit; exponent 0 is
 * subnormal (mant * 0.5).  Magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6. */
static double e2m1_value(uint8_t c) {
  const int sign = (c >> 3) & 1, ex = (c >> 1) & 3, man = c & 1;
  const double v = ex == 0 ? 0.5 * man : (1.0 + 0.5 * man) * ldexp(1.0, ex - 1);
  return sign ? -v : v;
}

/* OCP MX E8M0 block scale: 2^(s - 127); 255 is NaN. */
static double e8m0_value(uint8_t s) { return s == 255 ? NAN : ldexp(1.0, (int)s - 127); }

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* Weight element (row i, column c) of a [rows][cols] expert matrix: bf16; fp8 e4m3 with
 * one fp32 scale per 128x128 block; or MXFP4 (two e2m1 codes per byte, the even column in
 * the low nibble, [rows][cols / 2]) with one E8M0 scale per 32 consecutive columns of a row
 * ([rows][cols / 32]). */
typedef struct {
  const uint16_t* bf16;
  const uint8_t* q;
  const float* s;
  int32_t cols;
  const uint8_t* q4;
  const uint8_t* s4;
} wmat;

static double wval(const wmat* m, int64_t i, int64_t c) {
  if (m->bf16) return bf16_value(m->bf16[i * m->cols + c]);
  if (m->q4) {
    const uint8_t byte = m->q4[i * (m->cols / 2) + c / 2];
    return e2m1_value((uint8_t)(c % 2 ? byte >> 4 : byte & 15)) * e8m0_value(m->s4[i * (m->cols / 32) + c / 32]);
  }
  return e4m3_value(m->q[i * m->cols + c]) * (double)m->s[(i / 128) * (m->cols / 128) + c / 128];
}

/* One expert's share of the layer output.  For every listed token row r
 * (x_rows[r] is that token's hidden vector) and slot j with
 * ids[rows[r]*k + j] == e, adds
 *     w[rows[r]*k + j] * W2 (silu(W1 x) * (W3 x))
 * to y[r][:] in fp64.  W1, W3: [I][H]; W2: [H][I].  Returns the number of
 * (row, slot) terms added. */
static int64_t expert_accumulate(int32_t e, const int32_t* ids, const float* w, int32_t k,
                                 const int32_t* rows, int32_t n_rows, const uint16_t* x_rows,
                                 int32_t H, int32_t I, const wmat* w1, const wmat* w3,
                                 const wmat* w2, double* y) {
  int64_t m = 0;
  for (int32_t r = 0; r < n_rows; ++r)
    for (int32_t j = 0; j < k; ++j)
      if (ids[(int64_t)rows[r] * k + j] == e) ++m;
  if (m == 0) return 0;
  int32_t* mr = (int32_t*)malloc(sizeof(int32_t) * (size_t)m);
  double* mw = (double*)malloc(sizeof(double) * (size_t)m);
  int64_t n = 0;
  for (int32_t r = 0; r < n_rows; ++r)
    for (int32_t j = 0; j < k; ++j)
      if (ids[(int64_t)rows[r] * k + j] == e) {
        mr[n] = r;
        mw[n] = (double)w[(int64_t)rows[r] * k + j];
        ++n;
      }
  double* xd = (double*)malloc(sizeof(double) * (size_t)m * H);
  for (int64_t a = 0; a < m; ++a)
    for (int32_t c = 0; c < H; ++c) xd[a * H + c] = bf16_value(x_rows[(int64_t)mr[a] * H + c]);
  double* hh = (double*)malloc(sizeof(double) * (size_t)m * I);

  /* h = silu(W1 x) * (W3 x), one intermediate feature at a time. */
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < I; ++i) {
    double* r1 = (double*)malloc(sizeof(double) * (size_t)H);
    double* r3 = (double*)malloc(sizeof(double) * (size_t)H);
    for (int32_t c = 0; c < H; ++c) {
      r1[c] = wval(w1, i, c);
      r3[c] = wval(w3, i, c);
    }
    for (int64_t a = 0; a < m; ++a) {
      double g = 0.0, u = 0.0;
      for (int32_t c = 0; c < H; ++c) {
        g += r1[c] * xd[a * H + c];
        u += r3[c] * xd[a * H + c];
      }
      hh[a * I + i] = silu(g) * u;
    }
    free(r1);
    free(r3);
  }

  /* y += w * (W2 h), one output feature at a time. */
#pragma omp parallel for schedule(static)
  for (int32_t c = 0; c < H; ++c) {
    double* r2 = (double*)malloc(sizeof(double) * (size_t)I);
    for (int32_t i = 0; i < I; ++i) r2[i] = wval(w2, c, i);
    for (int64_t a = 0; a < m; ++a) {
      double o = 0.0;
      for (int32_t i = 0; i < I; ++i) o += r2[i] * hh[a * I + i];
      y[(int64_t)mr[a] * H + c] += mw[a] * o;
    }
    free(r2);
  }
  free(mr);
  free(mw);
  free(xd);
  free(hh);
  return m;
}

int64_t oracle_moe_expert_bf16(int32_t e, const int32_t* ids, const float* w, int32_t k,
                               const int32_t* rows, int32_t n_rows, const uint16_t* x_rows,
                               int32_t H, int32_t I, const uint16_t* w1, const uint16_t* w3,
                               const uint16_t* w2, double* y) {
  wmat m1 = {w1, 0, 0, H, 0, 0}, m3 = {w3, 0, 0, H, 0, 0}, m2 = {w2, 0, 0, I, 0, 0};
  return expert_accumulate(e, ids, w, k, rows, n_rows, x_rows, H, I, &m1, &m3, &m2, y);
}

/* fp8 e4m3 weights with one fp32 scale per 128x128 block: the weight value
 * is q * s exactly (in fp64).  s1, s3: [I/128][H/128]; s2: [H/128][I/128]. */
int64_t oracle_moe_expert_fp8(int32_t e, const int32_t* ids, const float* w, int32_t k,
                              const int32_t* rows, int32_t n_rows, const uint16_t* x_rows,
                              int32_t H, int32_t I, const uint8_t* q1, const float* s1,
                              const uint8_t* q3, const float* s3, const uint8_t* q2,
                              const float* s2, double* y) {
  wmat m1 = {0, q1, s1, H, 0, 0}, m3 = {0, q3, s3, H, 0, 0}, m2 = {0, q2, s2, I, 0, 0};
  return expert_accumulate(e, ids, w, k, rows, n_rows, x_rows, H, I, &m1, &m3, &m2, y);
}

/* MXFP4 weights (OCP Microscaling: e2m1 elements, one E8M0 scale per 32 elements along a
 * row): the weight value is e2m1(q) * 2^(s - 127) exactly (in fp64).  q1, q3: [I][H / 2];
 * s1, s3: [I][H / 32]; q2: [H][I / 2]; s2: [H][I / 32]. */
int64_t oracle_moe_expert_mxfp4(int32_t e, const int32_t* ids, const float* w, int32_t k,
                                const int32_t* rows, int32_t n_rows, const uint16_t* x_rows,
                                int32_t H, int32_t I, const uint8_t* q1, const uint8_t* s1,
                                const uint8_t* q3, const uint8_t* s3, const uint8_t* q2,
                                const uint8_t* s2, double* y) {
  wmat m1 = {0, 0, 0, H, q1, s1}, m3 = {0, 0, 0, H, q3, s3}, m2 = {0, 0, 0, I, q2, s2};
  return expert_accumulate(e, ids, w, k, rows, n_rows, x_rows, H, I, &m1, &m3, &m2, y);
}

/* Decoded value of one MXFP4 element (tests pin the decode through this). */
double oracle_mxfp4_value(uint8_t code, uint8_t scale) { return e2m1_value(code & 15) * e8m0_value(scale); }

/* ------------------------------------------------------------------------- */
/* Offline tuning (Sec. III-A Alg. 1, Sec. IV-A)                              */
/* ------------------------------------------------------------------------- */

/* Philox4x32-10 counter-based generator (Salmon, Moraes, Dror, Shaw, SC'11):
 * ten rounds of two 32x32->64 multiplies with the published multipliers and
 * Weyl key increments. */
static void philox(uint32_t c[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t y0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    const uint32_t y1 = (uint32_t)p1;
    const uint32_t y2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    const uint32_t y3 = (uint32_t)p0;
    c[0] = y0; c[1] = y1; c[2] = y2; c[3] = y3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

/* Two uniforms in (0,1) with 53-bit resolution from the Philox block at
 * counter (n, e, s, tag) under key seed. */
static void uniform_pair(uint64_t seed, uint32_t n, uint32_t e, uint32_t s, uint32_t tag,
                         double* u0, double* u1) {
  uint32_t c[4] = {n, e, s, tag};
  philox(c, (uint32_t)seed, (uint32_t)(seed >> 32));
  const double scale = 1.0 / 9007199254740992.0; /* 2^-53 */
  *u0 = ((double)(((uint64_t)(c[0] >> 5) << 26) | (c[1] >> 6)) + 0.5) * scale;
  *u1 = ((double)(((uint64_t)(c[2] >> 5) << 26) | (c[3] >> 6)) + 0.5) * scale;
}

/* log of a Gamma(alpha) variate for draw (e, s):
 *   G ~ Gamma(alpha + 1) by Marsaglia and Tsang (2000): d = a - 1/3,
 *   c = 1/sqrt(9d); x ~ N(0,1) (Box-Muller, cosine branch), v = (1 + c x)^3,
 *   accept when v > 0 and log u < x^2/2 + d - d v + d log v; G = d v.
 *   log Gamma(alpha) = log G + log(U) / alpha (the boost for shape < 1,
 *   applied for every alpha so the stream layout does not depend on it).
 * Attempt i reads blocks (2i, e, s, 0) and (2i+1, e, s, 0); the boost
 * uniform is block (0, e, s, 1). */
static double log_gamma_variate(uint64_t seed, double alpha, uint32_t e, uint32_t s) {
  const double a = alpha + 1.0;
  const double d = a - 1.0 / 3.0;
  const double c = 1.0 / sqrt(9.0 * d);
  double g = 0.0;
  for (uint32_t i = 0;; ++i) {
    double u1, u2, ua, ub;
    uniform_pair(seed, 2 * i, e, s, 0, &u1, &u2);
    uniform_pair(seed, 2 * i + 1, e, s, 0, &ua, &ub);
    const double x = sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
    double v = 1.0 + c * x;
    if (v <= 0.0) continue;
    v = v * v * v;
    if (log(ua) < 0.5 * x * x + d - d * v + d * log(v)) {
      g = d * v;
      break;
    }
  }
  double ub0, ub1;
  uniform_pair(seed, 0, e, s, 1, &ub0, &ub1);
  return log(g) + log(ub0) / alpha;
}

/* eff_exp of one sample p ~ Dir(alpha * 1_E) (Sec. II-D, Eq. (1)): the
 * Gamma construction p_e = G_e / sum G, evaluated from log G, then Eq. (2)
 * applied to p as Alg. 1 does. */
static double effexp_of_dirichlet_sample(uint64_t seed, double alpha, int32_t E, uint32_t s,
                                         double* logg) {
  double mx = -INFINITY;
  for (int32_t e = 0; e < E; ++e) {
    logg[e] = log_gamma_variate(seed, alpha, (uint32_t)e, s);
    if (logg[e] > mx) mx = logg[e];
  }
  double z = 0.0;
  for (int32_t e = 0; e < E; ++e) z += exp(logg[e] - mx);
  double sp = 0.0, sp2 = 0.0;
  for (int32_t e = 0; e < E; ++e) {
    const double p = exp(logg[e] - mx) / z;
    sp += p;
    sp2 += p * p;
  }
  return sp * sp / sp2;
}

/* Alg. 1 (Sec. III-A): the concentration of a symmetric Dirichlet whose mean
 * Effective Experts over S samples equals the target.  The mean grows with
 * alpha, so the algorithm brackets the root in [1e-6, 1e6] and halves the
 * bracket `iters` times at its arithmetic midpoint, keeping the half whose
 * mean straddles the target; the midpoint of the last halving is the answer.
 * The paper leaves S and the number of halvings open (taken as inputs).  The
 * samples use the same random numbers (key `seed`) at every alpha, so the
 * mean is a deterministic function of alpha. */
double oracle_alpha_search(int32_t E, double target, int32_t S, int32_t iters, uint64_t seed) {
  double lo = 1e-6, hi = 1e6, mid = 0.5 * (lo + hi);
  double* logg = (double*)malloc(sizeof(double) * (size_t)E);
  for (int32_t t = 0; t < iters; ++t) {
    mid = 0.5 * (lo + hi);
    double v = 0.0;
    for (int32_t s = 0; s < S; ++s) v += effexp_of_dirichlet_sample(seed, mid, E, (uint32_t)s, logg);
    v /= S;
    if (v < target) lo = mid;
    else hi = mid;
  }
  free(logg);
  return mid;
}

/* Mean eff_exp of S samples of Dir(alpha) under the same random numbers as
 * oracle_alpha_search (exposed for the monotonicity and moment checks). */
double oracle_mean_effexp(int32_t E, double alpha, int32_t S, uint64_t seed) {
  double* logg = (double*)malloc(sizeof(double) * (size_t)E);
  double v = 0.0;
  for (int32_t s = 0; s < S; ++s) v += effexp_of_dirichlet_sample(seed, alpha, E, (uint32_t)s, logg);
  free(logg);
  return v / S;
}

/* Exemplar of Sec. IV-A from S token-count vectors counts[S][E]: each
 * vector sorted in descending order and L2-normalised, the centroid of the
 * normalised vectors, renormalised to unit L2 norm, and quantised as
 * Q[r] = round-half-even(u[r] * 2^15).  An all-zero sample contributes a
 * zero vector. */
void oracle_exemplar(const int64_t* counts, int32_t S, int32_t E, int32_t* Q) {
  double* cen = (double*)calloc((size_t)E, sizeof(double));
  int64_t* s = (int64_t*)malloc(sizeof(int64_t) * (size_t)E);
  for (int32_t i = 0; i < S; ++i) {
    memcpy(s, counts + (int64_t)i * E, sizeof(int64_t) * (size_t)E);
    qsort(s, (size_t)E, sizeof(int64_t), cmp_desc_i64);
    double nn = 0.0;
    for (int32_t r = 0; r < E; ++r) nn += (double)s[r] * (double)s[r];
    nn = sqrt(nn);
    if (nn > 0.0)
      for (int32_t r = 0; r < E; ++r) cen[r] += (double)s[r] / nn / S;
  }
  double cn = 0.0;
  for (int32_t r = 0; r < E; ++r) cn += cen[r] * cen[r];
  cn = sqrt(cn);
  for (int32_t r = 0; r < E; ++r) Q[r] = (int32_t)rint(cn > 0.0 ? cen[r] / cn * 32768.0 : 0.0);
  free(cen);
  free(s);
}

/* Kernel choice of Sec. IV-A for one distribution: the variant with the
 * lowest mean latency over the S samples (lat[s][v]); ties to the lower
 * variant index. */
int32_t oracle_fastest_mean(const double* lat, int32_t S, int32_t V) {
  int32_t best = -1;
  double best_mean = 0.0;
  for (int32_t v = 0; v < V; ++v) {
    double m = 0.0;
    for (int32_t s = 0; s < S; ++s) m += lat[(int64_t)s * V + v];
    m /= S;
    if (best < 0 || m < best_mean) {
      best = v;
      best_mean = m;
    }
  }
  return best;
}

/* One sample p ~ Dir(alpha * 1_E) as log p (the construction used by
 * Alg. 1 above), exposed for the moment checks of Eq. (1). */
void oracle_dirichlet_logp(int32_t E, double alpha, uint32_t s, uint64_t seed, double* logp) {
  double mx = -INFINITY;
  for (int32_t e = 0; e < E; ++e) {
    logp[e] = log_gamma_variate(seed, alpha, (uint32_t)e, s);
    if (logp[e] > mx) mx = logp[e];
  }
  double z = 0.0;
  for (int32_t e = 0; e < E; ++e) z += exp(logp[e] - mx);
  const double lz = mx + log(z);
  for (int32_t e = 0; e < E; ++e) logp[e] -= lz;
}

/* ------------------------------------------------------------------------- */
/* Router (the gating step in front of the path)                              */
/* ------------------------------------------------------------------------- */

/* Sec. II-A, selection and gates from given logits [T][E] (fp64): the token's slots are its
 * k largest logits in descending order, equal logits taken lowest expert id first; the gates
 * are the softmax over those k logits (the reading of the gate form taken for this build). */
void oracle_topk_softmax(const double* logits, int32_t T, int32_t E, int32_t k, int32_t* ids, double* w) {
  for (int32_t t = 0; t < T; ++t) {
    const double* l = logits + (int64_t)t * E;
    int32_t* id = ids + (int64_t)t * k;
    for (int32_t j = 0; j < k; ++j) {
      int32_t best = -1;
      for (int32_t e = 0; e < E; ++e) {
        int taken = 0;
        for (int32_t q = 0; q < j; ++q) taken |= id[q] == e;
        if (taken) continue;
        if (best < 0 || l[e] > l[best]) best = e;
      }
      id[j] = best;
    }
    double z = 0.0;
    for (int32_t j = 0; j < k; ++j) z += exp(l[id[j]] - l[id[0]]);
    for (int32_t j = 0; j < k; ++j) w[(int64_t)t * k + j] = exp(l[id[j]] - l[id[0]]) / z;
  }
}

/* Sec. II-A: the gating network scores every expert for each token and the token goes to the
 * k best.  Here the gate is a linear layer,
 *   logits[t][e] = sum_h x[t][h] * wg[e][h] + bias[e],
 * in fp64 from the bf16 x [T][H] and wg [E][H] (bias fp32 [E], or NULL), followed by the
 * selection and gates above. */
void oracle_router(const uint16_t* x, const uint16_t* wg, const float* bias, int32_t T, int32_t H,
                   int32_t E, int32_t k, double* logits, int32_t* ids, double* w) {
#pragma omp parallel for schedule(static)
  for (int32_t t = 0; t < T; ++t)
    for (int32_t e = 0; e < E; ++e) {
      double s = 0.0;
      for (int32_t h = 0; h < H; ++h)
        s += bf16_value(x[(int64_t)t * H + h]) * bf16_value(wg[(int64_t)e * H + h]);
      logits[(int64_t)t * E + e] = s + (bias ? (double)bias[e] : 0.0);
    }
  oracle_topk_softmax(logits, T, E, k, ids, w);
}

/* ------------------------------------------------------------------------- */
/* Effective-Experts-only dispatch (the scalar statistic of Sec. III-A used   */
/* as the matcher instead of the exemplar match of Sec. IV-B)                 */
/* ------------------------------------------------------------------------- */

/* Map from the Effective Experts bucket (-1 .. 13, Eq. (2) and the ddist:X grid) to a
 * variant, derived from one token bucket's exemplar table: each exemplar Q_x (a sorted,
 * quantised unit vector of counts) has its own Effective Experts (sum Q)^2 / sum Q^2 and so
 * its own bucket; bucket b maps to the kernel of the first exemplar in b, else to that of
 * the nearest bucket holding an exemplar (the lower one on a tie); bucket -1 (no tokens)
 * maps to the NoDA kernel.  map[b + 1], 15 entries (the reading of the cheaper matcher taken
 * for this build). */
void oracle_effexp_map(const int32_t* Q, const int32_t* kid, int32_t n_ex, int32_t E, int32_t noda,
                       int32_t* map) {
  int32_t first[14];
  for (int b = 0; b < 14; ++b) first[b] = -1;
  for (int32_t x = 0; x < n_ex; ++x) {
    uint64_t s = 0, s2 = 0;
    for (int32_t e = 0; e < E; ++e) {
      s += (uint64_t)Q[(int64_t)x * E + e];
      s2 += (uint64_t)Q[(int64_t)x * E + e] * (uint64_t)Q[(int64_t)x * E + e];
    }
    const int32_t b = oracle_effexp_bucket(s * s, s2, E);
    if (b >= 0 && first[b] < 0) first[b] = x;
  }
  map[0] = noda;
  for (int b = 0; b < 14; ++b) {
    int32_t pick = -1;
    for (int d = 0; d < 14 && pick < 0; ++d) {
      if (b - d >= 0 && first[b - d] >= 0) pick = first[b - d];
      else if (b + d < 14 && first[b + d] >= 0) pick = first[b + d];
    }
    map[b + 1] = pick >= 0 ? kid[pick] : noda;
  }
}
