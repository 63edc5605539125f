/*
 * fathom_oracle.c -- plain, slow CPU oracle for the Fathom hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes or
 * calls this file; only the tests, the smoke check and the bench's CPU-baseline
 * leg load it.  It shares no code, header, table or constant with the HIP path.
 *
 * Paper: "Fathom: Per-Query Read Depth for Sparse Decoding over Offloaded KV
 * Caches" (arXiv 2609.17652).  Every function cites the passage it follows:
 *   Sec. 3.2, Eq. (2)        4-bit per-channel quantiser, fp16 block scales,
 *                            bit planes, prefix dequantisation.
 *   Sec. 3.3, Eq. (g), (wf)  channel importance, reverse water-filling.
 *   Sec. 2 (SparQ)           grouped top-r channel rule (uniform-depth mode).
 *   Sec. 2 (Top-k decoding)  per-head top-k, sink + local protocol, exact
 *                            attention over the selected set.
 *   App. A                   worked example (the main pin of the oracle).
 *
 * Arithmetic is fp64 except two steps the paper leaves unspecified and this
 * oracle fixes in fp32: the importance g (Eq. (g), summed over heads in fp32)
 * and the fp32 score replica below.  Compile with -O2 -ffp-contract=off so
 * that no multiply-add is fused behind our back.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_SCALE_OVERFLOW 1u
#define ORC_NONFINITE 2u
#define ORC_TOPK_SHORT 8u

/* ------------------------------------------------------------------------- */
/* IEEE 754 binary16 conversions, written from the format's definition:       */
/* 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits; subnormals are    */
/* multiples of 2^-24; round to nearest, ties to even.                        */
/* ------------------------------------------------------------------------- */
uint16_t orc_f32_to_f16(float xf) {
  double x = (double)xf; /* exact */
  if (isnan(x)) return 0x7E00u;
  uint16_t sign = signbit(x) ? 0x8000u : 0u;
  double a = fabs(x);
  if (a >= 65520.0) return sign | 0x7C00u; /* 65504 + half an ulp (16) rounds up */
  if (a < ldexp(1.0, -14)) {               /* subnormal range: units of 2^-24 */
    double m = nearbyint(a * ldexp(1.0, 24)); /* default mode: nearest-even */
    return sign | (uint16_t)m;             /* m == 1024 is the smallest normal */
  }
  int E;
  frexp(a, &E); /* a = f * 2^E, f in [0.5, 1) */
  int e = E - 1; /* a in [2^e, 2^(e+1)) */
  double m = nearbyint(ldexp(a, 10 - e)); /* in [1024, 2048] */
  if (m == 2048.0) { m = 1024.0; e += 1; }
  if (e > 15) return sign | 0x7C00u;
  return sign | (uint16_t)(((e + 15) << 10) | ((int)m - 1024));
}

/* The conversion above applied element by element (for exhaustive checks). */
void orc_f32_to_f16_n(const float* x, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_f32_to_f16(x[i]);
}

double orc_f16_to_f64(uint16_t h) {
  int sign = (h >> 15) & 1, e = (h >> 10) & 31, f = h & 1023;
  double v;
  if (e == 0) v = ldexp((double)f, -24);
  else if (e == 31) v = f ? NAN : INFINITY;
  else v = ldexp(1024.0 + f, e - 25);
  return sign ? -v : v;
}

/* ------------------------------------------------------------------------- */
/* Sec. 3.2, Eq. (2): quantise one unit's keys and pack bit planes.           */
/*   K       [n][D] fp32, token-major (one KV head of one sequence)           */
/*   planes  [D][4][nb_cap] u64: word (j,p,b) holds bit p (0 = MSB) of the    */
/*           codes of tokens 64b..64b+63 of channel j, token 64b+i at bit i.  */
/*   scales  [D][nb_cap] fp16 bit patterns: a16 = fp16(block absmax).         */
/* Blocks at or beyond ceil(n/64) are written as zero words and zero scales.  */
/* Returns the device-status bits the kernel would raise.                     */
/* ------------------------------------------------------------------------- */
uint32_t orc_pack(const float* K, int64_t n, int D, int64_t nb_cap,
                  uint64_t* planes, uint16_t* scales) {
  uint32_t st = 0;
  int64_t nb = (n + 63) / 64;
  for (int j = 0; j < D; ++j) {
    for (int64_t b = 0; b < nb_cap; ++b) {
      uint64_t w[4] = {0, 0, 0, 0};
      uint16_t a16 = 0;
      if (b < nb) {
        int64_t i0 = 64 * b, i1 = i0 + 64 < n ? i0 + 64 : n;
        /* block absmax over the valid tokens (NaN keys ignored, flagged) */
        float a = 0.0f;
        for (int64_t i = i0; i < i1; ++i) {
          float k = K[i * D + j];
          if (!isfinite(k)) st |= ORC_NONFINITE;
          if (isnan(k)) continue;
          float ak = fabsf(k);
          if (ak > a) a = ak;
        }
        a16 = orc_f32_to_f16(a);
        double a16d = orc_f16_to_f64(a16);
        int overflow = isinf(a16d);
        if (overflow) st |= ORC_SCALE_OVERFLOW;
        double s = a16d / 8.0; /* cell width s = a/8 */
        for (int64_t i = i0; i < i1; ++i) {
          double k = (double)K[i * D + j];
          int c;
          if (a16d == 0.0 || overflow || isnan(k)) {
            c = 8; /* zero scale, overflowed scale or NaN key: the zero code */
          } else {
            /* exact real floor: |k/s| <= ~8 and s has 11 significant bits, so
             * the fp64 quotient cannot cross an integer */
            double m = floor(k / s);
            if (m < -8.0) m = -8.0;
            if (m > 7.0) m = 7.0;
            c = (int)m + 8;
          }
          for (int p = 0; p < 4; ++p)
            if ((c >> (3 - p)) & 1) w[p] |= (uint64_t)1 << (i - i0);
        }
      }
      for (int p = 0; p < 4; ++p) planes[((int64_t)j * 4 + p) * nb_cap + b] = w[p];
      scales[(int64_t)j * nb_cap + b] = a16;
    }
  }
  return st;
}

/* code prefix c^(t) of token i, channel j, read from the first t planes */
static int prefix_code(const uint64_t* planes, int64_t nb_cap, int j, int t, int64_t i) {
  int64_t b = i / 64;
  int bit = (int)(i % 64);
  int c = 0;
  for (int p = 0; p < t; ++p)
    c = 2 * c + (int)((planes[((int64_t)j * 4 + p) * nb_cap + b] >> bit) & 1);
  return c;
}

/* Sec. 3.2: dequantised depth-t value (c^(t) + 1/2 - 2^(t-1)) * a / 2^(t-1), fp64 (exact). */
double orc_dequant(const uint64_t* planes, const uint16_t* scales, int64_t nb_cap,
                   int j, int t, int64_t i) {
  if (t == 0) return 0.0;
  int c = prefix_code(planes, nb_cap, j, t, i);
  double a = orc_f16_to_f64(scales[(int64_t)j * nb_cap + i / 64]);
  return ((double)c + 0.5 - ldexp(1.0, t - 1)) * a * ldexp(1.0, 1 - t);
}

/* ------------------------------------------------------------------------- */
/* Sec. 3.3, Eq. (g): g_j = sum_h (q_j^(h))^2 Var(k_j), in fp32 in the order  */
/* fl(fl(sum_h fl(q^2)) * var), heads ascending, no fused multiply-add.       */
/* ------------------------------------------------------------------------- */
void orc_importance(const float* q, int G, int D, const float* var, float* g) {
  for (int j = 0; j < D; ++j) {
    float s = 0.0f;
    for (int h = 0; h < G; ++h) {
      float p = q[h * D + j] * q[h * D + j];
      s = s + p;
    }
    g[j] = s * var[j];
  }
}

static int cmp_desc_double(const void* x, const void* y) {
  double a = *(const double*)x, b = *(const double*)y;
  return (a < b) - (a > b);
}

/* ------------------------------------------------------------------------- */
/* Sec. 3.3, Eq. (wf), closed form of the water line.                         */
/* t_j(theta) = clip(round(log4(g_j/theta)), 0, 4) with round-half-up (App. A */
/* places the one-plane interval at 0.5 <= log4(g/theta) < 1.5), so           */
/* t_j(theta) >= m  <=>  g_j * 2^-(2m-1) >= theta.  The depths sum is the     */
/* number of candidates c_{j,m} = g_j 2^-(2m-1) (m = 1..4) that are >= theta; */
/* the smallest theta at which it is <= B is approached from above at         */
/* theta* = the (B+1)-th largest candidate (0 if B >= 4D), where              */
/* t_j = #{m : c_{j,m} > theta*}.  Candidates are exact in fp64.              */
/* ------------------------------------------------------------------------- */
uint32_t orc_alloc_waterfill(const float* q, int G, int D, const float* var, int B,
                             uint8_t* depths, float* theta) {
  uint32_t st = 0;
  float* g = (float*)malloc(sizeof(float) * D);
  double* cand = (double*)malloc(sizeof(double) * 4 * D);
  orc_importance(q, G, D, var, g);
  for (int j = 0; j < D; ++j) {
    if (!isfinite(g[j]) || g[j] < 0.0f) st |= ORC_NONFINITE;
    for (int m = 1; m <= 4; ++m) cand[4 * j + (m - 1)] = ldexp((double)g[j], -(2 * m - 1));
  }
  double* sorted = (double*)malloc(sizeof(double) * 4 * D);
  memcpy(sorted, cand, sizeof(double) * 4 * D);
  qsort(sorted, (size_t)4 * D, sizeof(double), cmp_desc_double);
  double th = (B < 4 * D) ? sorted[B] : 0.0;
  for (int j = 0; j < D; ++j) {
    int t = 0;
    for (int m = 0; m < 4; ++m) t += cand[4 * j + m] > th;
    depths[j] = (uint8_t)t;
  }
  if (theta) *theta = (float)th;
  free(g); free(cand); free(sorted);
  return st;
}

/* Eq. (wf) evaluated directly at one theta: fp64 log4, round half up, clip. */
int orc_depths_at(const double* g, int D, double theta, uint8_t* depths) {
  int sum = 0;
  for (int j = 0; j < D; ++j) {
    int t = 0;
    if (g[j] > 0.0) {
      double x = log(g[j] / theta) / log(4.0);
      double r = floor(x + 0.5);
      t = r < 0.0 ? 0 : (r > 4.0 ? 4 : (int)r);
    }
    depths[j] = (uint8_t)t;
    sum += t;
  }
  return sum;
}

/* ------------------------------------------------------------------------- */
/* Sec. 3.3 and App. A: the paper's own search -- geometric bisection on      */
/* theta from a bracket [lo, hi]; each trial is sqrt(lo*hi); a trial whose    */
/* depth sum exceeds B becomes lo, otherwise hi.  Records every trial.        */
/* Returns the final upper end (the water line the paper reports).            */
/* ------------------------------------------------------------------------- */
double orc_bisect(const double* g, int D, int B, double lo, double hi, int steps,
                  double* trial_theta, int* trial_sum, uint8_t* depths_out) {
  uint8_t* d = (uint8_t*)malloc((size_t)D);
  for (int s = 0; s < steps; ++s) {
    double th = sqrt(lo * hi);
    int sum = orc_depths_at(g, D, th, d);
    if (trial_theta) trial_theta[s] = th;
    if (trial_sum) trial_sum[s] = sum;
    if (sum > B) lo = th; else hi = th;
  }
  if (depths_out) orc_depths_at(g, D, hi, depths_out);
  free(d);
  return hi;
}

/* ------------------------------------------------------------------------- */
/* Sec. 2 (SparQ) and App. A: grouped top-r rule.  w_j = sum_h |q_j^(h)| in   */
/* fp32, heads ascending; the r channels first in (w desc, j asc) order are   */
/* read at all 4 planes, the rest not at all.  theta = w of the r-th pick.    */
/* ------------------------------------------------------------------------- */
uint32_t orc_alloc_topr(const float* q, int G, int D, int r, uint8_t* depths, float* theta) {
  uint32_t st = 0;
  float* w = (float*)malloc(sizeof(float) * D);
  for (int j = 0; j < D; ++j) {
    float s = 0.0f;
    for (int h = 0; h < G; ++h) s = s + fabsf(q[h * D + j]);
    if (!isfinite(s)) st |= ORC_NONFINITE;
    w[j] = s;
  }
  float th = 0.0f;
  for (int j = 0; j < D; ++j) {
    int rank = 0; /* position of j in (w desc, j asc) order */
    for (int i = 0; i < D; ++i) rank += (w[i] > w[j]) || (w[i] == w[j] && i < j);
    depths[j] = rank < r ? 4 : 0;
    if (rank == r - 1) th = w[j];
  }
  if (theta) *theta = th;
  free(w);
  return st;
}

/* ------------------------------------------------------------------------- */
/* Sec. 3.2-3.3: approximate scores s_h(i) = sum_{j: t_j > 0} q_hj khat_ij,   */
/* raw q.khat without 1/sqrt(D) (App. A prints them that way).                */
/* Reference: fp64, channels ascending (every product is exact in fp64).      */
/* ------------------------------------------------------------------------- */
void orc_scores_f64(const uint64_t* planes, const uint16_t* scales, int64_t n, int64_t nb_cap,
                    int D, const float* q, int G, const uint8_t* depths, double* out,
                    double* abs_out) {
  for (int h = 0; h < G; ++h) {
    for (int64_t i = 0; i < n; ++i) {
      double s = 0.0, sa = 0.0;
      for (int j = 0; j < D; ++j) {
        if (depths[j] == 0) continue;
        double term = (double)q[h * D + j] * orc_dequant(planes, scales, nb_cap, j, depths[j], i);
        s += term;
        sa += fabs(term);
      }
      out[(int64_t)h * n + i] = s;
      if (abs_out) abs_out[(int64_t)h * n + i] = sa;
    }
  }
}

/* ------------------------------------------------------------------------- */
/* fp32 score replica (the paper states no score precision or order; this    */
/* is the order the GPU path must reproduce): per head and key, channels asc, */
/*   khat = (c^(t) + 1/2 - 2^(t-1)) * a16 * 2^(1-t)   (exact in fp32)         */
/*   acc  = fmaf(q_hj, khat, acc),  acc starting at +0.                       */
/* ------------------------------------------------------------------------- */
void orc_scores_f32(const uint64_t* planes, const uint16_t* scales, int64_t n, int64_t nb_cap,
                    int D, const float* q, int G, const uint8_t* depths, float* out) {
  for (int h = 0; h < G; ++h) {
    for (int64_t i = 0; i < n; ++i) {
      float acc = 0.0f;
      for (int j = 0; j < D; ++j) {
        int t = depths[j];
        if (t == 0) continue;
        float khat = (float)orc_dequant(planes, scales, nb_cap, j, t, i); /* exact */
        acc = fmaf(q[h * D + j], khat, acc);
      }
      out[(int64_t)h * n + i] = acc;
    }
  }
}

/* ------------------------------------------------------------------------- */
/* Sec. 2 (Top-k decoding): top-k of one head's scores over the eligible      */
/* range [lo, n - tail), ordered by (score desc, index asc); -0 equals +0;    */
/* NaN ranks below every number.  Slots beyond the eligible count get -1.     */
/* ------------------------------------------------------------------------- */
typedef struct { float s; int isnan_; int64_t i; } orc_item;

static int cmp_item(const void* x, const void* y) {
  const orc_item* a = (const orc_item*)x;
  const orc_item* b = (const orc_item*)y;
  if (a->isnan_ != b->isnan_) return a->isnan_ - b->isnan_; /* numbers first */
  if (!a->isnan_) {
    if (a->s > b->s) return -1; /* -0 == +0 under IEEE comparison */
    if (a->s < b->s) return 1;
  }
  return (a->i > b->i) - (a->i < b->i);
}

uint32_t orc_topk(const float* s, int64_t n, int k, int64_t lo, int64_t tail,
                  int32_t* idx, float* val) {
  uint32_t st = 0;
  int64_t hi = n - tail;
  if (lo < 0) lo = 0;
  int64_t m = hi > lo ? hi - lo : 0;
  orc_item* it = (orc_item*)malloc(sizeof(orc_item) * (size_t)(m > 0 ? m : 1));
  for (int64_t i = 0; i < m; ++i) {
    float v = s[lo + i];
    it[i].s = v;
    it[i].isnan_ = isnan(v) ? 1 : 0;
    it[i].i = lo + i;
    if (!isfinite(v)) st |= ORC_NONFINITE;
  }
  qsort(it, (size_t)m, sizeof(orc_item), cmp_item);
  for (int r = 0; r < k; ++r) {
    if (r < m) {
      idx[r] = (int32_t)it[r].i;
      if (val) val[r] = it[r].s;
    } else {
      idx[r] = -1;
      if (val) val[r] = NAN;
      st |= ORC_TOPK_SHORT;
    }
  }
  free(it);
  return st;
}

/* ------------------------------------------------------------------------- */
/* Sec. 2 (Top-k decoding) and Sec. 4: exact attention over the selected set  */
/* S_h = sink [0, ns) U local [max(ns, n - nl), n) U {idx_h entries inside    */
/* [ns, max(ns, n - nl))}, with ns = min(n_sink, n); entries < 0 or outside   */
/* that middle range are skipped.  fp64 throughout.                           */
/* ------------------------------------------------------------------------- */
void orc_sparse_attn(const float* q, const uint16_t* K16, const uint16_t* V16, int64_t n,
                     int G, int D, const int32_t* idx, int k, int n_sink, int n_local,
                     double sm_scale, double* out) {
  int64_t ns = n_sink < n ? n_sink : n;
  int64_t l0 = n - n_local > ns ? n - n_local : ns;
  int64_t cap = ns + (n - l0) + k;
  int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)(cap > 0 ? cap : 1));
  double* z = (double*)malloc(sizeof(double) * (size_t)(cap > 0 ? cap : 1));
  for (int h = 0; h < G; ++h) {
    int64_t m = 0;
    for (int64_t i = 0; i < ns; ++i) rows[m++] = i;
    for (int64_t i = l0; i < n; ++i) rows[m++] = i;
    for (int r = 0; r < k; ++r) {
      int64_t i = idx[(int64_t)h * k + r];
      if (i >= ns && i < l0) rows[m++] = i;
    }
    double zmax = -INFINITY;
    for (int64_t r = 0; r < m; ++r) {
      double d = 0.0;
      for (int c = 0; c < D; ++c) d += (double)q[h * D + c] * orc_f16_to_f64(K16[rows[r] * D + c]);
      z[r] = d * sm_scale;
      if (z[r] > zmax) zmax = z[r];
    }
    double den = 0.0;
    for (int64_t r = 0; r < m; ++r) { z[r] = exp(z[r] - zmax); den += z[r]; }
    for (int c = 0; c < D; ++c) {
      double o = 0.0;
      for (int64_t r = 0; r < m; ++r) o += z[r] * orc_f16_to_f64(V16[rows[r] * D + c]);
      out[(int64_t)h * D + c] = m > 0 ? o / den : 0.0;
    }
  }
  free(rows); free(z);
}
