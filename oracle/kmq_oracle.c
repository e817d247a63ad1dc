/*
 * kmq_oracle.c -- plain CPU oracle (TEST INFRASTRUCTURE ONLY; see kmq_oracle.h).
 *
 * Written for a reader checking it against the paper by eye: one loop per
 * definition, fp64 sums, exact integer sums, OpenMP only across independent
 * points (or independent dimensions) so results do not depend on the thread
 * count.  Build with -ffp-contract=off so every fp32 expression is evaluated
 * exactly as written (no silent fused multiply-adds).
 */
#include "kmq_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

static inline int bit_of(const uint32_t *row, int32_t i) { return (int)((row[i >> 5] >> (i & 31)) & 1u); }

/* ------------------------------------------------------------------------ */
/* SQ8 (Sec. 3.1): bias b and scale s; here one (lo, hi) pair per dimension. */

void orc_sq8_fit(const float *X, int64_t n, int32_t d, float *lo, float *hi) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < d; ++i) {
    float mn = X[i], mx = X[i];
    for (int64_t r = 1; r < n; ++r) {
      float v = X[r * d + i];
      if (v < mn) mn = v;
      if (v > mx) mx = v;
    }
    lo[i] = mn;
    hi[i] = mx;
  }
}

void orc_sq8_encode(const float *X, int64_t n, int32_t d, const float *lo, const float *hi,
                    uint8_t *codes) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    for (int32_t i = 0; i < d; ++i) {
      /* s = (hi-lo)/255, code = clip(round((x - b)/s), 0, 255), computed as (x-lo)*(255/(hi-lo)). */
      float range = hi[i] - lo[i];
      float inv = range > 0.0f ? 255.0f / range : 0.0f;
      float t = rintf((X[r * d + i] - lo[i]) * inv);
      if (t < 0.0f) t = 0.0f;
      if (t > 255.0f) t = 255.0f;
      codes[r * d + i] = (uint8_t)t;
    }
  }
}

/* ------------------------------------------------------------------------ */
/* bfloat16 storage (Sec. 2.4 names 16-bit full-precision vectors).  A finite
 * value x = f * 2^e with 0.5 <= |f| < 1 has bfloat16 neighbours spaced
 * 2^(e-8) apart (never finer than the subnormal spacing 2^-133).  x / spacing is
 * exact in fp64, rint() rounds it to the nearest integer with ties to even (the
 * default rounding mode), and scaling back is exact again; the rounded value is
 * an fp32 number whose low 16 bits are zero. */
static uint16_t bf16_of(float x) {
  uint32_t u;
  if (isnan(x)) {
    memcpy(&u, &x, 4);
    return (uint16_t)((u >> 16) | 0x0040u); /* keep sign and payload top, force quiet */
  }
  float r = x;
  if (x != 0.0f && !isinf(x)) {
    int e;
    (void)frexp((double)x, &e);
    int se = e - 8 < -133 ? -133 : e - 8;
    double q = rint(ldexp((double)x, -se));
    r = (float)ldexp(q, se); /* exact unless it passes the fp32 range (then +-inf) */
  }
  memcpy(&u, &r, 4);
  return (uint16_t)(u >> 16);
}

void orc_bf16_round(const float *X, int64_t n, uint16_t *out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = bf16_of(X[i]);
}

/* ------------------------------------------------------------------------ */
/* 1-bit sign codes (Sec. 3.1, RabitQ without rotation). */

void orc_col_mean(const float *X, int64_t n, int32_t d, float *m) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < d; ++i) {
    double s = 0.0;
    for (int64_t r = 0; r < n; ++r) s += (double)X[r * d + i];
    m[i] = (float)(s / (double)n);
  }
}

void orc_sign1_encode(const float *X, int64_t n, int32_t d, const float *m, int32_t d0,
                      uint32_t *bits, float *alpha) {
  const int32_t W = d / 32;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    uint32_t *row = bits + r * W;
    for (int32_t w = 0; w < W; ++w) row[w] = 0u;
    double s2 = 0.0, s1 = 0.0;
    for (int32_t i = 0; i < d; ++i) {
      float ri = X[r * d + i] - m[i]; /* residual around the dataset mean */
      if (ri > 0.0f) row[i >> 5] |= 1u << (i & 31);
      if (i >= d0) {
        s2 += (double)ri * (double)ri;
        s1 += fabs((double)ri);
      }
    }
    /* alpha = ||r||^2 / ||r||_1 = (1/sqrt(d')) ||r|| / <xbar, x>: the decoding radius scale. */
    alpha[r] = s1 > 0.0 ? (float)(s2 / s1) : 0.0f;
  }
}

void orc_sign1_decode(const uint32_t *bits, const float *alpha, int64_t n, int32_t d, int32_t d0,
                      const float *m, float *out, int64_t ldo) {
  const int32_t W = d / 32;
  for (int64_t r = 0; r < n; ++r)
    for (int32_t i = d0; i < d; ++i) {
      float s = bit_of(bits + r * W, i) ? alpha[r] : -alpha[r];
      out[r * ldo + i] = m[i] + s;
    }
}

/* ------------------------------------------------------------------------ */
/* PCA (Sec. 3.1): mean, covariance, projection onto given eigenvectors. */

void orc_pca_cov(const float *X, int64_t n, int32_t d, double *mean, double *cov) {
  for (int32_t i = 0; i < d; ++i) {
    double s = 0.0;
    for (int64_t r = 0; r < n; ++r) s += (double)X[r * d + i];
    mean[i] = s / (double)n;
  }
#pragma omp parallel for schedule(dynamic)
  for (int32_t i = 0; i < d; ++i) {
    for (int32_t j = i; j < d; ++j) {
      double s = 0.0;
      for (int64_t r = 0; r < n; ++r)
        s += ((double)X[r * d + i] - mean[i]) * ((double)X[r * d + j] - mean[j]);
      cov[(int64_t)i * d + j] = s / (double)n;
      cov[(int64_t)j * d + i] = s / (double)n;
    }
  }
}

double orc_pca_cov_entry(const float *X, int64_t n, int32_t d, const double *mean, int32_t i,
                         int32_t j) {
  double s = 0.0;
  for (int64_t r = 0; r < n; ++r)
    s += ((double)X[r * d + i] - mean[i]) * ((double)X[r * d + j] - mean[j]);
  return s / (double)n;
}

void orc_project(const float *X, int64_t n, int32_t d, const float *mean, const float *W,
                 int32_t dout, float *Y) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    for (int32_t o = 0; o < dout; ++o) {
      double s = 0.0;
      for (int32_t i = 0; i < d; ++i)
        s += ((double)X[r * d + i] - (double)mean[i]) * (double)W[(int64_t)i * dout + o];
      Y[r * dout + o] = (float)s;
    }
  }
}

/* ------------------------------------------------------------------------ */
/* STEP 2 (Sec. 2.3): nearest centroid by squared L2. */

void orc_assign_f32(const float *X, int64_t n, int32_t d, int64_t ldx, const float *C, int32_t k,
                    int32_t *a, double *dist) {
  double *cn = (double *)malloc(sizeof(double) * (size_t)k);
  for (int32_t j = 0; j < k; ++j) {
    double s = 0.0;
    for (int32_t i = 0; i < d; ++i) s += (double)C[(int64_t)j * d + i] * (double)C[(int64_t)j * d + i];
    cn[j] = s;
  }
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    const float *x = X + r * ldx;
    int32_t best = 0;
    double bs = 0.0;
    for (int32_t j = 0; j < k; ++j) {
      double dot = 0.0;
      for (int32_t i = 0; i < d; ++i) dot += (double)x[i] * (double)C[(int64_t)j * d + i];
      double s = cn[j] - 2.0 * dot; /* ||x-c||^2 minus the x-only term ||x||^2 */
      if (j == 0 || s < bs) {
        bs = s;
        best = j;
      }
    }
    a[r] = best;
    if (dist) {
      double e = 0.0;
      for (int32_t i = 0; i < d; ++i) {
        double t = (double)x[i] - (double)C[(int64_t)best * d + i];
        e += t * t;
      }
      dist[r] = e;
    }
  }
  free(cn);
}

void orc_assign_sq8(const uint8_t *X, int64_t n, int32_t d, const uint8_t *C, int32_t k, int32_t *a,
                    int64_t *dist) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    const uint8_t *x = X + r * d;
    int32_t best = 0;
    int64_t bd = 0;
    for (int32_t j = 0; j < k; ++j) {
      int64_t e = 0; /* distance computed directly in the quantised domain */
      for (int32_t i = 0; i < d; ++i) {
        int64_t t = (int64_t)x[i] - (int64_t)C[(int64_t)j * d + i];
        e += t * t;
      }
      if (j == 0 || e < bd) {
        bd = e;
        best = j;
      }
    }
    a[r] = best;
    if (dist) dist[r] = bd;
  }
}

double orc_prune_factor(int32_t D, int32_t d, double eps0) {
  const double g = 1.0 + eps0 / sqrt((double)D);
  return g * g * (double)D / (double)d;
}

void orc_assign_pruned_f32(const float *X, int64_t n, int32_t d, const float *C, int32_t k, const int32_t *prev,
                           double eps0, int32_t d_front, int32_t step, int32_t *a, double *dist,
                           int64_t *counters) {
  int64_t tested = 0, passed = 0, full = 0;
#pragma omp parallel for schedule(static) reduction(+ : tested, passed, full)
  for (int64_t r = 0; r < n; ++r) {
    const float *x = X + r * d;
    const int32_t pj = prev[r];
    double tau = 0.0;
    for (int32_t i = 0; i < d; ++i) {
      const double t = (double)x[i] - (double)C[(int64_t)pj * d + i];
      tau += t * t;
    }
    int32_t best = pj;
    double bd = tau;
    for (int32_t j = 0; j < k; ++j) {
      if (j == pj) continue;
      const float *c = C + (int64_t)j * d;
      double p = 0.0;
      int32_t i = 0, alive = 1;
      for (int32_t D = d_front; D < d; D += step) { /* checkpoints */
        for (; i < D; ++i) {
          const double t = (double)x[i] - (double)c[i];
          p += t * t;
        }
        const int first = D == d_front;
        tested += first;
        if (p > tau * orc_prune_factor(D, d, eps0)) {
          alive = 0;
          break;
        }
        passed += first;
      }
      if (!alive) continue;
      for (; i < d; ++i) {
        const double t = (double)x[i] - (double)c[i];
        p += t * t;
      }
      ++full;
      if (p < bd || (p == bd && j < best)) {
        bd = p;
        best = j;
      }
    }
    a[r] = best;
    if (dist) dist[r] = bd;
  }
  if (counters) {
    counters[0] = tested;
    counters[1] = passed;
    counters[2] = full;
  }
}

void orc_assign_pruned_sq8(const uint8_t *X, int64_t n, int32_t d, const uint8_t *C, int32_t k,
                           const int32_t *prev, double eps0, int32_t d_front, int32_t step, int32_t *a,
                           int64_t *dist, int64_t *counters) {
  int64_t tested = 0, passed = 0, full = 0;
#pragma omp parallel for schedule(static) reduction(+ : tested, passed, full)
  for (int64_t r = 0; r < n; ++r) {
    const uint8_t *x = X + r * d;
    const int32_t pj = prev[r];
    int64_t tau = 0;
    for (int32_t i = 0; i < d; ++i) {
      const int64_t t = (int64_t)x[i] - (int64_t)C[(int64_t)pj * d + i];
      tau += t * t;
    }
    const float tauf = (float)tau;
    int32_t best = pj;
    int64_t bd = tau;
    for (int32_t j = 0; j < k; ++j) {
      if (j == pj) continue;
      const uint8_t *c = C + (int64_t)j * d;
      int64_t p = 0;
      int32_t i = 0, alive = 1;
      for (int32_t D = d_front; D < d; D += step) {
        for (; i < D; ++i) {
          const int64_t t = (int64_t)x[i] - (int64_t)c[i];
          p += t * t;
        }
        const int first = D == d_front;
        tested += first;
        const float lim = tauf * (float)orc_prune_factor(D, d, eps0);
        if ((float)p > lim) {
          alive = 0;
          break;
        }
        passed += first;
      }
      if (!alive) continue;
      for (; i < d; ++i) {
        const int64_t t = (int64_t)x[i] - (int64_t)c[i];
        p += t * t;
      }
      ++full;
      if (p < bd || (p == bd && j < best)) {
        bd = p;
        best = j;
      }
    }
    a[r] = best;
    if (dist) dist[r] = bd;
  }
  if (counters) {
    counters[0] = tested;
    counters[1] = passed;
    counters[2] = full;
  }
}

void orc_sign1_prep(const float *C, int32_t k, int32_t d, const float *m, int32_t d0, int8_t *q,
                    float *sigma, int32_t *T, int32_t *Q, float *u) {
  const int32_t dt = d - d0;
  for (int32_t j = 0; j < k; ++j) {
    const float *c = C + (int64_t)j * d;
    float mx = 0.0f;
    for (int32_t i = d0; i < d; ++i) {
      float t = fabsf(c[i] - m[i]);
      if (t > mx) mx = t;
    }
    float s = mx > 0.0f ? mx / 127.0f : 1.0f;
    int32_t tsum = 0, qsum = 0;
    for (int32_t i = d0; i < d; ++i) {
      float t = mx > 0.0f ? rintf((c[i] - m[i]) / s) : 0.0f;
      if (t > 127.0f) t = 127.0f;
      if (t < -127.0f) t = -127.0f;
      int32_t qi = (int32_t)t;
      q[(int64_t)j * dt + (i - d0)] = (int8_t)qi;
      tsum += qi;
      qsum += qi * qi;
    }
    sigma[j] = s;
    T[j] = tsum;
    Q[j] = qsum;
    u[j] = (s * s) * (float)qsum;
  }
}

/* 1-bit score of one point against centroid j (Eq. 4 with the residual centroid in
 * symmetric int8): ||xhat - chat||^2 - alpha^2 d' = sigma^2 Q - 2 alpha sigma <2b-1, q>. */
static inline float sign1_score(const uint32_t *row, float alpha, int32_t d, int32_t d0,
                                const int8_t *qj, float sigma, int32_t T, float u) {
  int32_t D = 0;
  for (int32_t i = d0; i < d; ++i)
    if (bit_of(row, i)) D += qj[i - d0];
  int32_t s = 2 * D - T; /* <2b-1, q> = 2 (sum of q on set bits) - (sum of q) */
  float v = alpha * (2.0f * sigma);
  return fmaf(-v, (float)s, u);
}

static inline double sign1_decoded_dist(const uint32_t *row, float alpha, int32_t d, int32_t d0,
                                        const int8_t *qj, float sigma) {
  double e = 0.0;
  for (int32_t i = d0; i < d; ++i) {
    double xs = (double)alpha * (bit_of(row, i) ? 1.0 : -1.0);
    double cs = (double)sigma * (double)qj[i - d0];
    e += (xs - cs) * (xs - cs);
  }
  return e;
}

void orc_assign_sign1(const uint32_t *bits, const float *alpha, int64_t n, int32_t d, int32_t d0,
                      const int8_t *q, const float *sigma, const int32_t *T, const float *u,
                      int32_t k, int32_t *a, float *score, double *dist) {
  const int32_t W = d / 32, dt = d - d0;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    const uint32_t *row = bits + r * W;
    int32_t best = 0;
    float bs = 0.0f;
    for (int32_t j = 0; j < k; ++j) {
      float s = sign1_score(row, alpha[r], d, d0, q + (int64_t)j * dt, sigma[j], T[j], u[j]);
      if (j == 0 || s < bs) {
        bs = s;
        best = j;
      }
    }
    a[r] = best;
    if (score) score[r] = bs;
    if (dist) dist[r] = sign1_decoded_dist(row, alpha[r], d, d0, q + (int64_t)best * dt, sigma[best]);
  }
}

/* ------------------------------------------------------------------------ */
/* RabitQ with SQ4 centroid codes (Sec. 3.1, Eq. 3-5). */

void orc_rabitq_prep(const float *C, int32_t k, int32_t d, int8_t *q, float *s, float *b, int32_t *T,
                     float *N) {
  for (int32_t j = 0; j < k; ++j) {
    const float *c = C + (int64_t)j * d;
    float lo = c[0], hi = c[0];
    double nn = 0.0;
    for (int32_t i = 0; i < d; ++i) {
      if (c[i] < lo) lo = c[i];
      if (c[i] > hi) hi = c[i];
      nn += (double)c[i] * (double)c[i];
    }
    const float sc = hi > lo ? (hi - lo) / 15.0f : 1.0f;
    int32_t tsum = 0;
    for (int32_t i = 0; i < d; ++i) {
      float t = rintf((c[i] - lo) / sc);
      if (t < 0.0f) t = 0.0f;
      if (t > 15.0f) t = 15.0f;
      q[(int64_t)j * d + i] = (int8_t)t;
      tsum += (int32_t)t;
    }
    s[j] = sc;
    b[j] = lo;
    T[j] = tsum;
    N[j] = (float)nn;
  }
}

/* Eq. 5: <2 xbar - 1, b + s q> = s (2 D - T) + b (2 P - d), D = sum of q on set bits. */
static inline float rabitq_score(const uint32_t *row, float alpha, int32_t d, const int8_t *qj, float s,
                                 float b, int32_t T, float N) {
  int32_t D = 0, P = 0;
  for (int32_t i = 0; i < d; ++i)
    if (bit_of(row, i)) {
      D += qj[i];
      P += 1;
    }
  const float inner = fmaf(s, (float)(2 * D - T), b * (float)(2 * P - d));
  return fmaf(-(2.0f * alpha), inner, N);
}

void orc_assign_rabitq(const uint32_t *bits, const float *alpha, int64_t n, int32_t d, const int8_t *q,
                       const float *s, const float *b, const int32_t *T, const float *N, int32_t k,
                       int32_t *a, float *score, double *dist) {
  const int32_t W = d / 32;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    const uint32_t *row = bits + r * W;
    int32_t best = 0;
    float bs = 0.0f;
    for (int32_t j = 0; j < k; ++j) {
      const float sc = rabitq_score(row, alpha[r], d, q + (int64_t)j * d, s[j], b[j], T[j], N[j]);
      if (j == 0 || sc < bs) {
        bs = sc;
        best = j;
      }
    }
    a[r] = best;
    if (score) score[r] = bs;
    if (dist) dist[r] = (double)alpha[r] * (double)alpha[r] * (double)d + (double)bs;
  }
}

/* ------------------------------------------------------------------------ */
/* LVQ4 (Sec. 3.1, Eq. 1-2). */

void orc_lvq4_encode(const float *X, int64_t n, int32_t d, uint8_t *codes, float *par) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    const float *v = X + r * d;
    float lo = v[0], hi = v[0];
    for (int32_t i = 1; i < d; ++i) {
      if (v[i] < lo) lo = v[i];
      if (v[i] > hi) hi = v[i];
    }
    const float s = hi > lo ? (hi - lo) / 15.0f : 1.0f;
    int32_t S = 0, Q = 0;
    for (int32_t i = 0; i < d; ++i) {
      float t = rintf((v[i] - lo) / s);
      if (t < 0.0f) t = 0.0f;
      if (t > 15.0f) t = 15.0f;
      const int32_t c = (int32_t)t;
      codes[r * d + i] = (uint8_t)c;
      S += c;
      Q += c * c;
    }
    const float db = (float)d * lo;
    par[4 * r + 0] = s;
    par[4 * r + 1] = lo;
    par[4 * r + 2] = fmaf(s, (float)S, db);
    par[4 * r + 3] = fmaf(s * s, (float)Q, fmaf(2.0f * lo * s, (float)S, db * lo));
  }
}

void orc_lvq4_decode(const uint8_t *codes, const float *par, int64_t n, int32_t d, float *out) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r)
    for (int32_t i = 0; i < d; ++i) out[r * d + i] = fmaf(par[4 * r], (float)codes[r * d + i], par[4 * r + 1]);
}

void orc_assign_lvq4(const uint8_t *xc, const float *xpar, int64_t n, int32_t d, const uint8_t *yc,
                     const float *ypar, const int32_t *yS, int32_t k, int32_t *a, float *score, double *dist) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    const uint8_t *x = xc + r * d;
    const float sx = xpar[4 * r], bx = xpar[4 * r + 1], Ax = xpar[4 * r + 2];
    int32_t best = 0;
    float bs = 0.0f;
    for (int32_t j = 0; j < k; ++j) {
      const uint8_t *y = yc + (int64_t)j * d;
      int32_t dot = 0;
      for (int32_t i = 0; i < d; ++i) dot += (int32_t)x[i] * (int32_t)y[i];
      const float sy = ypar[4 * j], by = ypar[4 * j + 1], Ny = ypar[4 * j + 3];
      /* Eq. 2 without the point-only N_x: N_y - 2 (sx sy <xbar,ybar> + by A_x + bx sy S_y) */
      const float t = fmaf(bx * sy, (float)yS[j], fmaf(by, Ax, (sx * sy) * (float)dot));
      const float sc = fmaf(-2.0f, t, Ny);
      if (j == 0 || sc < bs) {
        bs = sc;
        best = j;
      }
    }
    a[r] = best;
    if (score) score[r] = bs;
    if (dist) dist[r] = (double)xpar[4 * r + 3] + (double)bs;
  }
}

void orc_assign_hybrid(const float *front, const uint32_t *bits, const float *alpha, int64_t n,
                       int32_t d, int32_t d0, const float *C, const int8_t *q, const float *sigma,
                       const int32_t *T, const float *u, int32_t k, int32_t *a, double *dist) {
  const int32_t W = d / 32, dt = d - d0;
  double *cn = (double *)malloc(sizeof(double) * (size_t)k);
  for (int32_t j = 0; j < k; ++j) {
    double s = 0.0;
    for (int32_t i = 0; i < d0; ++i) s += (double)C[(int64_t)j * d + i] * (double)C[(int64_t)j * d + i];
    cn[j] = s;
  }
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    const float *x = front + r * d0;
    const uint32_t *row = bits + r * W;
    int32_t best = 0;
    double bs = 0.0;
    for (int32_t j = 0; j < k; ++j) {
      /* segment decomposition: ||x-y||^2 = ||x'-y'||^2 + ||x''-y''||^2 (Sec. 3.1, SuperKMeans) */
      double dot = 0.0;
      for (int32_t i = 0; i < d0; ++i) dot += (double)x[i] * (double)C[(int64_t)j * d + i];
      double s = cn[j] - 2.0 * dot +
                 (double)sign1_score(row, alpha[r], d, d0, q + (int64_t)j * dt, sigma[j], T[j], u[j]);
      if (j == 0 || s < bs) {
        bs = s;
        best = j;
      }
    }
    a[r] = best;
    if (dist) {
      double e = 0.0;
      for (int32_t i = 0; i < d0; ++i) {
        double t = (double)x[i] - (double)C[(int64_t)best * d + i];
        e += t * t;
      }
      dist[r] = e + sign1_decoded_dist(row, alpha[r], d, d0, q + (int64_t)best * dt, sigma[best]);
    }
  }
  free(cn);
}

/* ------------------------------------------------------------------------ */
/* STEP 3 (Sec. 2.3): averaging; clusters left empty take half of a large cluster. */

static void count_members(const int32_t *a, int64_t n, int32_t k, int64_t *cnt) {
  for (int32_t j = 0; j < k; ++j) cnt[j] = 0;
  for (int64_t r = 0; r < n; ++r)
    if (a[r] >= 0 && a[r] < k) cnt[a[r]]++;
}

/* Donor for an empty cluster: the largest current count, ties to the smallest index. */
static int32_t donor_of(const int64_t *cnt, int32_t k) {
  int32_t b = 0;
  for (int32_t j = 1; j < k; ++j)
    if (cnt[j] > cnt[b]) b = j;
  return b;
}

/* Split on clustering-space vectors Z (k x d): for empty j in ascending order, with donor b
 * of count >= 2: Z_j = Z_b (1 + eps p), Z_b = Z_b (1 - eps p), p_i = (-1)^i, eps = 2^-10.
 * fresh[j] marks rows that now hold a new value. */
static void split_float(float *Z, int32_t k, int32_t d, const int64_t *cnt0, uint8_t *fresh) {
  int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
  memcpy(cnt, cnt0, sizeof(int64_t) * (size_t)k);
  const float up = 1.0f + 0x1p-10f, dn = 1.0f - 0x1p-10f;
  for (int32_t j = 0; j < k; ++j) {
    if (cnt0[j] != 0) continue;
    int32_t b = donor_of(cnt, k);
    if (cnt[b] < 2) continue;
    for (int32_t i = 0; i < d; ++i) {
      float t = Z[(int64_t)b * d + i];
      int even = (i % 2) == 0;
      Z[(int64_t)j * d + i] = t * (even ? up : dn);
      Z[(int64_t)b * d + i] = t * (even ? dn : up);
    }
    cnt[j] = cnt[b] / 2;
    cnt[b] = cnt[b] - cnt[j];
    fresh[j] = 1;
  }
  free(cnt);
}

static void split_codes(uint8_t *Z, int32_t k, int32_t d, const int64_t *cnt0, uint8_t *fresh) {
  int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
  memcpy(cnt, cnt0, sizeof(int64_t) * (size_t)k);
  for (int32_t j = 0; j < k; ++j) {
    if (cnt0[j] != 0) continue;
    int32_t b = donor_of(cnt, k);
    if (cnt[b] < 2) continue;
    for (int32_t i = 0; i < d; ++i) {
      int t = Z[(int64_t)b * d + i];
      int p = (i % 2) == 0 ? 1 : -1;
      int up = t + p, dn = t - p;
      Z[(int64_t)j * d + i] = (uint8_t)(up < 0 ? 0 : up > 255 ? 255 : up);
      Z[(int64_t)b * d + i] = (uint8_t)(dn < 0 ? 0 : dn > 255 ? 255 : dn);
    }
    cnt[j] = cnt[b] / 2;
    cnt[b] = cnt[b] - cnt[j];
    fresh[j] = 1;
  }
  free(cnt);
}

void orc_update_f32(const float *X, int64_t n, int32_t d, int64_t ldx, const int32_t *a, int32_t k,
                    float *C, int64_t *counts, int32_t policy) {
  int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
  double *S = (double *)calloc((size_t)k * (size_t)d, sizeof(double));
  float *Z = (float *)malloc(sizeof(float) * (size_t)k * (size_t)d);
  uint8_t *fresh = (uint8_t *)calloc((size_t)k, 1);
  count_members(a, n, k, cnt);
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < d; ++i)
    for (int64_t r = 0; r < n; ++r)
      if (a[r] >= 0 && a[r] < k) S[(int64_t)a[r] * d + i] += (double)X[r * ldx + i];
  for (int32_t j = 0; j < k; ++j) {
    fresh[j] = cnt[j] > 0;
    for (int32_t i = 0; i < d; ++i)
      Z[(int64_t)j * d + i] = cnt[j] > 0 ? (float)(S[(int64_t)j * d + i] / (double)cnt[j]) : 0.0f;
  }
  if (policy == ORC_EMPTY_SPLIT) split_float(Z, k, d, cnt, fresh);
  for (int32_t j = 0; j < k; ++j)
    if (fresh[j]) memcpy(C + (int64_t)j * d, Z + (int64_t)j * d, sizeof(float) * (size_t)d);
  if (counts) memcpy(counts, cnt, sizeof(int64_t) * (size_t)k);
  free(cnt);
  free(S);
  free(Z);
  free(fresh);
}

void orc_update_lvq4(const uint8_t *xc, const float *xpar, int64_t n, int32_t d, const int32_t *a, int32_t k,
                     float *C, int64_t *counts, int32_t policy) {
  int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
  double *S = (double *)calloc((size_t)k * (size_t)d, sizeof(double));
  float *Z = (float *)malloc(sizeof(float) * (size_t)k * (size_t)d);
  uint8_t *fresh = (uint8_t *)calloc((size_t)k, 1);
  count_members(a, n, k, cnt);
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < d; ++i)
    for (int64_t r = 0; r < n; ++r)
      if (a[r] >= 0 && a[r] < k)
        S[(int64_t)a[r] * d + i] += (double)fmaf(xpar[4 * r], (float)xc[r * d + i], xpar[4 * r + 1]);
  for (int32_t j = 0; j < k; ++j) {
    fresh[j] = cnt[j] > 0;
    for (int32_t i = 0; i < d; ++i)
      Z[(int64_t)j * d + i] = cnt[j] > 0 ? (float)(S[(int64_t)j * d + i] / (double)cnt[j]) : 0.0f;
  }
  if (policy == ORC_EMPTY_SPLIT) split_float(Z, k, d, cnt, fresh);
  for (int32_t j = 0; j < k; ++j)
    if (fresh[j]) memcpy(C + (int64_t)j * d, Z + (int64_t)j * d, sizeof(float) * (size_t)d);
  if (counts) memcpy(counts, cnt, sizeof(int64_t) * (size_t)k);
  free(cnt);
  free(S);
  free(Z);
  free(fresh);
}

void orc_update_sq8(const uint8_t *X, int64_t n, int32_t d, const int32_t *a, int32_t k, uint8_t *C,
                    int64_t *counts, int32_t policy) {
  int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
  int64_t *S = (int64_t *)calloc((size_t)k * (size_t)d, sizeof(int64_t));
  uint8_t *Z = (uint8_t *)malloc((size_t)k * (size_t)d);
  uint8_t *fresh = (uint8_t *)calloc((size_t)k, 1);
  count_members(a, n, k, cnt);
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < d; ++i)
    for (int64_t r = 0; r < n; ++r)
      if (a[r] >= 0 && a[r] < k) S[(int64_t)a[r] * d + i] += X[r * d + i];
  for (int32_t j = 0; j < k; ++j) {
    fresh[j] = cnt[j] > 0;
    for (int32_t i = 0; i < d; ++i) {
      /* averaging in the quantised domain, rounded half up: floor((2S + n) / (2n)) */
      int64_t v = cnt[j] > 0 ? (2 * S[(int64_t)j * d + i] + cnt[j]) / (2 * cnt[j]) : 0;
      Z[(int64_t)j * d + i] = (uint8_t)v;
    }
  }
  if (policy == ORC_EMPTY_SPLIT) split_codes(Z, k, d, cnt, fresh);
  for (int32_t j = 0; j < k; ++j)
    if (fresh[j]) memcpy(C + (int64_t)j * d, Z + (int64_t)j * d, (size_t)d);
  if (counts) memcpy(counts, cnt, sizeof(int64_t) * (size_t)k);
  free(cnt);
  free(S);
  free(Z);
  free(fresh);
}

void orc_update_sign1(const float *front, const uint32_t *bits, const float *alpha, int64_t n,
                      int32_t d, int32_t d0, const float *m, const int32_t *a, int32_t k, float *C,
                      int64_t *counts, int32_t policy) {
  const int32_t W = d / 32;
  int64_t *cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
  double *S = (double *)calloc((size_t)k * (size_t)d, sizeof(double));
  float *Z = (float *)malloc(sizeof(float) * (size_t)k * (size_t)d);
  uint8_t *fresh = (uint8_t *)calloc((size_t)k, 1);
  count_members(a, n, k, cnt);
  /* fused decode-averaging: sum of alpha_x (2 b_x - 1) per dim; the front dims sum x' */
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < d; ++i)
    for (int64_t r = 0; r < n; ++r) {
      if (a[r] < 0 || a[r] >= k) continue;
      double v = i < d0 ? (double)front[r * d0 + i]
                        : (bit_of(bits + r * W, i) ? (double)alpha[r] : -(double)alpha[r]);
      S[(int64_t)a[r] * d + i] += v;
    }
  for (int32_t j = 0; j < k; ++j) {
    fresh[j] = cnt[j] > 0;
    for (int32_t i = 0; i < d; ++i)
      Z[(int64_t)j * d + i] = cnt[j] > 0 ? (float)(S[(int64_t)j * d + i] / (double)cnt[j]) : 0.0f;
  }
  /* the split acts on the clustering-space vector: front values and tail residuals */
  if (policy == ORC_EMPTY_SPLIT) split_float(Z, k, d, cnt, fresh);
  for (int32_t j = 0; j < k; ++j) {
    if (!fresh[j]) continue;
    for (int32_t i = 0; i < d; ++i)
      C[(int64_t)j * d + i] = i < d0 ? Z[(int64_t)j * d + i] : m[i] + Z[(int64_t)j * d + i];
  }
  if (counts) memcpy(counts, cnt, sizeof(int64_t) * (size_t)k);
  free(cnt);
  free(S);
  free(Z);
  free(fresh);
}

/* ------------------------------------------------------------------------ */

double orc_cost_f32(const float *X, int64_t n, int32_t d, int64_t ldx, const float *C,
                    const int32_t *a) {
  double tot = 0.0;
  for (int64_t r = 0; r < n; ++r) {
    double e = 0.0;
    for (int32_t i = 0; i < d; ++i) {
      double t = (double)X[r * ldx + i] - (double)C[(int64_t)a[r] * d + i];
      e += t * t;
    }
    tot += e;
  }
  return tot;
}

double orc_partition_cost(const float *X, int64_t n, int32_t d, const int32_t *a, int32_t k) {
  int64_t *cnt = (int64_t *)calloc((size_t)k, sizeof(int64_t));
  double *S = (double *)calloc((size_t)k * (size_t)d, sizeof(double));
  for (int64_t r = 0; r < n; ++r) {
    cnt[a[r]]++;
    for (int32_t i = 0; i < d; ++i) S[(int64_t)a[r] * d + i] += (double)X[r * d + i];
  }
  for (int32_t j = 0; j < k; ++j)
    for (int32_t i = 0; i < d; ++i)
      if (cnt[j]) S[(int64_t)j * d + i] /= (double)cnt[j];
  double tot = 0.0;
  for (int64_t r = 0; r < n; ++r)
    for (int32_t i = 0; i < d; ++i) {
      double t = (double)X[r * d + i] - S[(int64_t)a[r] * d + i];
      tot += t * t;
    }
  free(cnt);
  free(S);
  return tot;
}
