/*
 * kmq_oracle.h -- plain, slow CPU oracle for Lloyd k-means on compressed vectors.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes or
 * calls this code; only the test-suite, the smoke check and the CPU-baseline leg
 * of the benchmark do.  It shares no source with the HIP library.
 *
 * Every routine is written from the paper's definitions (Sec. 2.3 STEPs 1-3,
 * Sec. 3.1 SQ / RabitQ / PCA / segment decomposition), with fp64 accumulation
 * for floating point and exact integers for the integer paths.  Where a float
 * decides an integer (a quantised code, a 1-bit score) the oracle takes that
 * decision in the same fp32 operation order as the product, so both sides can
 * be compared bit for bit.
 *
 * Layouts: all matrices are row-major.  1-bit codes: bit i of a vector lives in
 * 32-bit word i/32 at bit position i%32 (LSB first); a row holds d/32 words.
 * Dimension ranges [d0, d) select the tail used by the hybrid (front fp32 +
 * 1-bit tail) scheme; d0 = 0 means the whole vector.
 */
#ifndef KMQ_ORACLE_H
#define KMQ_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Empty-cluster policies. */
#define ORC_EMPTY_SPLIT 0
#define ORC_EMPTY_KEEP 1

/* ---- Preprocessing (Sec. 3.1) ---------------------------------------- */

/* SQ8 parameters per dimension: lo_i = min_x x_i, hi_i = max_x x_i. */
void orc_sq8_fit(const float *X, int64_t n, int32_t d, float *lo, float *hi);
/* SQ8 codes: inv_i = 255/(hi_i-lo_i) (0 if hi_i==lo_i), code = clip(rint((x-lo)*inv),0,255). */
void orc_sq8_encode(const float *X, int64_t n, int32_t d, const float *lo, const float *hi,
                    uint8_t *codes);
/* Column mean m (fp64 sum, fp32 result). */
void orc_col_mean(const float *X, int64_t n, int32_t d, float *m);
/* 1-bit sign codes of r = x - m over all d dims, and the per-vector scale
 * alpha = sum r_i^2 / sum |r_i| over dims [d0, d) (0 if the denominator is 0). */
void orc_sign1_encode(const float *X, int64_t n, int32_t d, const float *m, int32_t d0,
                      uint32_t *bits, float *alpha);
/* PCA statistics: mean (fp64) and covariance (1/n) sum (x-mu)(x-mu)^T (fp64, d x d). */
void orc_pca_cov(const float *X, int64_t n, int32_t d, double *mean, double *cov);
/* One covariance entry (i, j) in fp64, for sampled checks of large inputs. */
double orc_pca_cov_entry(const float *X, int64_t n, int32_t d, const double *mean, int32_t i,
                         int32_t j);
/* Projection Y = (X - mean) W, W is d x dout row-major; fp64 sums, fp32 output. */
void orc_project(const float *X, int64_t n, int32_t d, const float *mean, const float *W,
                 int32_t dout, float *Y);

/* 16-bit storage of full-precision vectors (Sec. 2.4): bfloat16, i.e. the fp32
 * exponent range with 8 significant bits.  Each value is rounded to the nearest
 * bfloat16, ties to the even significand; the result is returned as its 16-bit
 * pattern (the top half of the rounded value's fp32 pattern).  NaN stays NaN;
 * magnitudes that round past the largest bfloat16 become infinities. */
void orc_bf16_round(const float *X, int64_t n, uint16_t *out);

/* ---- STEP 2: assignment (ties go to the smallest centroid index) ------- */

/* fp32 points: a = argmin_j ||c_j||^2 - 2<x,c_j> (fp64), dist = ||x - c_a||^2 (fp64). */
void orc_assign_f32(const float *X, int64_t n, int32_t d, int64_t ldx, const float *C, int32_t k,
                    int32_t *a, double *dist);
/* SQ8 codes, code-space L2 with exact integers: dist = sum (x-c)^2. */
void orc_assign_sq8(const uint8_t *X, int64_t n, int32_t d, const uint8_t *C, int32_t k, int32_t *a,
                    int64_t *dist);
/* Per-centroid symmetric int8 quantisation of the centroid residual c - m over dims [d0,d):
 * sigma_j = max|c-m|/127 (1 if that max is 0), q = clip(rint((c-m)/sigma), -127, 127),
 * T_j = sum q, Q_j = sum q^2, u_j = (sigma_j*sigma_j)*Q_j (fp32).  q is k x (d-d0). */
void orc_sign1_prep(const float *C, int32_t k, int32_t d, const float *m, int32_t d0, int8_t *q,
                    float *sigma, int32_t *T, int32_t *Q, float *u);
/* 1-bit scores over dims [d0,d): D = sum of q on set bits, s = 2D - T (exact),
 * score = fmaf(-(alpha*(2*sigma)), s, u) in fp32.  Writes a and the winning score.
 * If dist != NULL it also writes the decoded-point distance (fp64):
 * sum_i (alpha(2b_i-1) - sigma q_i)^2. */
void orc_assign_sign1(const uint32_t *bits, const float *alpha, int64_t n, int32_t d, int32_t d0,
                      const int8_t *q, const float *sigma, const int32_t *T, const float *u,
                      int32_t k, int32_t *a, float *score, double *dist);
/* Hybrid: exact fp32-input L2 on the front dims [0,d0) (fp64) plus the 1-bit score on
 * [d0,d).  front is n x d0, C is k x d.  dist = ||x'-c'||^2 + decoded tail distance. */
void orc_assign_hybrid(const float *front, const uint32_t *bits, const float *alpha, int64_t n,
                       int32_t d, int32_t d0, const float *C, const int8_t *q, const float *sigma,
                       const int32_t *T, const float *u, int32_t k, int32_t *a, double *dist);

/* RabitQ as the paper runs it (Sec. 3.1, Eq. 3-5), on 1-bit codes of the rotated,
 * centred residual (centre 0 in the rotated space).  Centroid residuals are coded
 * with a per-centroid SQ4: b_j = min_i c_ji, s_j = (max_i c_ji - b_j) / 15 (1 when
 * the range is 0), q_ji = clip(rint((c_ji - b_j) / s_j), 0, 15) in fp32;
 * T_j = sum q, N_j = ||c_j||^2 (fp64 sum, fp32 result). */
void orc_rabitq_prep(const float *C, int32_t k, int32_t d, int8_t *q, float *s, float *b, int32_t *T,
                     float *N);
/* Eq. 4-5: with D = sum of q on set bits, P = number of set bits,
 * inner = fmaf(s_j, 2D - T_j, b_j * (2P - d)) and score = fmaf(-(2 alpha), inner, N_j),
 * fp32 in this order (alpha = ||x_r - m|| / (sqrt(d) <xbar, x>)).  Ties go to the
 * smallest index.  dist (nullable) = alpha^2 d + score in fp64, the estimated squared
 * distance with the decoded point's norm in place of ||x_r - m||^2. */
void orc_assign_rabitq(const uint32_t *bits, const float *alpha, int64_t n, int32_t d, const int8_t *q,
                       const float *s, const float *b, const int32_t *T, const float *N, int32_t k,
                       int32_t *a, float *score, double *dist);

/* LVQ4 (Sec. 3.1 LVQ, Eq. 1-2): each vector (point or centroid) v is coded with its
 * own bias b = min_i v_i and scale s = (max_i v_i - b) / 15 (1 when the range is 0),
 * code_i = clip(rint((v_i - b) / s), 0, 15) in fp32; S = sum code, Q = sum code^2
 * (exact), and in fp32, in this order: A = fmaf(s, S, d * b),
 * N = fmaf(s * s, Q, fmaf(2 * b * s, S, d * b * b)).  codes: uint8[n][d] (one code per
 * byte; the product packs two per byte), par: float[n][4] = (s, b, A, N).
 * Decoding is fmaf(s, code, b). */
void orc_lvq4_encode(const float *X, int64_t n, int32_t d, uint8_t *codes, float *par);
/* Decoding: out = fmaf(s, code, b) per value (fp32). */
void orc_lvq4_decode(const uint8_t *codes, const float *par, int64_t n, int32_t d, float *out);
/* Eq. 2 for the argmin: score = fmaf(-2, fmaf(bx * sy, Sy, fmaf(by, Ax, (sx * sy) * dot)), Ny)
 * with dot = <xbar, ybar> exact; fp32 in this order.  dist (nullable) = Nx + score (fp64). */
void orc_assign_lvq4(const uint8_t *xc, const float *xpar, int64_t n, int32_t d, const uint8_t *yc,
                     const float *ypar, const int32_t *yS, int32_t k, int32_t *a, float *score, double *dist);
/* Update: c_j = (1/n_j) sum of the decoded members fmaf(s, code, b) (fp64 sums, fp32 result),
 * empty-cluster split as for fp32 points. */
void orc_update_lvq4(const uint8_t *xc, const float *xpar, int64_t n, int32_t d, const int32_t *a, int32_t k,
                     float *C, int64_t *counts, int32_t policy);

/* ---- STEP 3: update (mean of members, empty-cluster split) ------------- */

/* fp32 points: c_j = mean of members (fp64 sums, fp32 result).  counts = member counts. */
void orc_update_f32(const float *X, int64_t n, int32_t d, int64_t ldx, const int32_t *a, int32_t k,
                    float *C, int64_t *counts, int32_t policy);
/* SQ8: c_j = floor((2 S + n_j) / (2 n_j)) per dim, S = exact sum of member codes. */
void orc_update_sq8(const uint8_t *X, int64_t n, int32_t d, const int32_t *a, int32_t k, uint8_t *C,
                    int64_t *counts, int32_t policy);
/* 1-bit (dims [d0,d)) and, for d0>0, fp32 front (dims [0,d0) from `front`, n x d0):
 * tail residual = (1/n_j) sum alpha_x (2b_x - 1), c = m + residual (fp32). */
void orc_update_sign1(const float *front, const uint32_t *bits, const float *alpha, int64_t n,
                      int32_t d, int32_t d0, const float *m, const int32_t *a, int32_t k, float *C,
                      int64_t *counts, int32_t policy);

/* Decoding of a 1-bit row (dims [d0,d)): out_i = m_i + alpha*(2b_i-1) in fp32. */
void orc_sign1_decode(const uint32_t *bits, const float *alpha, int64_t n, int32_t d, int32_t d0,
                      const float *m, float *out, int64_t ldo);

/* ---- Dimension pruning (Sec. 3.1 SuperKMeans; ADSampling test) ----------- */

/* Factor of the ADSampling test at a checkpoint after D of d dims: a candidate
   whose squared distance over the first D dims is p is dropped when
   p > tau * r, r = (1 + eps0 / sqrt(D))^2 * D / d, tau = the squared distance to
   the point's previous centroid (the current best). */
double orc_prune_factor(int32_t D, int32_t d, double eps0);

/* One pruned STEP 2: for every point, best = prev[r] at distance tau; every other
   centroid j is tested at the checkpoints d_front, d_front + step, ... (< d) on
   its partial squared distance and, if never dropped, compared on its full
   distance (smaller wins, ties to the smaller index).  fp32 points: sums and the
   test in fp64.  SQ8 codes: exact integer sums, test (float)p > (float)tau *
   (float)r.  dist: the winning squared distance.  counters (nullable, int64[3]):
   candidates tested at d_front, candidates that passed it, candidates compared on
   the full distance. */
void orc_assign_pruned_f32(const float *X, int64_t n, int32_t d, const float *C, int32_t k, const int32_t *prev,
                           double eps0, int32_t d_front, int32_t step, int32_t *a, double *dist,
                           int64_t *counters);
void orc_assign_pruned_sq8(const uint8_t *X, int64_t n, int32_t d, const uint8_t *C, int32_t k,
                           const int32_t *prev, double eps0, int32_t d_front, int32_t step, int32_t *a,
                           int64_t *dist, int64_t *counters);

/* ---- Objective ---------------------------------------------------------- */

/* Sum over points of ||x - c_{a(x)}||^2 in fp64 (fp32 inputs). */
double orc_cost_f32(const float *X, int64_t n, int32_t d, int64_t ldx, const float *C,
                    const int32_t *a);
/* Full-precision partition cost: sum ||x - mu_{a(x)}||^2, mu = fp64 member means. */
double orc_partition_cost(const float *X, int64_t n, int32_t d, const int32_t *a, int32_t k);

int orc_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
