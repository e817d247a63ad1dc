/*
 * kmq.h -- C ABI of the MI355X (gfx950) library for Lloyd k-means on vectors
 * compressed before clustering ("approximate first, then cluster", Sec. 3).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Buffers are caller-owned DEVICE pointers (memory of the current HIP
 *   device) unless a parameter says "host".  The library never frees or keeps
 *   a caller pointer after the call returns.
 * - Every call is asynchronous on `stream` (a hipStream_t; NULL = the legacy
 *   default stream): results are valid once the stream has synchronised.
 * - All argument checks run on the host before any allocation or launch, so a
 *   non-OK status means nothing was written.  Assignment values read from
 *   device memory are range-checked inside the kernels: an index outside
 *   [0, k) makes that point belong to no cluster (it is skipped).
 * - Internal scratch memory is taken from the device's stream-ordered pool
 *   (hipMallocAsync on `stream`) and given back on the same stream before the
 *   call returns; km_release() trims the pool.  Calls on different streams
 *   do not share scratch.
 * - No exception crosses the ABI.  km_last_error() gives a thread-local
 *   message for the last non-OK status of the calling thread.
 * - Layouts are row-major.  1-bit codes: bit i of a vector sits in 32-bit
 *   word i/32 at bit position i%32 (least significant first); a row holds
 *   d/32 words.
 */
#ifndef KMQ_H
#define KMQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

struct ihipStream_t;                     /* = hipStream_t */
typedef struct ihipStream_t *km_stream;  /* hipStream_t */

typedef enum {
  KM_OK = 0,
  KM_EINVAL = -1,       /* bad argument (null pointer, bad size, bad alignment, ...) */
  KM_EUNSUPPORTED = -2, /* format not valid for this call */
  KM_ENOMEM = -3,       /* scratch allocation failed */
  KM_EDEVICE = -4       /* a HIP runtime error (message from hipGetErrorString) */
} km_status;

typedef enum {
  KM_F32 = 0,    /* fp32 vectors (raw, PCA-projected or a dimension prefix) */
  KM_BF16 = 1,   /* bfloat16 vectors (16-bit storage of full-precision vectors, Sec. 2.4) */
  KM_SQ8 = 2,    /* uint8 scalar-quantised codes, one (lo, hi) pair per dimension */
  KM_SIGN1 = 3,  /* 1-bit sign codes of x - m plus one fp32 scale alpha per vector */
  KM_HYBRID = 4, /* fp32 front dims [0, d_front) + 1-bit codes on the tail [d_front, d) */
  KM_RABITQ = 5, /* 1-bit codes of the randomly rotated, centred residual; SQ4 centroid codes */
  KM_LVQ4 = 6    /* 4-bit codes with a per-vector scale and bias (LVQ) */
} km_format;

typedef enum {
  KM_EMPTY_SPLIT = 0, /* an empty cluster takes half of the largest cluster */
  KM_EMPTY_KEEP = 1   /* an empty cluster keeps its previous centroid */
} km_empty_policy;

/* quantize() flags */
#define KM_Q_FIT_PARAMS 1 /* compute the parameters from X; otherwise use those passed in */

/*
 * The points being clustered, in their compressed form.
 *   KM_F32:    data = float[n][ld], d <= ld, ld % 4 == 0, data 16-byte aligned, d % 4 == 0.
 *   KM_BF16:   data = bfloat16 (uint16 bit patterns)[n][ld], d <= ld, ld % 8 == 0,
 *              d % 8 == 0, 16-byte aligned.
 *   KM_SQ8:    data = uint8[n][ld] codes, ld % 16 == 0, d % 16 == 0, 16-byte aligned.
 *   KM_SIGN1:  data = uint32[n][d/32] bits, d % 32 == 0; alpha = float[n];
 *              center = m, float[d] (the mean the codes were taken around).
 *   KM_HYBRID: data = uint32[n][d/32] bits of the FULL d dims (only words
 *              d_front/32 .. d/32-1 are read); alpha = float[n] computed over the
 *              tail dims; center = float[d]; front = float[n][d_front];
 *              d_front % 32 == 0, 0 < d_front < d.
 *   KM_RABITQ: data = uint32[n][d/32] bits of y = (x - m) P, the centred residual
 *              rotated by an orthogonal d x d matrix P (Sec. 3.1 RabitQ; see
 *              rabitq_encode), alpha = float[n] = ||y||^2 / ||y||_1, center must be
 *              NULL (the codes are of the residual: the clustering space is the
 *              rotated residual space, centre 0).  d % 32 == 0.
 *   KM_LVQ4:   data = uint8[n][ld] codes, two per byte (dim 2i in the low nibble, dim
 *              2i+1 in the high one), ld >= d/2, ld % 16 == 0, d % 32 == 0, 16-byte
 *              aligned; vparams = float[n][4] per vector (s, b, A, N): scale, bias,
 *              A = fmaf(s, S, d b) and N = fmaf(s s, Q, fmaf(2 b s, S, (d b) b)) with S,
 *              Q the sum and the sum of squares of its codes (as quantize writes them).
 * `ld` is ignored for the 1-bit formats.
 * raw (nullable): fp32 rows of the same points in the clustering space (the
 *   original vectors for KM_SIGN1 / KM_HYBRID / KM_BF16, the rotated residual y for
 *   KM_RABITQ), float[n][raw_ld], raw_ld >= d, raw_ld % 4 == 0, d % 4 == 0,
 *   16-byte aligned.  kmeans_fit then computes its last update from these rows
 *   (the raw-vector last iteration of Sec. 4.1).  Not allowed for KM_SQ8.
 */
typedef struct km_points {
  int32_t fmt;          /* km_format */
  int32_t d;            /* logical dimensionality */
  int64_t n;            /* number of points, 1 <= n < 2^31 */
  const void *data;
  int64_t ld;           /* row stride in elements (F32: floats, BF16: 16-bit values, SQ8 and LVQ4: bytes) */
  const float *alpha;
  const float *center;
  const float *front;
  int32_t d_front;
  int32_t reserved;     /* must be 0 */
  const float *raw;     /* nullable, see above */
  int64_t raw_ld;       /* row stride of raw in floats */
  const float *vparams; /* KM_LVQ4: per-vector (s, b, A, N), float[n][4]; NULL otherwise */
} km_points;

/*
 * quantize -- compress fp32 points before clustering (Sec. 3.1).
 *   X: float[n][ldx] (ldx % 4 == 0, 16-byte aligned).
 *   fmt == KM_SQ8 (Sec. 3.1 "SQ8"): per-dimension bias lo_i and scale
 *     (hi_i - lo_i)/255; codes = uint8[n][d] with
 *     code = clip(rint((x - lo) * (255 / (hi - lo))), 0, 255) in fp32 (0 where hi == lo);
 *     params = float[2*d]: lo[0..d) then hi[0..d).  d % 16 == 0.
 *   fmt == KM_SIGN1 (Sec. 3.1 "RabitQ", without the random rotation):
 *     params = m, float[d] (column mean, fp64 sums); codes = uint32[n][d/32] with
 *     bit i = [x_i - m_i > 0]; alpha = float[n], alpha = sum r_i^2 / sum |r_i| over
 *     dims [d_front, d) with r = x - m (fp64 sums; 0 when x == m on those dims).
 *     alpha equals (1/sqrt(d')) ||r|| / <x_bar, x> of Eq. 4, the decoding radius.
 *     If d_front > 0 and front != NULL, front = float[n][d_front] receives a copy
 *     of the first d_front dims (the hybrid layout).  d % 32 == 0, d_front % 32 == 0;
 *     params and front 16-byte aligned.
 *   fmt == KM_LVQ4 (Sec. 3.1 LVQ, B = 4): per vector b = min_i x_i, s = (max_i x_i - b)/15
 *     (1 when the range is 0), code_i = clip(rint((x_i - b)/s), 0, 15) in fp32; codes =
 *     uint8[n][d/2] packed as in km_points; params = float[n][4] receives (s, b, A, N).
 *     d % 32 == 0; alpha, front unused; flags ignored.
 *   fmt == KM_BF16 (16-bit storage, Sec. 2.4): codes = bfloat16[n][d], each value
 *     rounded to the nearest bfloat16 with ties to the even significand (NaN stays
 *     NaN, overflow gives infinities).  params, alpha, front: unused (may be NULL);
 *     d % 8 == 0, d_front == 0, flags ignored.
 *   flags & KM_Q_FIT_PARAMS: compute params from X first (one extra pass over X);
 *     otherwise params are inputs.
 */
km_status quantize(const float *X, int64_t n, int32_t d, int64_t ldx, int32_t fmt, void *codes,
                   float *params, float *alpha, int32_t d_front, float *front, int32_t flags,
                   km_stream stream);

/*
 * rabitq_encode -- RabitQ codes (Sec. 3.1 RabitQ): y = (x - m) P for an orthogonal
 * P, then bit i = [y_i > 0] and alpha = ||y||^2 / ||y||_1 (fp64 sums; 0 when y = 0),
 * which is ||x - m|| / (sqrt(d) <xbar, x>) of Eq. 4.
 *   X: float[n][ldx] (ldx % 4 == 0, 16-byte aligned); P: float[d][d] row-major (the
 *   caller draws it; the library does not check orthogonality); m: float[d], the
 *   centre: computed as the column mean (fp64 sums) when flags & KM_Q_FIT_PARAMS,
 *   else an input.  bits: uint32[n][d/32]; alpha: float[n].  d % 32 == 0.
 *   Y (nullable): float[n][d], receives the rotated residual rows y (the raw rows
 *   of a kmeans_fit last update); when NULL they live in scratch for the call.
 */
km_status rabitq_encode(const float *X, int64_t n, int32_t d, int64_t ldx, const float *P, float *m,
                        uint32_t *bits, float *alpha, float *Y, int32_t flags, km_stream stream);

/*
 * pca_fit_cov -- PCA statistics (Sec. 3.1 PCA; Sec. 4.2): mean = float[d] column
 * mean, cov = float[d][d] = (1/n) sum (x - mean)(x - mean)^T (symmetric, both
 * halves written).  X: float[n][d], d % 4 == 0.  The eigendecomposition of cov
 * (d x d, small) is done by the caller on the host.
 */
km_status pca_fit_cov(const float *X, int64_t n, int32_t d, float *mean, float *cov, km_stream stream);

/*
 * pca_project -- Y = (X - mean) W: X float[n][d], mean float[d], W float[d][d_out]
 * (columns = principal directions), Y float[n][d_out].  d % 4 == 0, d_out % 4 == 0.
 */
km_status pca_project(const float *X, int64_t n, int32_t d, const float *mean, const float *W,
                      int32_t d_out, float *Y, km_stream stream);

/*
 * kmeans_assign -- STEP 2 (Sec. 2.3): for every point, the index of the nearest
 * centroid (ties to the smallest index), without materialising the n x k
 * distance matrix.
 *   C: centroids in the clustering space, k x d, row-major:
 *      KM_F32 / KM_BF16: float; KM_SQ8: uint8 codes; KM_SIGN1 / KM_HYBRID: float in
 *      the original space (the 1-bit part is compared against int8 residual codes
 *      q = rint((c - m)/sigma), sigma = max|c - m|/127, rebuilt on each call);
 *      KM_RABITQ: float in the rotated residual space, coded on each call with a
 *      per-centroid SQ4 (Eq. 5): b = min_i c_i, s = (max_i c_i - b)/15 (1 when the
 *      range is 0), q = clip(rint((c - b)/s), 0, 15); KM_LVQ4: float, coded on each
 *      call with LVQ4 like the points.
 *      KM_BF16 compares the points with the centroids rounded to bfloat16 (nearest,
 *      ties to even), products exact, fp32 accumulation.
 *   assign: int32[n].  score (nullable): float[n], the winning score, i.e. the
 *      in-space squared distance minus the point-only term:
 *      F32: ||c||^2 - 2<x,c>;  BF16: the same on the bfloat16 values;
 *      SQ8: ||c~||^2 - 2<x~,c~> with x~ = code - 128;
 *      SIGN1: fmaf(-alpha*2*sigma, <2b-1, q>, sigma^2 ||q||^2);
 *      HYBRID: front F32 score + tail SIGN1 score;
 *      LVQ4 (Eq. 2 without N_x): fmaf(-2, fmaf(b_x s_y, S_y, fmaf(b_y, A_x,
 *      (s_x s_y) <xbar, ybar>)), N_y), fp32 in this order;
 *      RABITQ (Eq. 4-5): fmaf(-2 alpha, fmaf(s, 2D - T, b (2P - d)), ||c||^2) with
 *      D = sum of q on set bits, T = sum of q, P = number of set bits (fp32, in this
 *      order).
 *   objective (nullable): double[1], receives sum over points of the in-space
 *      distance (score plus the point-only term), fp64.  For the 1-bit formats the
 *      point-only term is the decoded point's squared norm alpha^2 d; for LVQ4 it is N_x.
 *   1 <= k.
 */
km_status kmeans_assign(const km_points *P, const void *C, int32_t k, int32_t *assign, float *score,
                        double *objective, km_stream stream);

/*
 * kmeans_assign_noalloc -- kmeans_assign for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  Same arguments, checks, kernels and results as kmeans_assign; its
 * scratch (centroid preparation, the (score, index) keys of the centroid-tile
 * groups, objective partials) lives in a static device array of 64 MiB that the
 * library holds on every device it runs on until the process ends, so the call
 * makes no allocation of any kind.
 *   KM_EINVAL when the call would need more than 64 MiB of scratch: about
 *   16 bytes per point with the objective, 8 without (fp32, bfloat16 and SQ8
 *   points in centroid-tile groups), plus the prepared centroids (k x d bytes for
 *   SQ8 and the 1-bit formats, 2 k d for bfloat16) and 16 k bytes.
 *   Every call on one device shares that device's array, which keeps the last
 *   call's contents: calls that overlap on one device (on different streams, or
 *   from different threads without ordering) race and give undefined results.
 *   Calls on different devices do not share it.
 */
km_status kmeans_assign_noalloc(const km_points *P, const void *C, int32_t k, int32_t *assign, float *score,
                                double *objective, km_stream stream);

/*
 * kmeans_update -- STEP 3 (Sec. 2.3): each centroid becomes the mean of its
 * members, in the clustering space:
 *   KM_F32: fp32 mean; KM_BF16: fp32 mean of the stored bfloat16 values;
 *   KM_SQ8: floor((2 S + n_j) / (2 n_j)) with S the exact code sum
 *   (averaging in the quantised domain, Sec. 3.1); KM_SIGN1: m + (1/n_j) sum alpha (2b - 1)
 *   (fused decode-averaging, Sec. 3.1); KM_HYBRID: front mean and tail decode-average;
 *   KM_RABITQ: (1/n_j) sum alpha (2b - 1) in the rotated residual space;
 *   KM_LVQ4: the fp32 mean of the decoded members fmaf(s, code, b).
 *   C: in = previous centroids, out = new ones (same type as kmeans_assign).
 *   counts (nullable): int64[k] member counts of `assign`.
 *   policy KM_EMPTY_SPLIT: empty clusters, in ascending order, take a split of the
 *   cluster with the largest current count (ties to the smallest index) when that
 *   count is >= 2: c_j = c_b (1 + eps p), c_b = c_b (1 - eps p), p_i = (-1)^i,
 *   eps = 2^-10, on the clustering-space vector (1-bit dims: the residual c - m;
 *   SQ8: c_j = clip(c_b + p), c_b = clip(c_b - p)); the donor's count is halved
 *   for later choices.  KM_EMPTY_KEEP leaves empty clusters unchanged.
 *   Deterministic: the result does not depend on scheduling.
 */
km_status kmeans_update(const km_points *P, const int32_t *assign, int32_t k, void *C, int64_t *counts,
                        int32_t policy, km_stream stream);

/* Per-stage device times of one kmeans_fit call (milliseconds, from HIP events
 * recorded on the call's stream around each launch). */
typedef struct km_fit_stats {
  double assign_ms;      /* fused assignment kernels only, summed over the passes */
  double prep_ms;        /* centroid preparation before each pass */
  double update_ms;      /* complete update step (sort, sums, split, compose) */
  double other_ms;       /* initial gather, point-only terms, objective sums */
  int32_t assign_passes; /* iters + 1 */
  int32_t updates;       /* iters */
} km_fit_stats;

/*
 * kmeans_fit -- Lloyd's algorithm (Sec. 2.3): STEP 1 (C = the points at
 * init_idx), then `iters` x (STEP 2, STEP 3), then a final STEP 2.  When
 * P->raw is set, the last STEP 3 averages the raw rows instead of the codes.
 *   init_idx: HOST int64[k], distinct, in [0, n); NULL = C already holds the
 *     initial centroids (resume from saved centroids).
 *   C: out (and in when init_idx is NULL), as in kmeans_assign.
 *   assign: int32[n], the final assignment.
 *   objective (nullable): DEVICE double[iters + 1]; entry t is the in-space
 *     objective of the t-th assignment pass (sum of in-space distances to the
 *     centroids that pass used).
 *   stats (nullable, HOST): per-stage device times; when given, the call waits
 *     for `stream` to finish before returning.  Otherwise nothing is
 *     synchronised: the call only enqueues work on `stream`.
 */
km_status kmeans_fit(const km_points *P, int32_t k, int32_t iters, const int64_t *init_idx, void *C,
                     int32_t *assign, double *objective, int32_t policy, km_fit_stats *stats,
                     km_stream stream);

/* Dimension pruning inside STEP 2 (Sec. 3.1 SuperKMeans, ADSampling test). */
typedef struct km_prune {
  double eps0;     /* ADSampling's epsilon_0 (> 0); 2.1 is the usual value */
  int32_t d_front; /* d', the dims of the first test; 0 = 12.5 % of d rounded up to 32 (at most d) */
  int32_t reserved; /* must be 0 */
} km_prune;

/*
 * kmeans_assign_pruned -- one STEP 2 with dimension pruning (Sec. 3.1 "SuperKMeans";
 * the ADSampling hypothesis test).  For every point, best = prev[i] at squared
 * distance tau; every other centroid j is tested at the checkpoints D = d',
 * d' + 64, d' + 128, ... (D < d) on its partial squared distance p(D) over the
 * first D dims and dropped when p(D) > tau * r(D), r(D) = (1 + eps0 / sqrt(D))^2
 * D / d; centroids never dropped are compared on the full distance (smaller wins,
 * ties to the smaller index).  Meant for points under a random orthogonal
 * rotation (the test assumes variance spread evenly over the dims); the result
 * can differ from the exact nearest centroid when the test drops it.
 *   P: KM_F32 (fp32 sums; r(D) rounded to fp32) or KM_SQ8 (exact integer distances
 *   in code space, the test on (float)p(D) > (float)tau * (float)r(D)); d <= d' + 2048,
 *   d' <= 256, d and d' multiples of 8 (F32) or of 16 (SQ8).  C as in kmeans_assign.
 *   prev: int32[n], the previous assignment (values in [0, k)); may be the same
 *   array as assign.  dist (nullable): DEVICE double[n], the winning squared distance.
 *   objective (nullable): DEVICE double[1], sum of dist.
 *   counters (nullable, HOST uint64[3]): candidates tested at d', candidates that
 *   passed d', candidates compared on the full distance; the call then waits for
 *   the stream.
 */
km_status kmeans_assign_pruned(const km_points *P, const void *C, int32_t k, const int32_t *prev, int32_t *assign,
                               double *dist, double *objective, const km_prune *pr, uint64_t *counters,
                               km_stream stream);

/*
 * kmeans_fit_pruned -- kmeans_fit whose assignment passes after the first one are
 * kmeans_assign_pruned from the previous assignment (SuperKMeans: the first pass
 * is a full one).  Arguments as in kmeans_fit; pr as in kmeans_assign_pruned;
 * counters (nullable, HOST uint64[3]) summed over the pruned passes (the call then
 * waits for the stream).
 */
km_status kmeans_fit_pruned(const km_points *P, int32_t k, int32_t iters, const int64_t *init_idx, void *C,
                            int32_t *assign, double *objective, int32_t policy, const km_prune *pr,
                            km_fit_stats *stats, uint64_t *counters, km_stream stream);

/* kmeans_fine() flags */
#define KM_FINE_C_GIVEN 1 /* C holds the initial fine centroids; otherwise they are taken from the points */
#define KM_FINE_SQRT 2    /* the paper's fine counts, k_i = round(sqrt(n_i)) (see kmeans_fine) */

/*
 * kmeans_fine -- FINE-CLUSTERING of hierarchical k-means (Sec. 4.4, Table 7):
 * Lloyd inside every meso-cluster, on that meso-cluster's points only.
 *   meso_assign: DEVICE int32[n], the meso-cluster of every point; points with an
 *     id outside [0, k_meso) take no part and get assign = -1.
 *   Fine clusters per meso-cluster (k_i; the paper sizes them by the meso-cluster
 *     size n_i without making them sum to k): one for every non-empty meso-cluster,
 *     the other k - m (m = number of non-empty meso-clusters) shared in proportion
 *     to n_i - 1: floor shares, then one more for the largest remainders (ties to
 *     the smaller meso index).  Fine centroid j of meso-cluster i is centroid
 *     off_i + j of C, off_i = k_0 + ... + k_{i-1}.  KM_EINVAL unless m <= k <= the
 *     number of points with a valid meso id.
 *   With flags & KM_FINE_SQRT, the counts of Sec. 4.4 taken literally: k_i = the
 *     integer nearest to sqrt(n_i) for every non-empty meso-cluster (their sum is
 *     set by the data); k is then the capacity of C: KM_EINVAL if the k_i sum to
 *     more, and the rows of C past their sum are left as they are.
 *   STEP 1 (unless flags has KM_FINE_C_GIVEN): centroid off_i + j = the member of
 *     meso-cluster i at position floor(j n_i / k_i) in ascending point order.
 *   Then `iters` x (STEP 2 against the point's own meso-cluster's centroids, STEP 3
 *   as in kmeans_update, where an empty fine cluster takes its split donor from its
 *   own meso-cluster), and a final STEP 2.
 *   C: k centroids (in, when KM_FINE_C_GIVEN; out), as in kmeans_assign.
 *   assign: int32[n] global fine-centroid ids.  k_fine (nullable, HOST int32[k_meso])
 *   receives k_i.  objective (nullable): DEVICE double[1], the in-space objective of
 *   the final pass.
 *   The call waits for `stream` once, to read the meso-cluster sizes; it keeps a
 *   meso-ordered copy of the points in scratch memory while it runs.
 */
km_status kmeans_fine(const km_points *P, const int32_t *meso_assign, int32_t k_meso, int32_t k, int32_t iters,
                      int32_t flags, void *C, int32_t *assign, int32_t *k_fine, double *objective, int32_t policy,
                      km_stream stream);

typedef struct km_hier_params {
  int32_t k_meso;       /* meso-clusters; 0 = the integer nearest to sqrt(k) */
  int32_t iters_meso;   /* Lloyd iterations of MESO-CLUSTERING */
  int32_t iters_fine;   /* Lloyd iterations inside every meso-cluster */
  int32_t iters_refine; /* vanilla Lloyd iterations over all points and all k centroids afterwards; 0 = none */
  int32_t flags;        /* KM_FINE_SQRT: the paper's fine counts; k is then the capacity of C and the refinement
                           runs on the fine centroids made (their number is the sum of k_fine) */
} km_hier_params;

/*
 * kmeans_fit_hier -- hierarchical k-means (Sec. 4.4, Table 7): MESO-CLUSTERING =
 * kmeans_fit with k_meso centroids from the rows init_meso (HOST int64[k_meso],
 * distinct) for iters_meso iterations; FINE-CLUSTERING = kmeans_fine with
 * iters_fine iterations; then, if iters_refine > 0, kmeans_fit from the fine
 * centroids with iters_refine iterations over all points (its last update from
 * P->raw when set; the meso and fine phases use the compressed points only).
 *   C, assign: out, as in kmeans_fit.  meso_assign (nullable): DEVICE int32[n],
 *   receives the meso partition (the upper level of the two-level clustering).
 *   k_fine: as in kmeans_fine.
 *   objective (nullable): DEVICE double[1], the in-space objective of the returned
 *   partition.  stats (nullable, HOST): stage times summed over the three phases;
 *   phase_ms (nullable, HOST double[3]): device time of the meso, fine and refine
 *   phases.  Either makes the call wait for `stream` at the end; the fine phase
 *   always waits once (see kmeans_fine).
 */
km_status kmeans_fit_hier(const km_points *P, int32_t k, const km_hier_params *hp, const int64_t *init_meso, void *C,
                          int32_t *assign, int32_t *meso_assign, int32_t *k_fine, double *objective, int32_t policy,
                          km_fit_stats *stats, double *phase_ms, km_stream stream);

/*
 * kmeans_cost -- sum over points of ||x - c_{assign(x)}||^2 in fp64 for fp32
 * points (the full-precision partition cost when C holds the member means of the
 * raw vectors, Sec. 4.2 "recompute").  X float[n][ldx], C float[k][d],
 * out: DEVICE double[1].  Points with an assignment outside [0, k) are skipped.
 */
km_status kmeans_cost(const float *X, int64_t n, int32_t d, int64_t ldx, const float *C, int32_t k,
                      const int32_t *assign, double *out, km_stream stream);

/* Thread-local message for the last non-OK status ("" if none). */
const char *km_last_error(void);

/* Return pooled scratch memory of the current device to the system. */
km_status km_release(void);

#ifdef __cplusplus
}
#endif
#endif /* KMQ_H */
