// Internal helpers shared by the HIP sources of libkmq (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/kmq.h"

namespace kmq {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;

// Launch-facing description of the points (validated copy of km_points).
struct Points {
  int fmt;
  int d;          // logical dims
  int64_t n;
  const void *data;
  int64_t ld;     // F32: floats, SQ8: bytes, 1-bit: words (= d/32)
  const float *alpha;
  const float *center;
  const float *front;  // hybrid: n x d_front
  int d_front;
  const float *raw;    // nullable: fp32 rows in the clustering space (last update of a fit)
  int64_t raw_ld;
  const float *vparams;  // LVQ4: per-vector (s, b, A, N)
};

// 1-bit point formats (codes + one scale per point)
__host__ __device__ constexpr bool is_bits_fmt(int fmt) {
  return fmt == KM_SIGN1 || fmt == KM_HYBRID || fmt == KM_RABITQ;
}

// Per-centroid data rebuilt before each assignment pass.
struct CentroidPrep {
  const float *cn;     // F32/HYBRID/BF16: ||c'||^2 over the fp32 dims; RABITQ, LVQ4: bias b
  const int *qsum;     // SQ8: -||c~||^2 ; SIGN1/HYBRID/RABITQ: T_j = sum q ; LVQ4: S_j = sum of codes
  const float *u;      // SIGN1/HYBRID: (sigma*sigma)*Q ; RABITQ: ||c||^2 ; LVQ4: N_j
  const float *sig2;   // SIGN1/HYBRID: 2*sigma ; RABITQ, LVQ4: scale s
  const int8_t *q;     // SIGN1/HYBRID: int8 residual codes, k x dt ; RABITQ: codes 0..15, k x d ; LVQ4: codes
                       // 0..15, k x d, each 8 dims ordered 0 2 4 6 1 3 5 7 (the unpacked point order)
  const uint16_t *cb;  // BF16: centroids rounded to bfloat16, k x d
  unsigned long long *keys;  // centroid-tile groups (F32/HYBRID/SQ8/BF16/LVQ4): per-point (score, index) keys
};

// Host-side error plumbing.
void set_error(const char *fmt, ...);
km_status hip_fail(hipError_t e, const char *what);

#define KMQ_HIP(call)                                         \
  do {                                                        \
    hipError_t _e = (call);                                   \
    if (_e != hipSuccess) return ::kmq::hip_fail(_e, #call);  \
  } while (0)

#define KMQ_LAUNCH_CHECK(what)                                \
  do {                                                        \
    hipError_t _e = hipGetLastError();                        \
    if (_e != hipSuccess) return ::kmq::hip_fail(_e, what);   \
  } while (0)

__host__ __device__ static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---- launchers implemented in the kernel sources ---------------------------

// pca.hip: compute units of the current device (256 if the query fails)
int cu_count();

// assign.hip
km_status launch_prep(const Points &P, const void *C, int k, void *ws_prep, CentroidPrep *out,
                      hipStream_t s);
size_t prep_bytes(const Points &P, int k);
// aoff is added to every stored centroid index (C and cp may be a slice of a larger set)
// One launch for many (row range, centroid range) segments of fp32, SQ8 or bf16
// points: segment i is rows [segs[i].x, + segs[i].y) against centroids
// [segs[i].z, + segs[i].w) of C and of the prepared constants; workgroup b takes
// point tile tiles[b].y of segment tiles[b].x (tiles of assign_segment_rows(P) rows;
// 0 = not supported for these points).  assign and score are indexed by absolute
// row; centroid indices are absolute.  tile_c: centroids per tile (128 or 256) of
// every segment of the launch (segment_tile_centroids picks it per segment).
int assign_segment_rows(const Points &P);
// 128 for a segment of at most 128 centroids, else 256: the 256-centroid kernel
// does more MFMA work per stage, which outweighs its extra padding from 129 on
int segment_tile_centroids(int k_seg);
km_status launch_assign_segments(const Points &P, const void *C, const CentroidPrep &cp, const int4 *segs,
                                 const int2 *tiles, int64_t ntiles, int tile_c, int32_t *assign, float *score,
                                 hipStream_t s);
km_status launch_assign(const Points &P, const void *C, const CentroidPrep &cp, int k, int32_t *assign,
                        float *score, hipStream_t s, int aoff = 0);
// cp restricted to centroids [off, ...) and, for the per-point keys, to points [pstart, ...)
CentroidPrep prep_slice(const Points &P, const CentroidPrep &cp, int off, int64_t pstart);
km_status launch_xconst(const Points &P, float *xc, hipStream_t s);
km_status launch_objective(const Points &P, const float *xc, const float *score, int64_t n, double *out,
                           double *partials, int nblk_max, hipStream_t s);
int objective_blocks(int64_t n);
km_status launch_gather_init(const Points &P, const int64_t *idx, int k, void *C, hipStream_t s);
km_status launch_cost(const float *X, int64_t n, int d, int64_t ldx, const float *C, int k,
                      const int32_t *assign, double *out, double *partials, hipStream_t s);

// update.hip
size_t update_bytes(const Points &P, int k);
// seg_lo / seg_hi (nullable, int[k]): the split takes the donor of empty cluster j
// from clusters [seg_lo[j], seg_hi[j]) only.
km_status launch_update(const Points &P, const int32_t *assign, int k, void *C, int64_t *counts,
                        int policy, void *ws, hipStream_t s, const int *seg_lo = nullptr,
                        const int *seg_hi = nullptr);
struct SortOut {
  const int *perm;    // [n]: point indices ordered by cluster, point order kept inside a cluster
  const int *cnt;     // [k]: members per cluster (ids outside [0, k) are left out)
  const int *cstart;  // [k]: first position of each cluster in perm
};
size_t sort_bytes(int64_t n, int k);
km_status launch_cluster_sort(const int32_t *assign, int64_t n, int k, void *ws, SortOut *out, hipStream_t s);

// hier.hip: contiguous per-meso-cluster copies of the points and the write-back
size_t permuted_bytes(const Points &P, int64_t nrows);
km_status launch_permute_points(const Points &P, const int *perm, int64_t nrows, void *ws, Points *out,
                                hipStream_t s);
Points slice_points(const Points &P, int64_t start, int64_t count);
km_status launch_scatter_assign(const int *perm, const int32_t *a_perm, int64_t nsel, int64_t n, int32_t *assign,
                                hipStream_t s);

// skm.hip: dimension pruning inside STEP 2
double prune_factor(int D, int d, double eps0);
int prune_front_default(int d);
size_t pruned_bytes(const Points &P, int k);
km_status launch_assign_pruned(const Points &P, const void *C, int k, const int32_t *prev, int32_t *assign,
                               double *dist, double *objective, double eps0, int D0,
                               unsigned long long *cnt, void *ws, hipStream_t s);
km_status launch_zero_counters(unsigned long long *c, hipStream_t s);

// quantize.hip
size_t quantize_bytes(int64_t n, int d, int fmt);
km_status launch_quantize(const float *X, int64_t n, int d, int64_t ldx, int fmt, void *codes,
                          float *params, float *alpha, int d_front, float *front, int flags, void *ws,
                          hipStream_t s);

size_t colmean_bytes(int64_t n, int d);
size_t rabitq_encode_bytes(int64_t n, int d, bool y_given);
km_status launch_rabitq_encode(const float *X, int64_t n, int d, int64_t ldx, const float *P, float *m,
                               uint32_t *bits, float *alpha, float *Y, int flags, void *ws, hipStream_t s);
km_status launch_colmean(const float *X, int64_t n, int d, int64_t ldx, float *m, void *ws, hipStream_t s);

// pca.hip
size_t pca_cov_bytes(int64_t n, int d);
km_status launch_pca_cov(const float *X, int64_t n, int d, float *mean, float *cov, void *ws,
                         hipStream_t s);
km_status launch_pca_project(const float *X, int64_t n, int d, int64_t ldx, const float *mean, const float *W,
                             int d_out, float *Y, void *ws, hipStream_t s);
size_t pca_project_bytes(int d, int d_out);

// ---- device helpers ---------------------------------------------------------

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Nearest bfloat16 of x, ties to the even significand, as its 16-bit pattern.
// bfloat16 keeps the top 16 bits of the fp32 pattern; adding 0x7FFF plus the
// lowest kept bit carries into the kept half exactly when the discarded half
// exceeds 0x8000, or equals it and the kept half is odd.  A carry out of the
// significand steps the exponent (up to infinity), which is the correct result.
// NaN keeps its sign and top payload bits and is made quiet.
__device__ __forceinline__ uint32_t bf16_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_value(uint32_t b) { return __uint_as_float(b << 16); }

// Deterministic block-wide sum of doubles (fixed tree order). blockDim.x == 256.
__device__ __forceinline__ double block_sum_f64(double v, double *sh) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
#pragma unroll
  for (int s = 128; s > 0; s >>= 1) {
    if (t < s) sh[t] += sh[t + s];
    __syncthreads();
  }
  double r = sh[0];
  __syncthreads();
  return r;
}

}  // namespace kmq
