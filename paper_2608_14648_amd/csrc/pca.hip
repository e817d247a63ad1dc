// PCA before clustering (Sec. 3.1 "PCA"; Sec. 4.2): covariance of the centred
// points and the projection onto the leading principal directions, both as
// fp32 MFMA contractions (v_mfma_f32_32x32x2_f32).
//
// Covariance: the d x d output is cut into 256 x 256 tiles (upper triangle only,
// mirrored at the end) and the n rows are split across workgroups.  Each stage
// stages 32 rows x 256 columns of both column blocks in LDS, centred on load.
// The fp32 accumulators are added into a per-workgroup fp64 partial tile every
// 2048 rows, and the partial tiles are folded in split order.
// Projection: 128 points x 128 outputs per workgroup, 32 dims per stage; the
// point rows are centred on load and W is pre-transposed so both MFMA operands
// are read as 16 contiguous bytes per lane (k permuted identically on both).
#include <algorithm>

#include "common.hpp"

namespace kmq {
namespace {

constexpr int kT = 128;           // projection tile
constexpr int kCT = 256;          // covariance output tile
constexpr int kCovRows = 32;      // rows per covariance stage
constexpr int kCovStride = kCT + 4;
constexpr int kFlushStages = 64;  // 2048 rows per fp32 accumulation run

__device__ __forceinline__ void tile_ij(int t, int T, int &ti, int &tj) {
  // enumerate the upper triangle row by row
  ti = 0;
  while (t >= T - ti) {
    t -= T - ti;
    ++ti;
  }
  tj = ti + t;
}

// One workgroup per (256 x 256 output tile, run of rows).  Each wave owns a
// 128 x 128 quarter as 4 x 4 blocks of 32 x 32 (fp32 MFMA, rows are the
// contraction index, read column-wise from row-major LDS tiles).  Every 2048 rows
// the fp32 accumulators are added into this workgroup's own fp64 partial tile
// in global memory (read-modify-write, no other workgroup touches it).
__global__ __launch_bounds__(256, 1) void cov_kernel(const float *X, int64_t n, int d, const float *mean, int T,
                                                     int ntiles, int64_t rows_per_split, double *partial) {
  __shared__ float Ai[2][kCovRows * kCovStride];
  __shared__ float Aj[2][kCovRows * kCovStride];
  const int tile = blockIdx.x % ntiles;
  const int split = blockIdx.x / ntiles;
  int ti, tj;
  tile_ij(tile, T, ti, tj);
  const int i0 = ti * kCT, j0 = tj * kCT;
  const int64_t rb = (int64_t)split * rows_per_split;
  const int64_t re = min<int64_t>(n, rb + rows_per_split);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int wi = wave & 1, wj = wave >> 1;
  double *out = partial + ((int64_t)split * ntiles + tile) * (kCT * kCT);

  const int nst = (int)cdiv(max<int64_t>(re - rb, 0), kCovRows);
  f32x4 ri[8], rj[8];
  auto load = [&](int st) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 6, c4 = idx & 63;
      const int64_t gr = rb + (int64_t)st * kCovRows + row;
      const bool rok = gr < re;
      const int64_t grc = rok ? gr : rb;
      const int ci = i0 + 4 * c4, cj = j0 + 4 * c4;
      const bool iok = rok && ci < d, jok = rok && cj < d;
      ri[q] = *reinterpret_cast<const f32x4 *>(X + grc * d + (iok ? ci : 0));
      rj[q] = *reinterpret_cast<const f32x4 *>(X + grc * d + (jok ? cj : 0));
    }
  };
  // centring and zero-fill happen when the stage is written to LDS, one stage
  // after the loads were issued
  auto store = [&](int st, int buf) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 6, c4 = idx & 63;
      const int64_t gr = rb + (int64_t)st * kCovRows + row;
      const bool rok = gr < re;
      const int ci = i0 + 4 * c4, cj = j0 + 4 * c4;
      const bool iok = rok && ci < d, jok = rok && cj < d;
      const f32x4 mi = *reinterpret_cast<const f32x4 *>(mean + (ci < d ? ci : 0));
      const f32x4 mj = *reinterpret_cast<const f32x4 *>(mean + (cj < d ? cj : 0));
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4 *>(&Ai[buf][row * kCovStride + 4 * c4]) = iok ? ri[q] - mi : z;
      *reinterpret_cast<f32x4 *>(&Aj[buf][row * kCovStride + 4 * c4]) = jok ? rj[q] - mj : z;
    }
  };

  if (nst > 0) {
    load(0);
    store(0, 0);
  }
  __syncthreads();
  const int nrun = (nst + kFlushStages - 1) / kFlushStages;
  for (int run = 0; run < nrun; ++run) {
    f32x16 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;
    const int st1 = min(nst, (run + 1) * kFlushStages);
    for (int st = run * kFlushStages; st < st1; ++st) {
      const bool nxt = st + 1 < nst;
      if (nxt) load(st + 1);
      const float *A = Ai[st & 1];
      const float *B = Aj[st & 1];
#pragma unroll 4
      for (int p = 0; p < kCovRows / 2; ++p) {
        float a[4], b[4];
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) a[cb] = A[(2 * p + h) * kCovStride + wi * 128 + cb * 32 + r];
#pragma unroll
        for (int pb = 0; pb < 4; ++pb) b[pb] = B[(2 * p + h) * kCovStride + wj * 128 + pb * 32 + r];
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
          for (int pb = 0; pb < 4; ++pb)
            acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[cb], b[pb], acc[cb][pb], 0, 0, 0);
      }
      if (nxt) store(st + 1, (st + 1) & 1);
      __syncthreads();
    }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int il = wi * 128 + cb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
          const int jl = wj * 128 + pb * 32 + r;
          double *o = out + il * kCT + jl;
          *o = (run == 0 ? 0.0 : *o) + (double)acc[cb][pb][v];
        }
  }
  if (nrun == 0) {  // no rows: the partial tile is zero
    for (int e = t; e < kCT * kCT; e += 256) out[e] = 0.0;
  }
}

__global__ __launch_bounds__(256) void cov_reduce_kernel(const double *partial, int ntiles, int nsplit, int T, int d,
                                                         int64_t n, float *cov) {
  const int tile = blockIdx.x;
  int ti, tj;
  tile_ij(tile, T, ti, tj);
  for (int e = blockIdx.y * 256 + threadIdx.x; e < kCT * kCT; e += gridDim.y * 256) {
    const int il = e / kCT, jl = e % kCT;
    const int i = ti * kCT + il, j = tj * kCT + jl;
    if (i >= d || j >= d) continue;
    double s = 0.0;
    for (int sp = 0; sp < nsplit; ++sp) s += partial[((int64_t)sp * ntiles + tile) * (kCT * kCT) + e];
    const float v = (float)(s / (double)n);
    cov[(int64_t)i * d + j] = v;
    cov[(int64_t)j * d + i] = v;
  }
}

__global__ void transpose_kernel(const float *W, int d, int d_out, float *Wt) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)d * d_out) return;
  const int i = (int)(e / d_out), o = (int)(e % d_out);
  Wt[(int64_t)o * d + i] = W[e];
}

constexpr int kPStride = 32 + 4;  // floats per LDS row of a projection stage

// Workgroups are numbered so that the output tiles of one point tile land on the
// same XCD one after another (consecutive ids are spread over the 8 XCDs), so the
// point rows come from HBM once and from that XCD's L2 for the other tiles.
__global__ __launch_bounds__(256) void project_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                      const float *mean, const float *Wt, int d_out, float *Y,
                                                      int n_ptiles, int n_otiles) {
  __shared__ float Xs[2][kT * kPStride];
  __shared__ float Ws[2][kT * kPStride];
  const int64_t b = blockIdx.x;
  const int64_t group = b / (8 * (int64_t)n_otiles);      // 8 point tiles per group
  const int rem = (int)(b % (8 * (int64_t)n_otiles));
  const int64_t ptile = group * 8 + rem % 8;
  const int otile = rem / 8;
  if (ptile >= n_ptiles) return;
  const int64_t p0 = ptile * kT;
  const int o0 = otile * kT;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int wm = wave & 1, wn = wave >> 1;
  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

  const int nst = (d + 31) / 32;
  f32x4 rx[4], rw[4];
  const int prmax = (int)min<int64_t>(n - 1 - p0, kT - 1);
  const int ormax = min(d_out - 1 - o0, kT - 1);
  auto load = [&](int st) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 3, c4 = idx & 7;
      const int dim = 32 * st + 4 * c4;
      const int dimc = dim < d ? dim : 0;
      rx[q] = *reinterpret_cast<const f32x4 *>(X + (p0 + min(row, prmax)) * ldx + dimc);
      rw[q] = *reinterpret_cast<const f32x4 *>(Wt + (int64_t)(o0 + min(row, ormax)) * d + dimc);
    }
  };
  // centring and zero-fill at store time, one stage after the loads were issued
  auto store = [&](int st, int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 3, c4 = idx & 7;
      const int dim = 32 * st + 4 * c4;
      const bool ok = dim < d;
      const f32x4 m = *reinterpret_cast<const f32x4 *>(mean + (ok ? dim : 0));
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4 *>(&Xs[buf][row * kPStride + 4 * c4]) = ok ? rx[q] - m : z;
      *reinterpret_cast<f32x4 *>(&Ws[buf][row * kPStride + 4 * c4]) = ok ? rw[q] : z;
    }
  };
  load(0);
  store(0, 0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const bool nxt = st + 1 < nst;
    if (nxt) load(st + 1);
    const float *A = Xs[st & 1];
    const float *B = Ws[st & 1];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      f32x4 a[2], b[2];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
        a[cb] = *reinterpret_cast<const f32x4 *>(&A[(wm * 64 + cb * 32 + r) * kPStride + 8 * g + 4 * h]);
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
        b[pb] = *reinterpret_cast<const f32x4 *>(&B[(wn * 64 + pb * 32 + r) * kPStride + 8 * g + 4 * h]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int pb = 0; pb < 2; ++pb)
            acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[cb][e], b[pb][e], acc[cb][pb], 0, 0, 0);
    }
    if (nxt) store(st + 1, (st + 1) & 1);
    __syncthreads();
  }
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t p = p0 + wm * 64 + cb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        const int o = o0 + wn * 64 + pb * 32 + r;
        if (p < n && o < d_out) Y[p * d_out + o] = acc[cb][pb][v];
      }
}

struct CovPlan {
  int T, ntiles, nsplit;
  int64_t rows_per_split;
};

// One covariance workgroup fills a CU (LDS), so the number of (tile, split)
// workgroups is kept just under a whole number of passes over the CUs.
CovPlan cov_plan(int64_t n, int d) {
  CovPlan p;
  p.T = (int)cdiv(d, kCT);
  p.ntiles = p.T * (p.T + 1) / 2;
  const int cus = cu_count();
  int want = std::max(1, (2 * cus) / p.ntiles);
  if (want * p.ntiles < cus) want = std::max(1, cus / p.ntiles);
  want = (int)std::min<int64_t>(want, std::max<int64_t>(1, cdiv(n, 4096)));
  p.rows_per_split = cdiv(n, want);
  p.nsplit = (int)cdiv(n, p.rows_per_split);
  return p;
}

}  // namespace

int cu_count() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        v > 0)
      cus = v;
    else
      cus = 256;
  }
  return cus;
}

size_t pca_cov_bytes(int64_t n, int d) {
  const CovPlan p = cov_plan(n, d);
  return (size_t)p.nsplit * p.ntiles * kCT * kCT * sizeof(double) + colmean_bytes(n, d) + 256;
}

km_status launch_pca_cov(const float *X, int64_t n, int d, float *mean, float *cov, void *ws, hipStream_t s) {
  const CovPlan p = cov_plan(n, d);
  double *partial = static_cast<double *>(ws);
  void *mws = static_cast<uint8_t *>(ws) + (((size_t)p.nsplit * p.ntiles * kCT * kCT * sizeof(double) + 255) & ~(size_t)255);
  km_status st = launch_colmean(X, n, d, d, mean, mws, s);
  if (st != KM_OK) return st;
  hipLaunchKernelGGL(cov_kernel, dim3(p.ntiles * p.nsplit), dim3(256), 0, s, X, n, d, mean, p.T, p.ntiles,
                     p.rows_per_split, partial);
  hipLaunchKernelGGL(cov_reduce_kernel, dim3(p.ntiles, 16), dim3(256), 0, s, partial, p.ntiles, p.nsplit, p.T, d, n,
                     cov);
  KMQ_LAUNCH_CHECK("pca_fit_cov");
  return KM_OK;
}

size_t pca_project_bytes(int d, int d_out) { return (size_t)d * d_out * sizeof(float) + 256; }

km_status launch_pca_project(const float *X, int64_t n, int d, int64_t ldx, const float *mean, const float *W,
                             int d_out, float *Y, void *ws, hipStream_t s) {
  float *Wt = static_cast<float *>(ws);
  const int64_t e = (int64_t)d * d_out;
  hipLaunchKernelGGL(transpose_kernel, dim3((unsigned)cdiv(e, 256)), dim3(256), 0, s, W, d, d_out, Wt);
  const int n_ptiles = (int)cdiv(n, kT), n_otiles = (int)cdiv(d_out, kT);
  const int64_t nblk = cdiv(n_ptiles, 8) * 8 * n_otiles;
  hipLaunchKernelGGL(project_kernel, dim3((unsigned)nblk), dim3(256), 0, s, X, n, d, ldx, mean, Wt, d_out, Y,
                     n_ptiles, n_otiles);
  KMQ_LAUNCH_CHECK("pca_project");
  return KM_OK;
}

}  // namespace kmq
