// PCA before clustering (Sec. 3.1 "PCA"; Sec. 4.2): covariance of the centred
// points and the projection onto the leading principal directions, both as
// fp32 MFMA contractions (v_mfma_f32_32x32x2_f32).
//
// Covariance: the d x d output is cut into 128 x 128 tiles (upper triangle only,
// mirrored at the end) and the n rows are split across workgroups.  Each stage
// stages 32 rows x 128 columns of both column blocks in LDS, centred on load.
// The fp32 accumulators are flushed into fp64 registers every 2048 rows, the
// per-split tiles are written in fp64 and folded in split order.
// Projection: 128 points x 128 outputs per workgroup, 32 dims per stage; the
// point rows are centred on load and W is pre-transposed so both MFMA operands
// are read as 16 contiguous bytes per lane (k permuted identically on both).
#include <algorithm>

#include "common.hpp"

namespace kmq {
namespace {

constexpr int kT = 128;
constexpr int kCovRows = 32;
constexpr int kCovStride = kT + 4;  // floats, padded
constexpr int kFlushStages = 64;    // 2048 rows per fp32 accumulation run

__device__ __forceinline__ void tile_ij(int t, int T, int &ti, int &tj) {
  // enumerate the upper triangle row by row
  ti = 0;
  while (t >= T - ti) {
    t -= T - ti;
    ++ti;
  }
  tj = ti + t;
}

__global__ __launch_bounds__(256) void cov_kernel(const float *X, int64_t n, int d, const float *mean, int T,
                                                  int ntiles, int64_t rows_per_split, double *partial) {
  __shared__ float Ai[2][kCovRows * kCovStride];
  __shared__ float Aj[2][kCovRows * kCovStride];
  const int tile = blockIdx.x % ntiles;
  const int split = blockIdx.x / ntiles;
  int ti, tj;
  tile_ij(tile, T, ti, tj);
  const int i0 = ti * kT, j0 = tj * kT;
  const int64_t rb = (int64_t)split * rows_per_split;
  const int64_t re = min<int64_t>(n, rb + rows_per_split);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int wi = wave & 1, wj = wave >> 1;

  f32x16 acc[2][2];
  double acc64[2][2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        acc[a][b][v] = 0.f;
        acc64[a][b][v] = 0.0;
      }

  const int nst = (int)cdiv(max<int64_t>(re - rb, 0), kCovRows);
  f32x4 ri[4], rj[4];
  auto load = [&](int st) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 5, c4 = idx & 31;
      const int64_t gr = rb + (int64_t)st * kCovRows + row;
      const int ci = i0 + 4 * c4, cj = j0 + 4 * c4;
      f32x4 z = {0.f, 0.f, 0.f, 0.f};
      ri[q] = z;
      rj[q] = z;
      if (gr < re) {
        if (ci < d) {
          const f32x4 v = *reinterpret_cast<const f32x4 *>(X + gr * d + ci);
          const f32x4 m = *reinterpret_cast<const f32x4 *>(mean + ci);
          ri[q] = v - m;
        }
        if (cj < d) {
          const f32x4 v = *reinterpret_cast<const f32x4 *>(X + gr * d + cj);
          const f32x4 m = *reinterpret_cast<const f32x4 *>(mean + cj);
          rj[q] = v - m;
        }
      }
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 5, c4 = idx & 31;
      *reinterpret_cast<f32x4 *>(&Ai[buf][row * kCovStride + 4 * c4]) = ri[q];
      *reinterpret_cast<f32x4 *>(&Aj[buf][row * kCovStride + 4 * c4]) = rj[q];
    }
  };

  if (nst > 0) {
    load(0);
    store(0);
  }
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const bool nxt = st + 1 < nst;
    if (nxt) load(st + 1);
    const float *A = Ai[st & 1];
    const float *B = Aj[st & 1];
#pragma unroll
    for (int p = 0; p < kCovRows / 2; ++p) {
      float a[2], b[2];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) a[cb] = A[(2 * p + h) * kCovStride + wi * 64 + cb * 32 + r];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) b[pb] = B[(2 * p + h) * kCovStride + wj * 64 + pb * 32 + r];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
          acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[cb], b[pb], acc[cb][pb], 0, 0, 0);
    }
    if ((st + 1) % kFlushStages == 0 || st + 1 == nst) {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            acc64[a][b][v] += (double)acc[a][b][v];
            acc[a][b][v] = 0.f;
          }
    }
    if (nxt) store((st + 1) & 1);
    __syncthreads();
  }
  double *out = partial + ((int64_t)split * ntiles + tile) * (kT * kT);
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int il = wi * 64 + cb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        const int jl = wj * 64 + pb * 32 + r;
        out[il * kT + jl] = acc64[cb][pb][v];
      }
}

__global__ __launch_bounds__(256) void cov_reduce_kernel(const double *partial, int ntiles, int nsplit, int T, int d,
                                                         int64_t n, float *cov) {
  const int tile = blockIdx.x;
  int ti, tj;
  tile_ij(tile, T, ti, tj);
  for (int e = threadIdx.x; e < kT * kT; e += 256) {
    const int il = e / kT, jl = e % kT;
    const int i = ti * kT + il, j = tj * kT + jl;
    if (i >= d || j >= d) continue;
    double s = 0.0;
    for (int sp = 0; sp < nsplit; ++sp) s += partial[((int64_t)sp * ntiles + tile) * (kT * kT) + e];
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

__global__ __launch_bounds__(256) void project_kernel(const float *X, int64_t n, int d, const float *mean,
                                                      const float *Wt, int d_out, float *Y) {
  __shared__ float Xs[2][kT * kPStride];
  __shared__ float Ws[2][kT * kPStride];
  const int64_t p0 = (int64_t)blockIdx.x * kT;
  const int o0 = blockIdx.y * kT;
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
  auto load = [&](int st) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 3, c4 = idx & 7;
      const int dim = 32 * st + 4 * c4;
      f32x4 z = {0.f, 0.f, 0.f, 0.f};
      rx[q] = z;
      rw[q] = z;
      if (dim < d) {
        const int64_t pr = min<int64_t>(p0 + row, n - 1);
        const f32x4 v = *reinterpret_cast<const f32x4 *>(X + pr * d + dim);
        const f32x4 m = *reinterpret_cast<const f32x4 *>(mean + dim);
        rx[q] = v - m;
        const int orow = min(o0 + row, d_out - 1);
        rw[q] = *reinterpret_cast<const f32x4 *>(Wt + (int64_t)orow * d + dim);
      }
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + 256 * q;
      const int row = idx >> 3, c4 = idx & 7;
      *reinterpret_cast<f32x4 *>(&Xs[buf][row * kPStride + 4 * c4]) = rx[q];
      *reinterpret_cast<f32x4 *>(&Ws[buf][row * kPStride + 4 * c4]) = rw[q];
    }
  };
  load(0);
  store(0);
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
    if (nxt) store((st + 1) & 1);
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

CovPlan cov_plan(int64_t n, int d) {
  CovPlan p;
  p.T = (int)cdiv(d, kT);
  p.ntiles = p.T * (p.T + 1) / 2;
  int want = (int)std::max<int64_t>(1, cdiv(1024, p.ntiles));
  want = (int)std::min<int64_t>(want, std::max<int64_t>(1, cdiv(n, 2048)));
  p.rows_per_split = cdiv(n, want);
  p.nsplit = (int)cdiv(n, p.rows_per_split);
  return p;
}

}  // namespace

size_t pca_cov_bytes(int64_t n, int d) {
  const CovPlan p = cov_plan(n, d);
  return (size_t)p.nsplit * p.ntiles * kT * kT * sizeof(double) + colmean_bytes(n, d) + 256;
}

km_status launch_pca_cov(const float *X, int64_t n, int d, float *mean, float *cov, void *ws, hipStream_t s) {
  const CovPlan p = cov_plan(n, d);
  double *partial = static_cast<double *>(ws);
  void *mws = static_cast<uint8_t *>(ws) + (((size_t)p.nsplit * p.ntiles * kT * kT * sizeof(double) + 255) & ~(size_t)255);
  km_status st = launch_colmean(X, n, d, d, mean, mws, s);
  if (st != KM_OK) return st;
  hipLaunchKernelGGL(cov_kernel, dim3(p.ntiles * p.nsplit), dim3(256), 0, s, X, n, d, mean, p.T, p.ntiles,
                     p.rows_per_split, partial);
  hipLaunchKernelGGL(cov_reduce_kernel, dim3(p.ntiles), dim3(256), 0, s, partial, p.ntiles, p.nsplit, p.T, d, n, cov);
  KMQ_LAUNCH_CHECK("pca_fit_cov");
  return KM_OK;
}

size_t pca_project_bytes(int d, int d_out) { return (size_t)d * d_out * sizeof(float) + 256; }

km_status launch_pca_project(const float *X, int64_t n, int d, const float *mean, const float *W, int d_out, float *Y,
                             void *ws, hipStream_t s) {
  float *Wt = static_cast<float *>(ws);
  const int64_t e = (int64_t)d * d_out;
  hipLaunchKernelGGL(transpose_kernel, dim3((unsigned)cdiv(e, 256)), dim3(256), 0, s, W, d, d_out, Wt);
  hipLaunchKernelGGL(project_kernel, dim3((unsigned)cdiv(n, kT), (unsigned)cdiv(d_out, kT)), dim3(256), 0, s, X, n, d,
                     mean, Wt, d_out, Y);
  KMQ_LAUNCH_CHECK("pca_project");
  return KM_OK;
}

}  // namespace kmq
