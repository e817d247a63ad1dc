// Data movement of hierarchical k-means (Sec. 4.4): the points of every
// meso-cluster are copied into one contiguous run of rows (the cluster-sorted
// order of the meso assignment), so each meso-cluster's FINE-CLUSTERING passes
// read a dense slice; the fine assignment is written back in point order
// afterwards.  Pure copies: no arithmetic of the method happens here.
#include <algorithm>
#include <type_traits>

#include "common.hpp"

namespace kmq {
namespace {

// dst row r = src row perm[r]; rows of `rb` bytes, VEC bytes per access.
template <int VEC>
__global__ __launch_bounds__(256) void permute_rows_kernel(const uint8_t *src, int64_t sld, uint8_t *dst, int64_t rb,
                                                           const int *perm, int64_t nrows) {
  using V = typename std::conditional<VEC == 16, uint4, uint32_t>::type;
  const int64_t per_row = rb / VEC;
  const int64_t total = nrows * per_row;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / per_row, c = i - r * per_row;
    const int64_t from = perm[r];
    *reinterpret_cast<V *>(dst + r * rb + c * VEC) = *reinterpret_cast<const V *>(src + from * sld + c * VEC);
  }
}

__global__ __launch_bounds__(256) void fill_assign_kernel(int32_t *a, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) a[i] = v;
}

__global__ __launch_bounds__(256) void scatter_assign_kernel(const int *perm, const int32_t *a_perm, int64_t nsel,
                                                             int32_t *assign) {
  for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < nsel; r += (int64_t)gridDim.x * 256)
    assign[perm[r]] = a_perm[r];
}

unsigned copy_grid(int64_t work) { return (unsigned)std::max<int64_t>(1, std::min<int64_t>(cdiv(work, 256), 8192)); }

km_status permute(const void *src, int64_t sld, void *dst, int64_t rb, const int *perm, int64_t nrows, hipStream_t s) {
  if (rb == 0 || nrows == 0) return KM_OK;
  const bool v16 = rb % 16 == 0 && sld % 16 == 0 && (reinterpret_cast<uintptr_t>(src) & 15u) == 0 &&
                   (reinterpret_cast<uintptr_t>(dst) & 15u) == 0;
  if (v16) {
    hipLaunchKernelGGL(permute_rows_kernel<16>, dim3(copy_grid(nrows * (rb / 16))), dim3(256), 0, s,
                       static_cast<const uint8_t *>(src), sld, static_cast<uint8_t *>(dst), rb, perm, nrows);
  } else {  // every row size here is a multiple of 4 bytes
    hipLaunchKernelGGL(permute_rows_kernel<4>, dim3(copy_grid(nrows * (rb / 4))), dim3(256), 0, s,
                       static_cast<const uint8_t *>(src), sld, static_cast<uint8_t *>(dst), rb, perm, nrows);
  }
  KMQ_LAUNCH_CHECK("permute rows");
  return KM_OK;
}

// bytes of one stored row of the points' main array, and its stride in bytes
int64_t row_bytes(const Points &P) {
  switch (P.fmt) {
    case KM_F32: return 4 * (int64_t)P.d;
    case KM_BF16: return 2 * (int64_t)P.d;
    case KM_SQ8: return P.d;
    case KM_LVQ4: return P.d / 2;
    default: return P.d / 8;  // 1-bit codes
  }
}

int64_t row_stride(const Points &P) {
  switch (P.fmt) {
    case KM_F32: return 4 * P.ld;
    case KM_BF16: return 2 * P.ld;
    case KM_SQ8:
    case KM_LVQ4: return P.ld;
    default: return P.d / 8;
  }
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

size_t permuted_bytes(const Points &P, int64_t nrows) {
  size_t b = al256((size_t)(nrows * row_bytes(P)));
  if (P.alpha) b += al256(4 * (size_t)nrows);
  if (P.vparams) b += al256(16 * (size_t)nrows);
  if (P.front) b += al256(4 * (size_t)nrows * (size_t)P.d_front);
  return b;
}

km_status launch_permute_points(const Points &P, const int *perm, int64_t nrows, void *ws, Points *out,
                                hipStream_t s) {
  uint8_t *w = static_cast<uint8_t *>(ws);
  Points q = P;
  q.n = nrows;
  q.raw = nullptr;
  q.raw_ld = 0;
  const int64_t rb = row_bytes(P);
  km_status st = permute(P.data, row_stride(P), w, rb, perm, nrows, s);
  if (st != KM_OK) return st;
  q.data = w;
  switch (P.fmt) {  // dense rows
    case KM_F32:
    case KM_BF16: q.ld = P.d; break;
    case KM_SQ8: q.ld = P.d; break;
    case KM_LVQ4: q.ld = P.d / 2; break;
    default: break;
  }
  w += al256((size_t)(nrows * rb));
  if (P.alpha) {
    st = permute(P.alpha, 4, w, 4, perm, nrows, s);
    if (st != KM_OK) return st;
    q.alpha = reinterpret_cast<const float *>(w);
    w += al256(4 * (size_t)nrows);
  }
  if (P.vparams) {
    st = permute(P.vparams, 16, w, 16, perm, nrows, s);
    if (st != KM_OK) return st;
    q.vparams = reinterpret_cast<const float *>(w);
    w += al256(16 * (size_t)nrows);
  }
  if (P.front) {
    st = permute(P.front, 4 * (int64_t)P.d_front, w, 4 * (int64_t)P.d_front, perm, nrows, s);
    if (st != KM_OK) return st;
    q.front = reinterpret_cast<const float *>(w);
  }
  *out = q;
  return KM_OK;
}

Points slice_points(const Points &P, int64_t start, int64_t count) {
  Points q = P;
  q.n = count;
  q.data = static_cast<const uint8_t *>(P.data) + start * row_stride(P);
  if (P.alpha) q.alpha = P.alpha + start;
  if (P.vparams) q.vparams = P.vparams + 4 * start;
  if (P.front) q.front = P.front + start * P.d_front;
  q.raw = nullptr;
  return q;
}

km_status launch_scatter_assign(const int *perm, const int32_t *a_perm, int64_t nsel, int64_t n, int32_t *assign,
                                hipStream_t s) {
  if (nsel < n) hipLaunchKernelGGL(fill_assign_kernel, dim3(copy_grid(n)), dim3(256), 0, s, assign, n, -1);
  if (nsel > 0)
    hipLaunchKernelGGL(scatter_assign_kernel, dim3(copy_grid(nsel)), dim3(256), 0, s, perm, a_perm, nsel, assign);
  KMQ_LAUNCH_CHECK("scatter assignment");
  return KM_OK;
}

}  // namespace kmq
