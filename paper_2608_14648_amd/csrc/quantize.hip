// Compression before clustering (Sec. 3.1): SQ8 with per-dimension (lo, hi) and
// 1-bit sign codes around the dataset mean with a per-vector scale.
//
// Column statistics (min/max, fp64 sums) are two-level reductions: 256-thread
// blocks own a run of rows and read them as coalesced float4 rows, writing one
// partial per column; a second kernel folds the partials in block order.
// SQ8 encode: one thread per 16 codes (4 float4 loads, one 16-byte store).
// 1-bit encode: one wave per row, one dim per lane; a wave ballot of (x - m > 0)
// is directly two 32-bit code words (bit i of the vector = lane i % 32 of word
// i / 32), and the fp64 sums of r^2 and |r| give alpha.
#include <algorithm>

#include "common.hpp"

namespace kmq {
namespace {

constexpr int kRowsPerBlock = 1024;

__global__ __launch_bounds__(256) void colminmax_partial_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                                float *pmin, float *pmax) {
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock;
  const int64_t r1 = min<int64_t>(n, r0 + kRowsPerBlock);
  auto fold = [](f32x4 &mn, f32x4 &mx, const f32x4 v) {
    mn.x = fminf(mn.x, v.x); mn.y = fminf(mn.y, v.y); mn.z = fminf(mn.z, v.z); mn.w = fminf(mn.w, v.w);
    mx.x = fmaxf(mx.x, v.x); mx.y = fmaxf(mx.y, v.y); mx.z = fmaxf(mx.z, v.z); mx.w = fmaxf(mx.w, v.w);
  };
  for (int g = threadIdx.x; g < d / 4; g += 256) {
    // four independent running extrema keep four row loads in flight per thread
    // (min and max are exact in any order)
    const f32x4 first = *reinterpret_cast<const f32x4 *>(X + r0 * ldx + 4 * g);
    f32x4 mn[4] = {first, first, first, first}, mx[4] = {first, first, first, first};
    int64_t r = r0 + 1;
    for (; r + 3 < r1; r += 4) {
      f32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const f32x4 *>(X + (r + u) * ldx + 4 * g);
#pragma unroll
      for (int u = 0; u < 4; ++u) fold(mn[u], mx[u], v[u]);
    }
    for (; r < r1; ++r) fold(mn[0], mx[0], *reinterpret_cast<const f32x4 *>(X + r * ldx + 4 * g));
#pragma unroll
    for (int u = 1; u < 4; ++u) {
      fold(mn[0], mx[0], mn[u]);
      fold(mn[0], mx[0], mx[u]);
    }
    *reinterpret_cast<f32x4 *>(pmin + (int64_t)blockIdx.x * d + 4 * g) = mn[0];
    *reinterpret_cast<f32x4 *>(pmax + (int64_t)blockIdx.x * d + 4 * g) = mx[0];
  }
}

// one workgroup per column: strided partial extrema, then a tree (min and max are
// exact in any order)
__global__ __launch_bounds__(256) void colminmax_final_kernel(const float *pmin, const float *pmax, int nb, int d,
                                                              float *lo, float *hi) {
  __shared__ float smn[256], smx[256];
  const int i = blockIdx.x;
  const int t = threadIdx.x;
  float mn = INFINITY, mx = -INFINITY;
  for (int b = t; b < nb; b += 256) {
    mn = fminf(mn, pmin[(int64_t)b * d + i]);
    mx = fmaxf(mx, pmax[(int64_t)b * d + i]);
  }
  smn[t] = mn;
  smx[t] = mx;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (t < st) {
      smn[t] = fminf(smn[t], smn[t + st]);
      smx[t] = fmaxf(smx[t], smx[t + st]);
    }
    __syncthreads();
  }
  if (t == 0) {
    lo[i] = smn[0];
    hi[i] = smx[0];
  }
}

__global__ __launch_bounds__(256) void colsum_partial_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                             int64_t rows_per_block, double *psum) {
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = min<int64_t>(n, r0 + rows_per_block);
  for (int g = threadIdx.x; g < d / 4; g += 256) {
    double s0 = 0, s1 = 0, s2 = 0, s3 = 0;
    int64_t r = r0;
    for (; r + 3 < r1; r += 4) {
      const f32x4 v0 = *reinterpret_cast<const f32x4 *>(X + r * ldx + 4 * g);
      const f32x4 v1 = *reinterpret_cast<const f32x4 *>(X + (r + 1) * ldx + 4 * g);
      const f32x4 v2 = *reinterpret_cast<const f32x4 *>(X + (r + 2) * ldx + 4 * g);
      const f32x4 v3 = *reinterpret_cast<const f32x4 *>(X + (r + 3) * ldx + 4 * g);
      s0 += v0.x; s1 += v0.y; s2 += v0.z; s3 += v0.w;
      s0 += v1.x; s1 += v1.y; s2 += v1.z; s3 += v1.w;
      s0 += v2.x; s1 += v2.y; s2 += v2.z; s3 += v2.w;
      s0 += v3.x; s1 += v3.y; s2 += v3.z; s3 += v3.w;
    }
    for (; r < r1; ++r) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(X + r * ldx + 4 * g);
      s0 += v.x; s1 += v.y; s2 += v.z; s3 += v.w;
    }
    double *o = psum + (int64_t)blockIdx.x * d + 4 * g;
    o[0] = s0; o[1] = s1; o[2] = s2; o[3] = s3;
  }
}

// one workgroup per column: strided partial sums, then a fixed-order tree
__global__ __launch_bounds__(256) void colmean_final_kernel(const double *psum, int nb, int d, int64_t n, float *m) {
  __shared__ double sh[256];
  const int i = blockIdx.x;
  double s = 0.0;
  for (int b = threadIdx.x; b < nb; b += 256) s += psum[(int64_t)b * d + i];
  s = block_sum_f64(s, sh);
  if (threadIdx.x == 0) m[i] = (float)(s / (double)n);
}

__global__ void sq8_inv_kernel(const float *lo, const float *hi, int d, float *inv) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= d) return;
  const float range = hi[i] - lo[i];
  inv[i] = range > 0.0f ? 255.0f / range : 0.0f;
}

__global__ __launch_bounds__(256) void sq8_encode_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                         const float *lo, const float *inv, uint8_t *codes) {
  const int per = d / 16;
  const int64_t total = n * per;
  for (int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x; g < total; g += (int64_t)gridDim.x * 256) {
    const int64_t r = g / per;
    const int c = (int)(g - r * per) * 16;
    const float *x = X + r * ldx + c;
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(x + 4 * q);
      uint32_t packed = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = c + 4 * q + e;
        float t = rintf((v[e] - lo[i]) * inv[i]);
        t = fminf(fmaxf(t, 0.0f), 255.0f);
        packed |= (uint32_t)t << (8 * e);
      }
      w[q] = packed;
    }
    *reinterpret_cast<uint4 *>(codes + r * d + c) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// 8 values per thread: two float4 loads, one 16-byte store of bfloat16 patterns.
__global__ __launch_bounds__(256) void bf16_encode_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                          uint16_t *codes) {
  const int per = d / 8;
  const int64_t total = n * per;
  for (int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x; g < total; g += (int64_t)gridDim.x * 256) {
    const int64_t r = g / per;
    const int c = (int)(g - r * per) * 8;
    const f32x4 a = *reinterpret_cast<const f32x4 *>(X + r * ldx + c);
    const f32x4 b = *reinterpret_cast<const f32x4 *>(X + r * ldx + c + 4);
    const uint4 w = make_uint4(bf16_bits(a[0]) | (bf16_bits(a[1]) << 16), bf16_bits(a[2]) | (bf16_bits(a[3]) << 16),
                               bf16_bits(b[0]) | (bf16_bits(b[1]) << 16), bf16_bits(b[2]) | (bf16_bits(b[3]) << 16));
    *reinterpret_cast<uint4 *>(codes + r * d + c) = w;
  }
}

// LVQ4: one wave per row.  Pass 1: the row's min and max (float4 per lane, wave
// reductions); pass 2: codes, two per byte, and the exact sums S and Q of the codes;
// lane 0 writes (s, b, A, N) with the fp32 expressions of the format definition.
// NV > 0: rows of at most 256 NV dims stay in registers between the passes (NV
// float4 per lane, all loads in flight at once), so a row is read once; NV = 0
// reads it again for pass 2.
template <int NV>
__global__ __launch_bounds__(256) void lvq4_encode_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                          uint8_t *codes, float *par) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const float *x = X + row * ldx;
  constexpr int R = NV > 0 ? NV : 1;
  f32x4 v[R];
  float lo = INFINITY, hi = -INFINITY;
  if constexpr (NV > 0) {
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int i = 4 * lane + 256 * j;  // d % 32 == 0: a float4 is wholly in or out
      v[j] = i < d ? *reinterpret_cast<const f32x4 *>(x + i) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      if (4 * lane + 256 * j < d) {
        lo = fminf(fminf(lo, v[j][0]), fminf(fminf(v[j][1], v[j][2]), v[j][3]));
        hi = fmaxf(fmaxf(hi, v[j][0]), fmaxf(fmaxf(v[j][1], v[j][2]), v[j][3]));
      }
    }
  } else {
    for (int i = 4 * lane; i < d; i += 256) {
      const f32x4 w = *reinterpret_cast<const f32x4 *>(x + i);
      lo = fminf(fminf(lo, w[0]), fminf(fminf(w[1], w[2]), w[3]));
      hi = fmaxf(fmaxf(hi, w[0]), fmaxf(fmaxf(w[1], w[2]), w[3]));
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    lo = fminf(lo, __shfl_xor(lo, off));
    hi = fmaxf(hi, __shfl_xor(hi, off));
  }
  const float s = hi > lo ? (hi - lo) / 15.0f : 1.0f;
  int S = 0, Q = 0;
  uint8_t *out = codes + row * (int64_t)(d / 2);
  auto encode4 = [&](const f32x4 &w, int i) {
    int c[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      c[e] = (int)fminf(fmaxf(rintf((w[e] - lo) / s), 0.0f), 15.0f);
      S += c[e];
      Q += c[e] * c[e];
    }
    *reinterpret_cast<uint16_t *>(out + i / 2) = (uint16_t)(c[0] | (c[1] << 4) | (c[2] << 8) | (c[3] << 12));
  };
  if constexpr (NV > 0) {
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (4 * lane + 256 * j < d) encode4(v[j], 4 * lane + 256 * j);
  } else {
    for (int i = 4 * lane; i < d; i += 256) encode4(*reinterpret_cast<const f32x4 *>(x + i), i);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    S += __shfl_xor(S, off);
    Q += __shfl_xor(Q, off);
  }
  if (lane == 0) {
    const float db = (float)d * lo;
    *reinterpret_cast<f32x4 *>(par + 4 * row) =
        f32x4{s, lo, fmaf(s, (float)S, db), fmaf(s * s, (float)Q, fmaf(2.0f * lo * s, (float)S, db * lo))};
  }
}

// One wave per row.  Lane l reads dims [base + 4l, base + 4l + 4) as a float4 and
// forms a 4-bit nibble of sign bits; the 8 lanes that share a 32-dim word OR
// their shifted nibbles together (3 xor-shuffles) and the first of them stores
// the word, so a wave stores 8 consecutive words per 256 dims.
__global__ __launch_bounds__(256) void sign1_encode_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                           const float *m, int d0, uint32_t *bits, float *alpha,
                                                           float *front) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const float *x = X + row * ldx;
  uint32_t *b = bits + row * (d / 32);
  double s2 = 0.0, s1 = 0.0;
  for (int base = 0; base < d; base += 256) {
    const int i0 = base + 4 * lane;
    const bool in = i0 < d;  // d % 32 == 0, so a float4 is either wholly in or out
    f32x4 xv = {0.f, 0.f, 0.f, 0.f}, mv = {0.f, 0.f, 0.f, 0.f};
    if (in) {
      xv = *reinterpret_cast<const f32x4 *>(x + i0);
      mv = *reinterpret_cast<const f32x4 *>(m + i0);
    }
    uint32_t nib = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float r = xv[e] - mv[e];
      nib |= (in && r > 0.0f) ? (1u << e) : 0u;
      if (in && i0 + e >= d0) {
        s2 += (double)r * (double)r;
        s1 += fabs((double)r);
      }
    }
    uint32_t w = nib << (4 * (lane & 7));
    w |= __shfl_xor(w, 1);
    w |= __shfl_xor(w, 2);
    w |= __shfl_xor(w, 4);
    if (in && (lane & 7) == 0) b[(i0 >> 5)] = w;
    if (front && in && i0 < d0) *reinterpret_cast<f32x4 *>(front + row * d0 + i0) = xv;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    s2 += __shfl_xor(s2, off);
    s1 += __shfl_xor(s1, off);
  }
  if (lane == 0) alpha[row] = s1 > 0.0 ? (float)(s2 / s1) : 0.0f;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float *v, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) v[i] = 0.0f;
}

}  // namespace

constexpr int kMaxSumBlocks = 1024;

size_t colmean_bytes(int64_t n, int d) {
  return (size_t)std::min<int64_t>(kMaxSumBlocks, cdiv(n, 64)) * d * sizeof(double) + 256;
}

km_status launch_colmean(const float *X, int64_t n, int d, int64_t ldx, float *m, void *ws, hipStream_t s) {
  const int64_t want = std::min<int64_t>(kMaxSumBlocks, cdiv(n, 64));
  const int64_t rpb = cdiv(n, want);
  const int nb = (int)cdiv(n, rpb);
  double *psum = static_cast<double *>(ws);
  hipLaunchKernelGGL(colsum_partial_kernel, dim3(nb), dim3(256), 0, s, X, n, d, ldx, rpb, psum);
  hipLaunchKernelGGL(colmean_final_kernel, dim3(d), dim3(256), 0, s, psum, nb, d, n, m);
  KMQ_LAUNCH_CHECK("column mean");
  return KM_OK;
}

size_t quantize_bytes(int64_t n, int d, int fmt) {
  if (fmt == KM_BF16 || fmt == KM_LVQ4) return 0;
  const int64_t nb = cdiv(n, kRowsPerBlock);
  if (fmt == KM_SQ8) return (size_t)nb * d * 2 * sizeof(float) + (size_t)d * sizeof(float) + 512;
  return colmean_bytes(n, d);
}

static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

// workspace: column-mean partials | transposed P | zero centre (d) | rotated rows y
// (n x d, only when the caller does not take them)
size_t rabitq_encode_bytes(int64_t n, int d, bool y_given) {
  return al256(colmean_bytes(n, d)) + al256(pca_project_bytes(d, d)) + al256((size_t)d * sizeof(float)) +
         (y_given ? 0 : al256((size_t)n * d * sizeof(float)));
}

// RabitQ codes (Sec. 3.1): centre (column mean when fitting), rotate with the
// projection kernel, then sign bits and alpha of the rotated residual (centre 0).
km_status launch_rabitq_encode(const float *X, int64_t n, int d, int64_t ldx, const float *P, float *m,
                               uint32_t *bits, float *alpha, float *Y, int flags, void *ws, hipStream_t s) {
  uint8_t *w = static_cast<uint8_t *>(ws);
  void *wmean = w;
  void *wproj = w + al256(colmean_bytes(n, d));
  float *zero = reinterpret_cast<float *>(w + al256(colmean_bytes(n, d)) + al256(pca_project_bytes(d, d)));
  if (Y == nullptr) Y = zero + al256((size_t)d * sizeof(float)) / sizeof(float);
  if (flags & KM_Q_FIT_PARAMS) {
    km_status st = launch_colmean(X, n, d, ldx, m, wmean, s);
    if (st != KM_OK) return st;
  }
  km_status st = launch_pca_project(X, n, d, ldx, m, P, d, Y, wproj, s);
  if (st != KM_OK) return st;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)cdiv(d, 256)), dim3(256), 0, s, zero, d);
  hipLaunchKernelGGL(sign1_encode_kernel, dim3((unsigned)cdiv(n, 4)), dim3(256), 0, s, Y, n, d, (int64_t)d, zero, 0,
                     bits, alpha, nullptr);
  KMQ_LAUNCH_CHECK("rabitq encode");
  return KM_OK;
}

km_status launch_quantize(const float *X, int64_t n, int d, int64_t ldx, int fmt, void *codes, float *params,
                          float *alpha, int d_front, float *front, int flags, void *ws, hipStream_t s) {
  const int nb = (int)cdiv(n, kRowsPerBlock);
  const dim3 gd((unsigned)cdiv(d, 256));
  if (fmt == KM_SQ8) {
    float *lo = params, *hi = params + d;
    float *pmin = static_cast<float *>(ws);
    float *pmax = pmin + (size_t)nb * d;
    float *inv = pmax + (size_t)nb * d;
    if (flags & KM_Q_FIT_PARAMS) {
      hipLaunchKernelGGL(colminmax_partial_kernel, dim3(nb), dim3(256), 0, s, X, n, d, ldx, pmin, pmax);
      hipLaunchKernelGGL(colminmax_final_kernel, dim3((unsigned)d), dim3(256), 0, s, pmin, pmax, nb, d, lo, hi);
    }
    hipLaunchKernelGGL(sq8_inv_kernel, gd, dim3(256), 0, s, lo, hi, d, inv);
    const int64_t work = n * (d / 16);
    const unsigned g = (unsigned)std::min<int64_t>(cdiv(work, 256), 65536);
    hipLaunchKernelGGL(sq8_encode_kernel, dim3(g), dim3(256), 0, s, X, n, d, ldx, lo, inv,
                       static_cast<uint8_t *>(codes));
    KMQ_LAUNCH_CHECK("quantize sq8");
    return KM_OK;
  }
  if (fmt == KM_LVQ4) {
    const dim3 g((unsigned)cdiv(n, 4));
    uint8_t *c8 = static_cast<uint8_t *>(codes);
    if (d <= 1024)
      hipLaunchKernelGGL(lvq4_encode_kernel<4>, g, dim3(256), 0, s, X, n, d, ldx, c8, params);
    else if (d <= 2048)
      hipLaunchKernelGGL(lvq4_encode_kernel<8>, g, dim3(256), 0, s, X, n, d, ldx, c8, params);
    else
      hipLaunchKernelGGL(lvq4_encode_kernel<0>, g, dim3(256), 0, s, X, n, d, ldx, c8, params);
    KMQ_LAUNCH_CHECK("quantize lvq4");
    return KM_OK;
  }
  if (fmt == KM_BF16) {
    const int64_t work = n * (d / 8);
    const unsigned g = (unsigned)std::min<int64_t>(cdiv(work, 256), 65536);
    hipLaunchKernelGGL(bf16_encode_kernel, dim3(g), dim3(256), 0, s, X, n, d, ldx, static_cast<uint16_t *>(codes));
    KMQ_LAUNCH_CHECK("quantize bf16");
    return KM_OK;
  }
  if (fmt == KM_SIGN1) {
    float *m = params;
    if (flags & KM_Q_FIT_PARAMS) {
      km_status st = launch_colmean(X, n, d, ldx, m, ws, s);
      if (st != KM_OK) return st;
    }
    hipLaunchKernelGGL(sign1_encode_kernel, dim3((unsigned)cdiv(n, 4)), dim3(256), 0, s, X, n, d, ldx, m, d_front,
                       static_cast<uint32_t *>(codes), alpha, d_front > 0 ? front : nullptr);
    KMQ_LAUNCH_CHECK("quantize sign1");
    return KM_OK;
  }
  return KM_EUNSUPPORTED;
}

}  // namespace kmq
