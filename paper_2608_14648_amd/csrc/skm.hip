// Dimension pruning inside STEP 2 (Sec. 3.1 "SuperKMeans" with the ADSampling
// test, Table 4): every point starts from its previous centroid, at squared
// distance tau; another centroid is dropped as soon as its partial squared
// distance p over the first D of d dims exceeds tau * r(D),
// r(D) = (1 + eps0 / sqrt(D))^2 * D / d, tested at D = d' (the front dims) and then
// every 64 dims; the survivors are compared on the full distance.
//
//   front norms  ||x'||^2 of the points and ||c'||^2 of the centroids over d'
//   tau          one wave per point: distance to the previous centroid (16-byte
//                loads per lane)
//   front        MFMA tile kernel (128 points x 128 centroids, fp32 or int8):
//                p(d') = ||x'||^2 + ||c'||^2 - 2 <x', c'> for every pair, the test
//                at d', one survivor bit per pair; each point's bits are one
//                row of W4 words (W4 = ceil(k/128) * 4), written 16 bytes per tile
//   refine       one wave per point, lanes over 64 consecutive dims: the point's
//                mask row is read with one load, then every survivor's row is
//                loaded whole and its distance grows chunk by chunk with the test
//                after each chunk; the last chunk gives the full distance
//
// SQ8 codes: exact integer distances, the test in fp32 on (float)p and
// (float)tau; fp32 points: fp32 sums.
#include <math.h>

#include <algorithm>

#include "common.hpp"

namespace kmq {
namespace {

constexpr int kFT = 128;                 // front tile edge (points and centroids)
constexpr int kFRow = 128;               // bytes of one row staged per chunk
constexpr int kFStride = kFRow + 16;     // padded LDS row
constexpr int kFTile = kFT * kFStride;   // bytes of one staged operand tile
constexpr int kMaxFront = 4;             // 64-dim chunks of the front: d' <= 256
constexpr int kMaxTail = 32;             // 64-dim chunks after d': d <= d' + 2048

struct SkmArgs {
  int64_t n;
  int d, k;
  const uint8_t *X;  // point rows (fp32 values or uint8 codes)
  int64_t xld;       // row stride in bytes
  const uint8_t *C;  // centroid rows, dense (d values)
  const int32_t *prev;
  const void *tau;   // F32: float[n]; SQ8: int[n]
  const void *xn;    // point front norms (float / int)
  const void *cn;    // centroid front norms (float / int)
  int D0;            // front dims d'
  int W4;            // words per point row of the survivor mask (multiple of 4)
  uint32_t *mask;    // [n][W4]
  int front_test;    // d' < d: the first checkpoint is inside the row
  float r0;          // r(d')
  float rt[kMaxTail];  // r(d' + 64 (t + 1)) for the checkpoints inside the row
  int32_t *assign;
  double *dist;
  unsigned long long *cnt;  // nullable: per-workgroup (front: 2 per group) / per-wave (refine) partial counts
};

template <int FMT>
using Val = typename std::conditional<FMT == KM_F32, float, int>::type;

template <int FMT>
__device__ __forceinline__ Val<FMT> elem(const uint8_t *row, int i) {
  if constexpr (FMT == KM_F32)
    return reinterpret_cast<const float *>(row)[i];
  else
    return (int)row[i];
}

// Sum over the wave; every lane receives lane 0's result, so fp32 branches on it
// stay uniform.
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return __shfl(v, 0);
}

// One wave per row: squared norm of the first D0 values (front norms).
template <int FMT>
__global__ __launch_bounds__(256) void skm_norm_kernel(const uint8_t *rows, int64_t ld, int64_t nrows, int D0,
                                                       void *out) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= nrows) return;
  const uint8_t *row = rows + r * ld;
  Val<FMT> s = 0;
  for (int i = lane; i < D0; i += 64) {
    Val<FMT> v = elem<FMT>(row, i);
    if constexpr (FMT == KM_SQ8) v -= 128;  // the int8 values the front MFMA multiplies
    s += v * v;
  }
  s = wave_sum(s);
  if (lane == 0) static_cast<Val<FMT> *>(out)[r] = s;
}

template <int FMT>
__global__ __launch_bounds__(256) void skm_tau_kernel(SkmArgs A, void *tau) {
  const int lane = threadIdx.x & 63;
  const int64_t p = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (p >= A.n) return;
  const int j = min(max(A.prev[p], 0), A.k - 1);
  Val<FMT> acc = 0;
  if constexpr (FMT == KM_F32) {  // d % 4 == 0
    const float *x = reinterpret_cast<const float *>(A.X + p * A.xld);
    const float *c = reinterpret_cast<const float *>(A.C) + (int64_t)j * A.d;
    for (int i = 4 * lane; i < A.d; i += 256) {
      const f32x4 xv = *reinterpret_cast<const f32x4 *>(x + i);
      const f32x4 cv = *reinterpret_cast<const f32x4 *>(c + i);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t = xv[e] - cv[e];
        acc += t * t;
      }
    }
  } else {  // d % 16 == 0
    const uint8_t *x = A.X + p * A.xld;
    const uint8_t *c = A.C + (int64_t)j * A.d;
    for (int i = 16 * lane; i < A.d; i += 1024) {
      const uint4 xv = *reinterpret_cast<const uint4 *>(x + i);
      const uint4 cv = *reinterpret_cast<const uint4 *>(c + i);
      const uint32_t xs[4] = {xv.x, xv.y, xv.z, xv.w}, cs[4] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int t = (int)((xs[e >> 2] >> (8 * (e & 3))) & 255u) - (int)((cs[e >> 2] >> (8 * (e & 3))) & 255u);
        acc += t * t;
      }
    }
  }
  acc = wave_sum(acc);
  if (lane == 0) static_cast<Val<FMT> *>(tau)[p] = acc;
}

// ---- front: all pairs over d' dims on the matrix cores, the test at d' -------
// One workgroup per 128-point tile walks every 128-centroid tile: the (tile,
// chunk) steps form one pipeline (the next step's rows are loaded into registers
// while the current one runs on the matrix cores), and after a tile's last chunk
// its survivor bits are written, 16 bytes per point.
template <int FMT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void skm_front_kernel(SkmArgs A) {
  __shared__ __align__(16) uint8_t lds[2][2][kFTile];  // [buffer][centroids, points]
  __shared__ Val<FMT> cnl[2][kFT];                    // front norms of a tile's centroids (by tile parity)
  __shared__ __align__(16) uint32_t mrow[kFT][4];     // the tile's 4 mask words of each point
  constexpr bool F = FMT == KM_F32;
  constexpr int esz = F ? 4 : 1;
  using Acc = typename std::conditional<F, f32x16, i32x16>::type;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, r = lane & 31, h = lane >> 5;
  const int wc = w & 1, wp = w >> 1;
  const int64_t p0 = (int64_t)blockIdx.x * kFT;
  const int nct = (int)cdiv(A.k, kFT);
  const int bytes = A.D0 * esz;
  const int nch = (bytes + kFRow - 1) / kFRow;
  const int total = nct * nch;

  // this lane's two points: previous centroid, front norm, threshold tau r(d')
  int pj[2];
  Val<FMT> xn[2];
  float lim[2];
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) {
    const int64_t pc = min<int64_t>(p0 + wp * 64 + pb * 32 + r, A.n - 1);
    pj[pb] = A.prev[pc];
    xn[pb] = static_cast<const Val<FMT> *>(A.xn)[pc];
    lim[pb] = (F ? static_cast<const float *>(A.tau)[pc] : (float)static_cast<const int *>(A.tau)[pc]) * A.r0;
  }

  Acc acc[2][2];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[cb][pb][v] = 0;

  uint4 rc[4], rp[4];
  Val<FMT> cnv = 0;
  auto load = [&](int ct, int ch) {
    const int c0 = ct * kFT;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = t + 256 * i;
      const int row = idx >> 3, col = idx & 7;
      const int b = ch * kFRow + 16 * col;
      const bool ok = b < bytes;
      const int64_t crow = min(c0 + row, A.k - 1);
      const int64_t prow = min<int64_t>(p0 + row, A.n - 1);
      rc[i] = ok ? *reinterpret_cast<const uint4 *>(A.C + crow * A.d * esz + b) : make_uint4(0, 0, 0, 0);
      rp[i] = ok ? *reinterpret_cast<const uint4 *>(A.X + prow * A.xld + b) : make_uint4(0, 0, 0, 0);
    }
    if (ch == 0 && t < kFT) cnv = static_cast<const Val<FMT> *>(A.cn)[min(c0 + t, A.k - 1)];
  };
  auto store = [&](int ct, int ch, int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = t + 256 * i;
      const int row = idx >> 3, col = idx & 7;
      const bool ok = ch * kFRow + 16 * col < bytes;
      uint4 vc = rc[i], vp = rp[i];
      if (!F) {  // uint8 code -> int8 (code - 128)
        vc = make_uint4(vc.x ^ 0x80808080u, vc.y ^ 0x80808080u, vc.z ^ 0x80808080u, vc.w ^ 0x80808080u);
        vp = make_uint4(vp.x ^ 0x80808080u, vp.y ^ 0x80808080u, vp.z ^ 0x80808080u, vp.w ^ 0x80808080u);
      }
      if (!ok) vc = vp = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(&lds[buf][0][row * kFStride + 16 * col]) = vc;
      *reinterpret_cast<uint4 *>(&lds[buf][1][row * kFStride + 16 * col]) = vp;
    }
    if (ch == 0 && t < kFT) cnl[ct & 1][t] = cnv;
  };

  unsigned tested = 0, passed = 0;  // per lane; at most 64 per tile
  load(0, 0);
  store(0, 0, 0);
  __syncthreads();
  for (int q = 0; q < total; ++q) {
    const int ct = q / nch, ch = q - ct * nch;
    const int buf = q & 1;
    const bool has_next = q + 1 < total;
    const int ct_n = ch + 1 == nch ? ct + 1 : ct, ch_n = ch + 1 == nch ? 0 : ch + 1;
    if (has_next) load(ct_n, ch_n);
    const uint8_t *cbuf = lds[buf][0];
    const uint8_t *pbuf = lds[buf][1];
#pragma unroll
    for (int g = 0; g < 4; ++g) {  // 32 bytes of every row per step
      uint4 av[2], bv[2];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
        av[cb] = *reinterpret_cast<const uint4 *>(cbuf + (wc * 64 + cb * 32 + r) * kFStride + 32 * g + 16 * h);
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
        bv[pb] = *reinterpret_cast<const uint4 *>(pbuf + (wp * 64 + pb * 32 + r) * kFStride + 32 * g + 16 * h);
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          if constexpr (F) {
            const f32x4 a = __builtin_bit_cast(f32x4, av[cb]);
            const f32x4 b = __builtin_bit_cast(f32x4, bv[pb]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc[cb][pb], 0, 0, 0);
          } else {
            const i32x4 a = {(int)av[cb].x, (int)av[cb].y, (int)av[cb].z, (int)av[cb].w};
            const i32x4 b = {(int)bv[pb].x, (int)bv[pb].y, (int)bv[pb].z, (int)bv[pb].w};
            acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[cb][pb], 0, 0, 0);
          }
        }
    }
    if (has_next) store(ct_n, ch_n, buf ^ 1);
    __syncthreads();
    if (ch + 1 < nch) continue;
    // epilogue of tile ct: lane (r, h) holds centroid rows 8 (v >> 2) + 4 h + (v & 3)
    // of each 32 x 32 block for point column r; the threshold test per pair, the
    // validity (j < k, j != previous centroid, point in range) per 32-bit word
    const int c0 = ct * kFT;
    const Val<FMT> *cnt_ = cnl[ct & 1];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const int64_t p = p0 + wp * 64 + pb * 32 + r;
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
        const int jb = c0 + wc * 64 + cb * 32;  // first centroid of the block (multiple of 32)
        uint32_t m = 0;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int off = 8 * (v >> 2) + 4 * h + (v & 3);
          const Val<FMT> cnj = cnt_[wc * 64 + cb * 32 + off];
          bool keep;
          if constexpr (F) {
            const float pd = fmaf(-2.0f, acc[cb][pb][v], xn[pb] + cnj);
            keep = !(pd > lim[pb]);
          } else {
            const int pd = xn[pb] + cnj - 2 * acc[cb][pb][v];
            keep = !((float)pd > lim[pb]);
          }
          m |= keep ? (1u << off) : 0u;
          acc[cb][pb][v] = 0;
        }
        m |= __shfl_xor(m, 32);
        const int nvalid = A.k - jb;
        uint32_t valid = (p < A.n && nvalid > 0) ? (nvalid >= 32 ? 0xFFFFFFFFu : (1u << nvalid) - 1u) : 0u;
        const int rel = pj[pb] - jb;
        if (rel >= 0 && rel < 32) valid &= ~(1u << rel);
        m = A.front_test ? (m & valid) : valid;
        if (h == 0) {
          mrow[wp * 64 + pb * 32 + r][wc * 2 + cb] = m;
          if (A.front_test) {
            tested += (unsigned)__popc(valid);
            passed += (unsigned)__popc(m);
          }
        }
      }
    }
    __syncthreads();
    if (t < kFT && p0 + t < A.n)  // words 4 ct .. 4 ct + 3 of the point's row (rows padded to W4 words)
      *reinterpret_cast<uint4 *>(A.mask + (p0 + t) * A.W4 + 4 * ct) = *reinterpret_cast<const uint4 *>(mrow[t]);
  }
  if (A.cnt) {  // per-workgroup partial counts (summed later in a fixed order)
    __shared__ unsigned long long cw[4][2];
    const unsigned long long tw = wave_sum((unsigned long long)tested);
    const unsigned long long pw = wave_sum((unsigned long long)passed);
    if (lane == 0) {
      cw[w][0] = tw;
      cw[w][1] = pw;
    }
    __syncthreads();
    if (t == 0) {
      A.cnt[2 * blockIdx.x] = cw[0][0] + cw[1][0] + cw[2][0] + cw[3][0];
      A.cnt[2 * blockIdx.x + 1] = cw[0][1] + cw[1][1] + cw[2][1] + cw[3][1];
    }
  }
}

// ---- refinement of the survivors: one wave per point ---------------------------
// The point's mask row is read first; a point without survivors keeps its previous
// centroid without touching its row.  Survivors are taken in groups of 8
// (ascending index), one survivor per 8 lanes: in each 64-dim chunk a lane sums
// 8 consecutive dims, the 8 lanes of a survivor add their sums, and every
// survivor stops at its first failed checkpoint.
constexpr int kGroup = 8;

template <int FMT>
__device__ __forceinline__ Val<FMT> sq8dims(const uint8_t *x, const uint8_t *c, int i, int lim) {
  // sum over the 8 dims [i, i + 8) below lim of (x - c)^2; i and lim are multiples of 8
  Val<FMT> s = 0;
  if (i < lim) {
    if constexpr (FMT == KM_F32) {
      const f32x4 x0 = *reinterpret_cast<const f32x4 *>(x + 4 * i), x1 = *reinterpret_cast<const f32x4 *>(x + 4 * i + 16);
      const f32x4 c0 = *reinterpret_cast<const f32x4 *>(c + 4 * i), c1 = *reinterpret_cast<const f32x4 *>(c + 4 * i + 16);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t0 = x0[e] - c0[e], t1 = x1[e] - c1[e];
        s += t0 * t0;
        s += t1 * t1;
      }
    } else {
      const uint2 xv = *reinterpret_cast<const uint2 *>(x + i), cv = *reinterpret_cast<const uint2 *>(c + i);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t xw = e < 4 ? xv.x : xv.y, cw = e < 4 ? cv.x : cv.y;
        const int t = (int)((xw >> (8 * (e & 3))) & 255u) - (int)((cw >> (8 * (e & 3))) & 255u);
        s += t * t;
      }
    }
  }
  return s;
}

// sum over the 8 lanes of a survivor; every lane of the group gets the first lane's result
template <typename T>
__device__ __forceinline__ T group8_sum(T v, int lane) {
  v += __shfl_xor(v, 4);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 1);
  return __shfl(v, lane & ~7);
}

template <int FMT>
__global__ __launch_bounds__(256) void skm_refine_kernel(SkmArgs A) {
  constexpr int esz = FMT == KM_F32 ? 4 : 1;
  const int lane = threadIdx.x & 63;
  const int gl = lane >> 3, u = lane & 7;  // survivor slot, sub-lane
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nw = (int64_t)gridDim.x * 4;
  const int d = A.d, D0 = A.D0;
  unsigned long long full = 0;
  for (int64_t p = wid; p < A.n; p += nw) {  // waves stride over the points
    const int pj = min(max(A.prev[p], 0), A.k - 1);
    const Val<FMT> tau = static_cast<const Val<FMT> *>(A.tau)[p];
    const float tauf = (float)tau;
    Val<FMT> bd = tau;
    int best = pj;
    const uint8_t *x = A.X + p * A.xld;
    const uint32_t *mrow = A.mask + p * A.W4;
    for (int w0 = 0; w0 < A.W4; w0 += 64) {  // 64 mask words (2048 centroids) per load
      const uint32_t wv = w0 + lane < A.W4 ? mrow[w0 + lane] : 0u;
      uint64_t nz = __ballot(wv != 0u);
      uint32_t bits = 0u;
      int wbase = 0;
      while (nz || bits) {
        // the next group of survivors, in ascending index; slot gl of this lane
        int jl = 0, ng = 0;
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
          if (!bits && nz) {
            const int wl = __ffsll((unsigned long long)nz) - 1;
            nz &= nz - 1;
            bits = __shfl(wv, wl);
            wbase = (w0 + wl) * 32;
          }
          if (bits) {
            const int j = wbase + __ffs(bits) - 1;
            bits &= bits - 1;
            if (g == gl) jl = j;
            ng = g + 1;
          }
        }
        const bool mine = gl < ng;
        const uint8_t *c = A.C + (int64_t)jl * d * esz;
        Val<FMT> acc = 0;
        for (int b = 0; b < D0; b += 64) acc += group8_sum(mine ? sq8dims<FMT>(x, c, b + 8 * u, D0) : (Val<FMT>)0, lane);
        bool alive = mine;
        for (int m = 0, b = D0; b < d; ++m, b += 64) {
          if (!__ballot(alive)) break;
          acc += group8_sum(alive ? sq8dims<FMT>(x, c, b + 8 * u, d) : (Val<FMT>)0, lane);
          if (b + 64 < d && alive && (float)acc > tauf * A.rt[m]) alive = false;  // checkpoint inside the row
        }
        // survivors reaching the full distance, compared in ascending index
        const uint64_t am = __ballot(alive && u == 0);
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
          if ((am >> (8 * g)) & 1ull) {
            const Val<FMT> v = __shfl(acc, 8 * g);
            const int j = __shfl(jl, 8 * g);
            ++full;
            if (v < bd || (v == bd && j < best)) {
              bd = v;
              best = j;
            }
          }
        }
      }
    }
    if (lane == 0) {
      A.assign[p] = best;
      A.dist[p] = (double)bd;
    }
  }
  if (A.cnt && lane == 0) A.cnt[wid] = full;
}

__global__ __launch_bounds__(256) void skm_zero_kernel(unsigned long long *c) {
  if (threadIdx.x < 3) c[threadIdx.x] = 0ull;
}

// adds the partial counts of one pass to the running totals (one block, fixed order)
__global__ __launch_bounds__(256) void skm_count_kernel(const unsigned long long *front, int64_t nfront,
                                                        const unsigned long long *refine, int64_t nrefine,
                                                        unsigned long long *cnt) {
  __shared__ unsigned long long sh[3][256];
  unsigned long long a = 0, b = 0, c = 0;
  for (int64_t i = threadIdx.x; i < nfront; i += 256) {
    a += front[2 * i];
    b += front[2 * i + 1];
  }
  for (int64_t i = threadIdx.x; i < nrefine; i += 256) c += refine[i];
  sh[0][threadIdx.x] = a;
  sh[1][threadIdx.x] = b;
  sh[2][threadIdx.x] = c;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (threadIdx.x < st)
      for (int q = 0; q < 3; ++q) sh[q][threadIdx.x] += sh[q][threadIdx.x + st];
    __syncthreads();
  }
  if (threadIdx.x < 3) cnt[threadIdx.x] += sh[threadIdx.x][0];
}

// fixed-order sum of doubles: per-block partials, then one block
__global__ __launch_bounds__(256) void skm_partial_kernel(const double *v, int64_t n, double *part) {
  __shared__ double sh[256];
  double s = 0.0;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) s += v[i];
  s = block_sum_f64(s, sh);
  if (threadIdx.x == 0) part[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void skm_final_kernel(const double *part, int np, double *out) {
  __shared__ double sh[256];
  double s = 0.0;
  for (int i = threadIdx.x; i < np; i += 256) s += part[i];
  s = block_sum_f64(s, sh);
  if (threadIdx.x == 0) *out = s;
}

constexpr int kSumBlocks = 1024;
constexpr int kRefineBlocks = 4096;  // 16384 waves striding over the points

int64_t front_blocks(int64_t n, int k) {
  (void)k;
  return cdiv(n, kFT);
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

double prune_factor(int D, int d, double eps0) {
  const double g = 1.0 + eps0 / sqrt((double)D);
  return g * g * (double)D / (double)d;
}

int prune_front_default(int d) { return std::min(d, 32 * ((d + 255) / 256)); }

size_t pruned_bytes(const Points &P, int k) {
  const size_t n = (size_t)P.n;
  const size_t W4 = 4 * (size_t)cdiv(k, kFT);
  return al256(4 * n) + al256(4 * n) + al256(4 * (size_t)k) + al256(4 * W4 * n) + al256(8 * n) +
         al256(8 * kSumBlocks) + al256(16 * (size_t)front_blocks(P.n, k)) + al256(8 * 4 * (size_t)kRefineBlocks);
}

km_status launch_assign_pruned(const Points &P, const void *C, int k, const int32_t *prev, int32_t *assign,
                               double *dist, double *objective, double eps0, int D0,
                               unsigned long long *cnt, void *ws, hipStream_t s) {
  const int64_t n = P.n;
  const int d = P.d;
  const int W4 = 4 * (int)cdiv(k, kFT);
  uint8_t *w = static_cast<uint8_t *>(ws);
  void *tau = w;
  w += al256(4 * (size_t)n);
  void *xn = w;
  w += al256(4 * (size_t)n);
  void *cn = w;
  w += al256(4 * (size_t)k);
  uint32_t *mask = reinterpret_cast<uint32_t *>(w);
  w += al256(4 * (size_t)W4 * (size_t)n);
  double *dscratch = reinterpret_cast<double *>(w);
  w += al256(8 * (size_t)n);
  double *part = reinterpret_cast<double *>(w);
  w += al256(8 * kSumBlocks);
  unsigned long long *cfront = reinterpret_cast<unsigned long long *>(w);
  w += al256(16 * (size_t)front_blocks(n, k));
  unsigned long long *crefine = reinterpret_cast<unsigned long long *>(w);

  SkmArgs A{};
  A.n = n;
  A.d = d;
  A.k = k;
  A.X = static_cast<const uint8_t *>(P.data);
  A.xld = P.fmt == KM_F32 ? 4 * P.ld : P.ld;
  A.C = static_cast<const uint8_t *>(C);
  A.prev = prev;
  A.tau = tau;
  A.xn = xn;
  A.cn = cn;
  A.D0 = D0;
  A.W4 = W4;
  A.mask = mask;
  A.front_test = D0 < d;
  A.r0 = (float)prune_factor(D0, d, eps0);
  for (int m = 0; m < kMaxTail; ++m) {
    const int D = D0 + 64 * (m + 1);
    A.rt[m] = D < d ? (float)prune_factor(D, d, eps0) : 0.0f;
  }
  A.assign = assign;
  A.dist = dist ? dist : dscratch;
  A.cnt = nullptr;

  const dim3 rows_grid((unsigned)cdiv(n, 4));
  const int64_t nfb = front_blocks(n, k);
  const dim3 front_grid((unsigned)nfb);
  const unsigned nrb = (unsigned)std::min<int64_t>(kRefineBlocks, cdiv(n, 4));
  const dim3 refine_grid(nrb);
  SkmArgs Af = A, Ar = A;  // counts go to per-group / per-wave partials
  if (cnt) {
    Af.cnt = cfront;
    Ar.cnt = crefine;
  }
  const size_t cld = P.fmt == KM_F32 ? 4 * (size_t)d : (size_t)d;
  if (P.fmt == KM_F32) {
    hipLaunchKernelGGL(skm_norm_kernel<KM_F32>, rows_grid, dim3(256), 0, s, A.X, A.xld, n, D0, xn);
    hipLaunchKernelGGL(skm_norm_kernel<KM_F32>, dim3((unsigned)cdiv(k, 4)), dim3(256), 0, s, A.C, (int64_t)cld,
                       (int64_t)k, D0, cn);
    hipLaunchKernelGGL(skm_tau_kernel<KM_F32>, rows_grid, dim3(256), 0, s, A, tau);
    hipLaunchKernelGGL(skm_front_kernel<KM_F32>, front_grid, dim3(256), 0, s, Af);
    hipLaunchKernelGGL(skm_refine_kernel<KM_F32>, refine_grid, dim3(256), 0, s, Ar);
  } else if (P.fmt == KM_SQ8) {
    hipLaunchKernelGGL(skm_norm_kernel<KM_SQ8>, rows_grid, dim3(256), 0, s, A.X, A.xld, n, D0, xn);
    hipLaunchKernelGGL(skm_norm_kernel<KM_SQ8>, dim3((unsigned)cdiv(k, 4)), dim3(256), 0, s, A.C, (int64_t)cld,
                       (int64_t)k, D0, cn);
    hipLaunchKernelGGL(skm_tau_kernel<KM_SQ8>, rows_grid, dim3(256), 0, s, A, tau);
    hipLaunchKernelGGL(skm_front_kernel<KM_SQ8>, front_grid, dim3(256), 0, s, Af);
    hipLaunchKernelGGL(skm_refine_kernel<KM_SQ8>, refine_grid, dim3(256), 0, s, Ar);
  } else {
    return KM_EUNSUPPORTED;
  }
  if (cnt) hipLaunchKernelGGL(skm_count_kernel, dim3(1), dim3(256), 0, s, cfront, nfb, crefine, (int64_t)nrb * 4, cnt);
  KMQ_LAUNCH_CHECK("pruned assignment");
  if (objective) {
    const int nb = (int)std::min<int64_t>(kSumBlocks, std::max<int64_t>(1, cdiv(n, 256)));
    hipLaunchKernelGGL(skm_partial_kernel, dim3(nb), dim3(256), 0, s, A.dist, n, part);
    hipLaunchKernelGGL(skm_final_kernel, dim3(1), dim3(256), 0, s, part, nb, objective);
    KMQ_LAUNCH_CHECK("pruned objective");
  }
  return KM_OK;
}

km_status launch_zero_counters(unsigned long long *c, hipStream_t s) {
  hipLaunchKernelGGL(skm_zero_kernel, dim3(1), dim3(256), 0, s, c);
  KMQ_LAUNCH_CHECK("zero counters");
  return KM_OK;
}

}  // namespace kmq
