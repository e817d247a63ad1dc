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
template <int FMT>
__global__ __launch_bounds__(256) void skm_front_kernel(SkmArgs A) {
  __shared__ __align__(16) uint8_t lds[2][2][kFTile];  // [buffer][centroids, points]
  __shared__ Val<FMT> cnl[kFT];                       // front norms of the tile's centroids
  __shared__ __align__(16) uint32_t mrow[kFT][4];     // the tile's 4 mask words of each point
  constexpr bool F = FMT == KM_F32;
  constexpr int esz = F ? 4 : 1;
  using Acc = typename std::conditional<F, f32x16, i32x16>::type;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, r = lane & 31, h = lane >> 5;
  const int wc = w & 1, wp = w >> 1;
  // the centroid tiles of one point tile run on one XCD (ids are dealt round-robin)
  const int64_t npt = cdiv(A.n, kFT);
  const int nct = (int)cdiv(A.k, kFT);
  const int64_t id = blockIdx.x;
  const int64_t pt = ((id >> 3) / nct) * 8 + (id & 7);
  const int ct = (int)((id >> 3) % nct);
  if (pt >= npt) {
    if (A.cnt && t == 0) A.cnt[2 * id] = A.cnt[2 * id + 1] = 0ull;
    return;
  }
  const int64_t p0 = pt * kFT;
  const int c0 = ct * kFT;
  const int bytes = A.D0 * esz;
  const int nch = (bytes + kFRow - 1) / kFRow;

  Acc acc[2][2];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[cb][pb][v] = 0;

  uint4 rc[4], rp[4];
  auto load = [&](int ch) {
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
  };
  auto store = [&](int ch, int buf) {
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
  };

  if (t < kFT) cnl[t] = static_cast<const Val<FMT> *>(A.cn)[min(c0 + t, A.k - 1)];
  load(0);
  store(0, 0);
  __syncthreads();
  for (int ch = 0; ch < nch; ++ch) {
    const int buf = ch & 1;
    if (ch + 1 < nch) load(ch + 1);
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
    if (ch + 1 < nch) store(ch + 1, buf ^ 1);
    __syncthreads();
  }

  // epilogue: lane (r, h) holds centroid rows 8 (v >> 2) + 4 h + (v & 3) of each
  // 32 x 32 block for point column r
  unsigned long long tested = 0, passed = 0;
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) {
    const int64_t p = p0 + wp * 64 + pb * 32 + r;
    const int64_t pc = min<int64_t>(p, A.n - 1);
    const int pj = A.prev[pc];
    const Val<FMT> xn = static_cast<const Val<FMT> *>(A.xn)[pc];
    const float lim = (F ? static_cast<const float *>(A.tau)[pc] : (float)static_cast<const int *>(A.tau)[pc]) * A.r0;
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      const int jb = c0 + wc * 64 + cb * 32;  // first centroid of the block (multiple of 32)
      uint32_t m = 0;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int off = 8 * (v >> 2) + 4 * h + (v & 3);
        const int j = jb + off;
        const bool cand = p < A.n && j < A.k && j != pj;
        bool keep = true;
        if (A.front_test) {
          const Val<FMT> cnj = cnl[wc * 64 + cb * 32 + off];
          if constexpr (F) {
            const float pd = fmaf(-2.0f, acc[cb][pb][v], xn + cnj);
            keep = !(pd > lim);
          } else {
            const int pd = xn + cnj - 2 * acc[cb][pb][v];
            keep = !((float)pd > lim);
          }
        }
        const bool bit = cand && keep;
        m |= (bit ? 1u : 0u) << off;
        tested += A.front_test && cand;
        passed += A.front_test && bit;
      }
      m |= __shfl_xor(m, 32);
      if (h == 0) mrow[wp * 64 + pb * 32 + r][wc * 2 + cb] = m;
    }
  }
  __syncthreads();
  if (t < kFT && p0 + t < A.n)  // words 4 ct .. 4 ct + 3 of the point's row (rows padded to W4 words)
    *reinterpret_cast<uint4 *>(A.mask + (p0 + t) * A.W4 + 4 * ct) = *reinterpret_cast<const uint4 *>(mrow[t]);
  if (A.cnt) {  // per-workgroup partial counts (summed later in a fixed order)
    __shared__ unsigned long long cw[4][2];
    tested = wave_sum(tested);
    passed = wave_sum(passed);
    if (lane == 0) {
      cw[w][0] = tested;
      cw[w][1] = passed;
    }
    __syncthreads();
    if (t == 0) {
      A.cnt[2 * id] = cw[0][0] + cw[1][0] + cw[2][0] + cw[3][0];
      A.cnt[2 * id + 1] = cw[0][1] + cw[1][1] + cw[2][1] + cw[3][1];
    }
  }
}

// ---- refinement of the survivors: one wave per point ---------------------------
// The point's mask row is read first; a point without survivors keeps its previous
// centroid without touching its row.  Survivors are taken in groups of kGroup
// (ascending index): chunk by chunk, the group's loads and reductions are
// independent of each other, and every survivor stops at its first failed
// checkpoint.
constexpr int kGroup = 8;

template <int FMT>
__global__ __launch_bounds__(256) void skm_refine_kernel(SkmArgs A) {
  constexpr bool F = FMT == KM_F32;
  constexpr int esz = F ? 4 : 1;
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nw = (int64_t)gridDim.x * 4;
  const int d = A.d, D0 = A.D0;
  const int nf = (D0 + 63) >> 6, nt = (d - D0 + 63) >> 6;
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
        // the next group of survivors, in ascending index
        int jg[kGroup];
        int ng = 0;
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
          jg[g] = 0;
          if (!bits && nz) {
            const int wl = __ffsll((unsigned long long)nz) - 1;
            nz &= nz - 1;
            bits = __shfl(wv, wl);
            wbase = (w0 + wl) * 32;
          }
          if (bits) {
            jg[g] = wbase + __ffs(bits) - 1;
            bits &= bits - 1;
            ng = g + 1;
          }
        }
        Val<FMT> acc[kGroup];
        uint32_t alive = (1u << ng) - 1u;
#pragma unroll
        for (int g = 0; g < kGroup; ++g) acc[g] = 0;
#pragma unroll
        for (int m = 0; m < kMaxFront; ++m) {
          if (m < nf) {
            const int i = 64 * m + lane;
            const Val<FMT> xv = i < D0 ? elem<FMT>(x, i) : (Val<FMT>)0;
            Val<FMT> cv[kGroup];
#pragma unroll
            for (int g = 0; g < kGroup; ++g)
              cv[g] = (g < ng && i < D0) ? elem<FMT>(A.C + (int64_t)jg[g] * d * esz, i) : xv;
#pragma unroll
            for (int g = 0; g < kGroup; ++g) {
              if (g < ng) {
                const Val<FMT> t = xv - cv[g];
                acc[g] += wave_sum(t * t);
              }
            }
          }
        }
#pragma unroll
        for (int m = 0; m < kMaxTail; ++m) {
          if (m < nt && alive) {
            const int i = D0 + 64 * m + lane;
            const Val<FMT> xv = i < d ? elem<FMT>(x, i) : (Val<FMT>)0;
            Val<FMT> cv[kGroup];
#pragma unroll
            for (int g = 0; g < kGroup; ++g)
              cv[g] = ((alive >> g) & 1u) && i < d ? elem<FMT>(A.C + (int64_t)jg[g] * d * esz, i) : xv;
            const bool inside = D0 + 64 * (m + 1) < d;  // a checkpoint inside the row
#pragma unroll
            for (int g = 0; g < kGroup; ++g) {
              if ((alive >> g) & 1u) {
                const Val<FMT> t = xv - cv[g];
                acc[g] += wave_sum(t * t);
                if (inside && (float)acc[g] > tauf * A.rt[m]) alive &= ~(1u << g);
              }
            }
          }
        }
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
          if ((alive >> g) & 1u) {  // compared on the full distance, in ascending index
            ++full;
            if (acc[g] < bd || (acc[g] == bd && jg[g] < best)) {
              bd = acc[g];
              best = jg[g];
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

int64_t front_blocks(int64_t n, int k) { return cdiv(cdiv(n, kFT), 8) * 8 * cdiv(k, kFT); }

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
