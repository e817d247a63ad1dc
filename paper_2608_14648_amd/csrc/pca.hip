// PCA before clustering (Sec. 3.1 "PCA"; Sec. 4.2): covariance of the centred
// points and the projection onto the leading principal directions, both as
// fp32 MFMA contractions (v_mfma_f32_32x32x2_f32).
//
// Covariance: the d x d output is cut into 256 x 256 tiles (upper triangle only,
// mirrored at the end) and the n rows are split across workgroups.  Each stage
// copies 32 rows x 256 columns of both column blocks into LDS, centred when read.
// The fp32 accumulators are added into a per-workgroup fp64 partial tile every
// 8192 rows, and the partial tiles are folded in split order.
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
constexpr int kFlushStages = 256;  // 8192 rows per fp32 accumulation run

__device__ __forceinline__ void tile_ij(int t, int T, int &ti, int &tj) {
  // enumerate the upper triangle row by row
  ti = 0;
  while (t >= T - ti) {
    t -= T - ti;
    ++ti;
  }
  tj = ti + t;
}

// Direct copy of 16 bytes per lane from global memory into LDS: the wave's 64 lanes
// fill 1 KB at LDS byte address lds (wave-uniform) in lane order, from a
// wave-uniform base plus a 32-bit per-lane byte offset.  Inline assembly, so that
// the compiler does not wait for the copy before the LDS reads of the other stage
// buffer; the caller waits (vmcnt) before the barrier that publishes the data.
typedef __attribute__((address_space(3))) uint8_t lds_u8;
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_copy16(const void *base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// One workgroup per (256 x 256 output tile, run of rows): 8 waves, two per SIMD,
// each owning 128 x 64 of the tile as 4 x 2 blocks of 32 x 32 (fp32 MFMA; rows are
// the contraction index, read column-wise from row-major LDS stages).  A stage is
// 32 rows of both 256-column blocks, copied straight from global memory into LDS,
// one 1 KB row-block per wave instruction (rows padded to 260 floats); the rows
// are centred when the MFMA operands are read (x - mean in fp32, the same operand
// a centring copy would store).  Rows past the end of the run are filled with the
// mean itself, so their centred values are exactly zero; columns past d are
// zero-filled and their outputs dropped by the reduction.  The copies of stage
// st + 1 go out during stage st's four steps.  Every 8192 rows the fp32
// accumulators are added into this workgroup's own fp64 partial tile in global
// memory (read-modify-write, no other workgroup touches it); the fold is a
// synchronous read-modify-write of 128 values per lane, so shorter runs cost
// (2048 rows: 7 % slower).
constexpr int kCovThreads = 512;

__global__ __launch_bounds__(kCovThreads, 1) void cov_kernel(const float *X, int64_t n, int d, const float *mean, int T,
                                                             int ntiles, int64_t rows_per_split, double *partial) {
  constexpr int BS = kCovRows * kCovStride;  // floats of one column block of a stage
  __shared__ __align__(16) float stA0[2 * BS];
  __shared__ __align__(16) float stA1[2 * BS];
  const int tile = blockIdx.x % ntiles;
  const int split = blockIdx.x / ntiles;
  int ti, tj;
  tile_ij(tile, T, ti, tj);
  const int i0 = ti * kCT, j0 = tj * kCT;
  const int64_t rb = (int64_t)split * rows_per_split;
  const int64_t re = min<int64_t>(n, rb + rows_per_split);
  const int t = threadIdx.x, lane = t & 63, wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int wi = wave & 1, wj = wave >> 1;
  double *out = partial + ((int64_t)split * ntiles + tile) * (kCT * kCT);
  const int nst = (int)cdiv(max<int64_t>(re - rb, 0), kCovRows);

  // the means of this lane's operand columns
  float mi[4], mj[2];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) mi[cb] = mean[min(i0 + wi * 128 + cb * 32 + r, d - 1)];
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) mj[pb] = mean[min(j0 + wj * 64 + pb * 32 + r, d - 1)];

  // the fill of a row past the run: the means of this lane's four columns of each
  // block (zeros past d), held in registers so that no load the compiler tracks
  // sits among the copies
  f32x4 fill[2];
#pragma unroll
  for (int blk = 0; blk < 2; ++blk) {
    const int col = (blk ? j0 : i0) + 4 * lane;
    fill[blk] = col < d ? *reinterpret_cast<const f32x4 *>(mean + col) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // copy q (0 .. 7) of wave w: row-block c = 8 q + w, column block c >> 5, row c & 31
  auto copy = [&](int st, float *dst, int q) {
    const int c = 8 * q + wave;
    const int blk = c >> 5, row = c & 31;
    const int col = (blk ? j0 : i0) + 4 * lane;
    float *w = dst + blk * BS + row * kCovStride;
    const int64_t gr = rb + (int64_t)st * kCovRows + row;
    if (gr < re && col < d) {
      lds_copy16(X + gr * d + (blk ? j0 : i0), (uint32_t)(16 * lane), (uint32_t)(size_t)(lds_u8 *)(w));
    } else {
      // a row past the run holds the mean (centred: zero); a column past d zeros
      *reinterpret_cast<f32x4 *>(w + 4 * lane) = gr >= re ? fill[blk] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  auto land = [&]() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  f32x16 acc[4][2];
  // one stage: 16 row pairs in 4 steps of 4; the operand reads of step g + 1 and
  // two of the next stage's copies go out before step g's MFMAs
  auto mfma_stage = [&](const float *buf, bool copying, int st_n, float *nxt) {
    const float *A = buf;
    const float *B = buf + BS;
    float av[2][4][4], bv[2][4][2];
    auto read = [&](int g, int set) {
#pragma unroll
      for (int pp = 0; pp < 4; ++pp) {
        const int row = 2 * (4 * g + pp) + h;
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) av[set][pp][cb] = A[row * kCovStride + wi * 128 + cb * 32 + r] - mi[cb];
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) bv[set][pp][pb] = B[row * kCovStride + wj * 64 + pb * 32 + r] - mj[pb];
      }
    };
    read(0, 0);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int cur = g & 1;
      if (g + 1 < 4) read(g + 1, cur ^ 1);
      __builtin_amdgcn_sched_barrier(0);
      if (copying) {
        copy(st_n, nxt, 2 * g);
        copy(st_n, nxt, 2 * g + 1);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int pp = 0; pp < 4; ++pp)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
          for (int pb = 0; pb < 2; ++pb)
            acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[cur][pp][cb], bv[cur][pp][pb], acc[cb][pb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  if (nst > 0) {
#pragma unroll
    for (int q = 0; q < 8; ++q) copy(0, stA0, q);
    land();
  }
  __syncthreads();
  const int nrun = (nst + kFlushStages - 1) / kFlushStages;
  for (int run = 0; run < nrun; ++run) {
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;
    const int st1 = min(nst, (run + 1) * kFlushStages);
    for (int st = run * kFlushStages; st < st1; ++st) {
      const bool nxt = st + 1 < nst;
      mfma_stage((st & 1) ? stA1 : stA0, nxt, st + 1, (st & 1) ? stA0 : stA1);
      if (nxt) land();
      __syncthreads();
    }
    // the lane's offset passes through an empty asm statement so that the element
    // addresses are formed here, not hoisted out of the run loop (they would hold
    // 128 register pairs for the whole loop); the pointer itself stays a global one
    // (a flat access here would make every LDS wait of the stage loop wait for
    // the copies too)
    int boff = (wi * 128 + 4 * h) * kCT + wj * 64 + r;
    asm volatile("" : "+v"(boff));
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          double *o = out + boff + (cb * 32 + 8 * (v >> 2) + (v & 3)) * kCT + pb * 32;
          *o = (run == 0 ? 0.0 : *o) + (double)acc[cb][pb][v];
        }
  }
  if (nrun == 0) {  // no rows: the partial tile is zero
    for (int e = t; e < kCT * kCT; e += kCovThreads) out[e] = 0.0;
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
__global__ __launch_bounds__(256) void project_staged_kernel(const float *X, int64_t n, int d, int64_t ldx,
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

// Projection, direct-copy design (d <= kProjMaxD, ldx % 4 == 0, 256 rows of X
// within 2 GB): the 8-wave shape of the fp32 assignment kernel with the points as
// the first MFMA operand and the rows of W^T as the second, so a lane's outputs
// are consecutive output dims of one point and the stores are coalesced.  A
// workgroup computes 256 points x 256 outputs; stages of 32 dims (128 bytes of
// every row: 256 point rows, then 256 rows of W^T) are copied straight from global
// memory into LDS in the XOR slot layout (chunk c of row R in slot c ^ ((R >> 1) &
// 7)), two stage buffers, one workgroup per CU.  The mean sits in LDS (zero past
// d) and the point operands are centred as they are read (x - mean in fp32, the
// value a centring copy would store).  Chunks past d are zero-filled; rows past n
// or d_out are clamped to the last one and their outputs are not stored.
constexpr int kProjMaxD = 4096;
constexpr int kPT = 256;  // points and outputs per workgroup

__global__ __launch_bounds__(512, 1) void project_kernel(const float *X, int64_t n, int d, int64_t ldx,
                                                         const float *mean, const float *Wt, int d_out, float *Y,
                                                         int n_ptiles, int n_otiles) {
  constexpr int NCP = kPT / 64;            // point copies per thread and stage
  constexpr int NCOPY = 2 * kPT / 64;      // all copies per thread and stage
  constexpr int STAGE = 2 * kPT * 128;     // bytes: point rows, then W^T rows
  __shared__ __align__(16) uint8_t pst0[STAGE];
  __shared__ __align__(16) uint8_t pst1[STAGE];
  __shared__ __align__(16) float msh[kProjMaxD + 32];
  // workgroup ids, tiles and bases are wave-uniform: computed in 32 bits and
  // pinned to scalar registers (the copies take their bases there)
  const int b = (int)blockIdx.x;
  const int group = __builtin_amdgcn_readfirstlane(b / (8 * n_otiles));  // 8 point tiles per group
  const int rem = __builtin_amdgcn_readfirstlane(b % (8 * n_otiles));
  const int ptile = group * 8 + rem % 8;
  const int otile = rem / 8;
  if (ptile >= n_ptiles) return;  // whole workgroup, before any barrier
  const int64_t p0 = (int64_t)ptile * kPT;
  const int o0 = otile * kPT;
  const int t = threadIdx.x, lane = t & 63, wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int wc = wave & 1, wp = wave >> 1;  // 128-point half, 64-output quarter
  const int prmax = (int)min<int64_t>(n - 1 - p0, kPT - 1);
  const int ormax = min(d_out - 1 - o0, kPT - 1);
  const int S = (d + 31) / 32;
  for (int i = t; i < 32 * S; i += 512) msh[i] = i < d ? mean[i] : 0.f;
  const float *xbase = X + p0 * ldx;
  const float *wbase = Wt + (int64_t)o0 * d;

  // copy i of a wave fills slots (8 i + wave) 64 .. + 63: rows 0 .. 255 are points,
  // rows 256 .. 511 rows of W^T; byte offsets from the stage's first dim
  uint32_t soff[NCOPY];
#pragma unroll
  for (int i = 0; i < NCOPY; ++i) {
    const int slot = (i * 8 + wave) * 64 + lane;
    const int row = slot >> 3;
    const int chunk = (slot & 7) ^ ((row >> 1) & 7);
    soff[i] = i < NCP ? (uint32_t)(min(row, prmax) * (int)ldx * 4 + 16 * chunk)
                      : (uint32_t)(min(row - kPT, ormax) * d * 4 + 16 * chunk);
  }
  auto copy = [&](int st, uint8_t *dst, int i) {
    const int slot = (i * 8 + wave) * 64 + lane;
    const int row = slot >> 3;
    const int chunk = (slot & 7) ^ ((row >> 1) & 7);
    lds_u8 *w = (lds_u8 *)dst + (i * 8 + wave) * 1024;
    // the stage's first dim of the points or of W^T, pinned to scalar registers
    const float *src = (i < NCP ? xbase : wbase) + 32 * st;
    const uint64_t su = (uint64_t)(size_t)src;
    const void *base = (const void *)(size_t)(((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(su >> 32)) << 32) |
                                              (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)su));
    if (32 * st + 4 * chunk < d) {
      lds_copy16(base, soff[i], (uint32_t)(size_t)w);
    } else {
      __attribute__((address_space(3))) uint32_t *z = (__attribute__((address_space(3))) uint32_t *)(w + 16 * lane);
      z[0] = z[1] = z[2] = z[3] = 0u;
    }
  };
  auto land = [&]() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  f32x16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][c][v] = 0.f;
  // one stage: four steps of 8 dims; the operand reads of step g + 1 and two of
  // the next stage's copies go out before step g's MFMAs
  auto mfma_stage = [&](int st, const uint8_t *buf, bool copying, uint8_t *nxt) {
    f32x4 av[2][4], bv[2][2];
    auto read = [&](int g, int set) {
      const int so = 16 * ((2 * g + h) ^ ((r >> 1) & 7));
      const f32x4 m4 = *reinterpret_cast<const f32x4 *>(&msh[32 * st + 8 * g + 4 * h]);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        av[set][cb] = *reinterpret_cast<const f32x4 *>(buf + (wc * 128 + cb * 32 + r) * 128 + so) - m4;
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
        bv[set][pb] = *reinterpret_cast<const f32x4 *>(buf + (kPT + wp * 64 + pb * 32 + r) * 128 + so);
    };
    read(0, 0);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int cur = g & 1;
      if (g + 1 < 4) read(g + 1, cur ^ 1);
      __builtin_amdgcn_sched_barrier(0);
      if (copying) {
        copy(st + 1, nxt, 2 * g);
        copy(st + 1, nxt, 2 * g + 1);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
          for (int pb = 0; pb < 2; ++pb)
            acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[cur][cb][e], bv[cur][pb][e], acc[cb][pb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

#pragma unroll
  for (int i = 0; i < NCOPY; ++i) copy(0, pst0, i);
  land();
  __syncthreads();  // also publishes the mean
  for (int st = 0; st < S; ++st) {
    const bool nxt = st + 1 < S;
    mfma_stage(st, (st & 1) ? pst1 : pst0, nxt, (st & 1) ? pst0 : pst1);
    if (nxt) land();
    __syncthreads();
  }
  // lane (r, h) of block (cb, pb) holds points wc 128 + cb 32 + 8 i4 + 4 h + e of
  // output wp 64 + pb 32 + r
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const int o = o0 + wp * 64 + pb * 32 + r;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t p = p0 + wc * 128 + cb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        if (p < n && o < d_out) Y[p * d_out + o] = acc[cb][pb][v];
      }
    }
}

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
  hipLaunchKernelGGL(cov_kernel, dim3(p.ntiles * p.nsplit), dim3(kCovThreads), 0, s, X, n, d, mean, p.T, p.ntiles,
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
  if (d <= kProjMaxD && ldx % 4 == 0 && (int64_t)kPT * ldx * 4 < ((int64_t)1 << 31)) {
    const int n_ptiles = (int)cdiv(n, kPT), n_otiles = (int)cdiv(d_out, kPT);
    const int64_t nblk = cdiv(n_ptiles, 8) * 8 * n_otiles;
    hipLaunchKernelGGL(project_kernel, dim3((unsigned)nblk), dim3(512), 0, s, X, n, d, ldx, mean, Wt, d_out, Y,
                       n_ptiles, n_otiles);
  } else {
    const int n_ptiles = (int)cdiv(n, kT), n_otiles = (int)cdiv(d_out, kT);
    const int64_t nblk = cdiv(n_ptiles, 8) * 8 * n_otiles;
    hipLaunchKernelGGL(project_staged_kernel, dim3((unsigned)nblk), dim3(256), 0, s, X, n, d, ldx, mean, Wt, d_out,
                       Y, n_ptiles, n_otiles);
  }
  KMQ_LAUNCH_CHECK("pca_project");
  return KM_OK;
}

}  // namespace kmq
