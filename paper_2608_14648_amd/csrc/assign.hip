// STEP 2 (Sec. 2.3): nearest-centroid assignment as a fused MFMA contraction with
// an in-register running argmin, plus the small kernels around it (centroid
// preparation, point-only terms, objective sum, initial gather, partition cost).
//
// Fused assignment kernel
// -----------------------
// One workgroup (256 threads, 4 waves) owns 128 points and sweeps every centroid
// in tiles of 128.  For a (centroid tile, point tile) pair the dot products
// <c, x> are accumulated over d on the matrix cores with the CENTROIDS as the
// MFMA row operand and the POINTS as the column operand, so each lane of the
// 32x32 output block holds 16 centroid rows of ONE point column: the argmin over
// centroids is then a lane-local compare-select, never a cross-lane shuffle,
// and the n x k score matrix never leaves registers.
//   - fp32 points (raw / PCA / hybrid front): v_mfma_f32_32x32x2_f32.
//   - SQ8 codes: code - 128 as int8 on both sides, v_mfma_i32_32x32x32_i8;
//     score = ||c~||^2 - 2 <x~, c~> is an exact int32.
//   - 1-bit codes: each bit is widened to a {0,1} byte while the tile is staged
//     in LDS, and multiplied with the centroid's int8 residual codes q on the
//     int8 matrix cores: D = sum of q on set bits, and <2b-1, q> = 2D - T (Eq. 5
//     with x_bar in {0,1}).  The fp32 epilogue follows Eq. 4 with the point's
//     cached scale alpha: score = fmaf(-(alpha * 2 sigma), 2D - T, sigma^2 Q).
//   - hybrid: an fp32 phase over the front dims and an int8 phase over the
//     1-bit tail accumulate separately; the scores add (segment decomposition
//     of the squared L2 distance, Sec. 3.1 SuperKMeans).
// Stages are 128 bytes of every row (32 floats or 128 int8 lanes), staged
// global -> registers -> LDS with double buffering and one barrier per stage.
// Both operands of an MFMA read 16 contiguous bytes per lane from the same
// LDS column offset, so the k-index permutation inside the instruction is the
// same on both sides and cancels in the dot product.
// Ties: within a lane candidates arrive in increasing centroid index and are
// taken only on a strict improvement; lanes and waves merge on (score, index),
// so the smallest index wins every exact tie.
#include <float.h>
#include <limits.h>

#include <algorithm>
#include <type_traits>

#include "common.hpp"

namespace kmq {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = 128;              // bytes of one row per stage
constexpr int kLdsStride = kRowBytes + 16;  // padded to spread LDS banks

struct AssignArgs {
  // fp32 phase: F32 points, hybrid front
  const float *pf;
  int64_t pfld;
  const float *cf;
  int64_t cfld;
  int df;
  // integer phase: SQ8 codes or 1-bit tail
  const uint8_t *pi8;
  int64_t pild;
  const uint32_t *pbits;
  int64_t pbw;  // words per 1-bit row
  int pbw0;     // first word of the integer phase
  const int8_t *ci8;
  int64_t cild;
  int di;
  const float *alpha;
  const float *vparams;  // LVQ4: per-point (s, b, A, N)
  CentroidPrep cp;
  int64_t n;
  int k;
  int32_t *assign;
  float *score;
  int aoff;  // added to every stored centroid index (a slice of a larger centroid set)
  // centroid-tile groups: workgroup (pt, g) scans centroid tiles g, g + ngroups, ...
  // of point tile pt and merges its argmin into keys[] (used when ngroups > 1)
  int ngroups;
  int64_t n_ptiles;
  unsigned long long *keys;
  // segmented launch (fp32): workgroup b takes point tile tiles[b].y of segment
  // tiles[b].x; segment i is rows [segs[i].x, + segs[i].y) against centroids
  // [segs[i].z, + segs[i].w) (indices into the full centroid and prepared arrays)
  const int4 *segs;
  const int2 *tiles;
};

// (score, index) as one 64-bit key whose unsigned order is the lexicographic
// order of (score, index): the fp32 pattern is mapped to an order-preserving
// unsigned integer (negative values complemented, positive ones offset by the
// sign bit), -0 taken as +0 so that equal scores tie on the index.
__device__ __forceinline__ unsigned long long score_key(float sc, int idx) {
  uint32_t u = __float_as_uint(sc == 0.0f ? 0.0f : sc);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)u << 32) | (uint32_t)idx;
}

// the same for an exact int32 score: the sign bit flipped is an order-preserving
// unsigned image
__device__ __forceinline__ unsigned long long int_score_key(int sc, int idx) {
  return ((unsigned long long)((uint32_t)sc ^ 0x80000000u) << 32) | (uint32_t)idx;
}

__device__ __forceinline__ float key_score(unsigned long long key) {
  uint32_t u = (uint32_t)(key >> 32);
  u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint32_t spread4(uint32_t b4) {
  // 4 bits -> 4 bytes holding 0 or 1 (bit j -> byte j)
  return (b4 * 0x00204081u) & 0x01010101u;
}

template <int FMT>
struct Cfg {
  static constexpr bool kFp = (FMT == KM_F32 || FMT == KM_HYBRID);
  static constexpr bool kInt = (FMT != KM_F32);
  static constexpr bool kBits = (FMT == KM_SIGN1 || FMT == KM_HYBRID);
  static constexpr bool kIntScore = (FMT == KM_SQ8);
};

// Raw loads of one stage (consumed only when the stage is written to LDS, one MFMA
// stage later, so the global latency hides under the matrix work).
// Tile geometry: waves are 2 (centroid halves) x 2 (point halves); each wave owns
// CB x PB blocks of 32 x 32, so a tile holds TC = 64 CB centroids and the
// workgroup TP = 64 PB points.
template <int CB, int PB>
struct Geo {
  static constexpr int TC = 64 * CB;
  static constexpr int TP = 64 * PB;
  static constexpr int CBYTES = TC * kLdsStride;
  static constexpr int PBYTES = TP * kLdsStride;
  static constexpr int STAGE = CBYTES + PBYTES;
  static constexpr int NC = TC / 32;  // 16-byte chunks of centroid rows per thread per stage
  static constexpr int NP = TP / 32;
  static_assert(TC <= kThreads, "one thread per tile centroid for the per-tile constants");
};

template <int CB, int PB>
struct StageRegs {
  uint4 c[Geo<CB, PB>::NC];
  uint4 p[Geo<CB, PB>::NP];
  float cpar[4];  // per-centroid constants of the next tile (stage 0 only)
};

__device__ __forceinline__ uint4 mask4(uint4 v, bool ok) {
  return make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
}

__device__ __forceinline__ uint4 flip4(uint4 v) {
  // uint8 code -> int8 (code - 128) in every byte
  return make_uint4(v.x ^ 0x80808080u, v.y ^ 0x80808080u, v.z ^ 0x80808080u, v.w ^ 0x80808080u);
}

// Stage order inside a centroid tile: fp32 formats have only fp32 stages, the
// integer formats only int8 stages; the hybrid runs its int8 (1-bit tail) stages
// first and its fp32 (front) stages after, so the two accumulators are never
// live together.  SI is the number of int8 stages.
template <int FMT>
__device__ __forceinline__ bool is_fp_stage(int s, int SI) {
  if constexpr (FMT == KM_F32) return true;
  else if constexpr (FMT == KM_HYBRID) return s >= SI;
  else return false;
}

template <int FMT>
__device__ __forceinline__ int fp_index(int s, int SI) {
  return FMT == KM_HYBRID ? s - SI : s;
}

// Every address is clamped into its buffer; lanes outside the data are zeroed at
// store time, so the loads are unconditional and branch-free.
template <int FMT, int CB, int PB>
__device__ __forceinline__ void load_stage(const AssignArgs &A, int s, int SI, int64_t c0, int64_t p0,
                                           StageRegs<CB, PB> &R) {
  typedef Geo<CB, PB> G;
  const int t = threadIdx.x;
  const int crmax = (int)min<int64_t>(A.k - 1 - c0, G::TC - 1);
  const int prmax = (int)min<int64_t>(A.n - 1 - p0, G::TP - 1);
  if (is_fp_stage<FMT>(s, SI)) {
    const float *cbase = A.cf + c0 * A.cfld;
    const float *pbase = A.pf + p0 * A.pfld;
    const int dim0 = 32 * fp_index<FMT>(s, SI);
#pragma unroll
    for (int i = 0; i < G::NC; ++i) {
      const int cidx = t + kThreads * i;
      const int row = cidx >> 3, col = cidx & 7;
      const int dim = dim0 + 4 * col;
      const int dimc = dim < A.df ? dim : 0;
      R.c[i] = *reinterpret_cast<const uint4 *>(cbase + (uint32_t)(min(row, crmax) * (int)A.cfld + dimc));
    }
#pragma unroll
    for (int i = 0; i < G::NP; ++i) {
      const int cidx = t + kThreads * i;
      const int row = cidx >> 3, col = cidx & 7;
      const int dim = dim0 + 4 * col;
      const int dimc = dim < A.df ? dim : 0;
      R.p[i] = *reinterpret_cast<const uint4 *>(pbase + (uint32_t)(min(row, prmax) * (int)A.pfld + dimc));
    }
  } else if constexpr (Cfg<FMT>::kInt) {
    const int si = s;
    const int b0 = kRowBytes * si;
    const int8_t *cbase = A.ci8 + c0 * A.cild;
#pragma unroll
    for (int i = 0; i < G::NC; ++i) {
      const int cidx = t + kThreads * i;
      const int row = cidx >> 3, col = cidx & 7;
      const int b = b0 + 16 * col;
      const int bc = b < A.di ? b : 0;
      R.c[i] = *reinterpret_cast<const uint4 *>(cbase + (uint32_t)(min(row, crmax) * (int)A.cild + bc));
    }
    if (FMT == KM_SQ8) {
      const uint8_t *pbase = A.pi8 + p0 * A.pild;
#pragma unroll
      for (int i = 0; i < G::NP; ++i) {
        const int cidx = t + kThreads * i;
        const int row = cidx >> 3, col = cidx & 7;
        const int b = b0 + 16 * col;
        const int bc = b < A.di ? b : 0;
        R.p[i] = *reinterpret_cast<const uint4 *>(pbase + (uint32_t)(min(row, prmax) * (int)A.pild + bc));
      }
    }
    if (Cfg<FMT>::kBits) {
      // TP rows x 4 words; NP/2 words per thread, kept in the .x lanes
      const uint32_t *pbase = A.pbits + p0 * A.pbw + A.pbw0;
#pragma unroll
      for (int i = 0; i < G::NP / 2; ++i) {
        const int w = t + kThreads * i;
        const int row = w >> 2, wi = w & 3;
        const int word = 4 * si + wi;
        R.p[i].x = pbase[(uint32_t)(min(row, prmax) * (int)A.pbw + (32 * word < A.di ? word : 0))];
      }
    }
  }
  if (s == 0) {
#pragma unroll
    for (int q = 0; q < G::TC / kThreads + (G::TC % kThreads ? 1 : 0); ++q) {
      const int jt = t + kThreads * q;
      if (jt < G::TC) {
        const int64_t j = c0 + min(jt, crmax);
        // rows past k get an infinite norm: their fp scores are +inf and never win
        if (Cfg<FMT>::kFp) R.cpar[0] = jt <= crmax ? A.cp.cn[j] : INFINITY;
        if (Cfg<FMT>::kInt) R.cpar[1] = __int_as_float(A.cp.qsum[j]);
        if (Cfg<FMT>::kBits) {
          R.cpar[2] = A.cp.u[j];
          R.cpar[3] = A.cp.sig2[j];
        }
      }
    }
  }
}

template <int FMT, int CB, int PB>
__device__ __forceinline__ void store_stage(const AssignArgs &A, int s, int SI, const StageRegs<CB, PB> &R,
                                            uint8_t *buf, float *cpar) {
  typedef Geo<CB, PB> G;
  const int t = threadIdx.x;
  uint8_t *ct = buf;
  uint8_t *pt = buf + G::CBYTES;
  const bool fp = is_fp_stage<FMT>(s, SI);
  const int si = s;
  const int sf = fp_index<FMT>(s, SI);
#pragma unroll
  for (int i = 0; i < G::NC; ++i) {
    const int cidx = t + kThreads * i;
    const int row = cidx >> 3, col = cidx & 7;
    const bool ok = fp ? (32 * sf + 4 * col < A.df) : (kRowBytes * si + 16 * col < A.di);
    uint4 cv = R.c[i];
    if (FMT == KM_SQ8) cv = flip4(cv);
    *reinterpret_cast<uint4 *>(ct + row * kLdsStride + 16 * col) = mask4(cv, ok);
  }
  if (fp || FMT == KM_SQ8) {
#pragma unroll
    for (int i = 0; i < G::NP; ++i) {
      const int cidx = t + kThreads * i;
      const int row = cidx >> 3, col = cidx & 7;
      const bool ok = fp ? (32 * sf + 4 * col < A.df) : (kRowBytes * si + 16 * col < A.di);
      uint4 pv = R.p[i];
      if (!fp) pv = flip4(pv);
      *reinterpret_cast<uint4 *>(pt + row * kLdsStride + 16 * col) = mask4(pv, ok);
    }
  } else if (Cfg<FMT>::kBits) {
    // each 32-bit code word widened to 32 bytes holding 0 or 1
#pragma unroll
    for (int i = 0; i < G::NP / 2; ++i) {
      const int w = t + kThreads * i;
      const int row = w >> 2, wi = w & 3;
      const uint32_t bits = (32 * (4 * si + wi) < A.di) ? R.p[i].x : 0u;
      *reinterpret_cast<uint4 *>(pt + row * kLdsStride + 32 * wi) =
          make_uint4(spread4(bits & 15u), spread4((bits >> 4) & 15u), spread4((bits >> 8) & 15u),
                     spread4((bits >> 12) & 15u));
      *reinterpret_cast<uint4 *>(pt + row * kLdsStride + 32 * wi + 16) =
          make_uint4(spread4((bits >> 16) & 15u), spread4((bits >> 20) & 15u), spread4((bits >> 24) & 15u),
                     spread4(bits >> 28));
    }
  }
  if (s == 0) {
#pragma unroll
    for (int q = 0; q < G::TC / kThreads + (G::TC % kThreads ? 1 : 0); ++q) {
      const int jt = t + kThreads * q;
      if (jt < G::TC) {
#pragma unroll
        for (int c = 0; c < 4; ++c) cpar[c * G::TC + jt] = R.cpar[c];
      }
    }
  }
}

template <int CB, int PB, bool FP>
__device__ __forceinline__ void mfma_stage(const uint8_t *cbuf, const uint8_t *pbuf, int wc, int wp, int r, int h,
                                           f32x16 (&facc)[CB][PB], i32x16 (&iacc)[CB][PB]) {
  uint4 av[2][CB], bv[2][PB];  // [register set][block]
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
    av[0][cb] = *reinterpret_cast<const uint4 *>(cbuf + (wc * 32 * CB + cb * 32 + r) * kLdsStride + 16 * h);
#pragma unroll
  for (int pb = 0; pb < PB; ++pb)
    bv[0][pb] = *reinterpret_cast<const uint4 *>(pbuf + (wp * 32 * PB + pb * 32 + r) * kLdsStride + 16 * h);
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int cur = g & 1, nxt = cur ^ 1;
    if (g + 1 < 4) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        av[nxt][cb] = *reinterpret_cast<const uint4 *>(cbuf + (wc * 32 * CB + cb * 32 + r) * kLdsStride +
                                                       32 * (g + 1) + 16 * h);
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
        bv[nxt][pb] = *reinterpret_cast<const uint4 *>(pbuf + (wp * 32 * PB + pb * 32 + r) * kLdsStride +
                                                       32 * (g + 1) + 16 * h);
    }
    if constexpr (FP) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int pb = 0; pb < PB; ++pb)
            facc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(av[cur][cb][e]),
                                                                __uint_as_float(bv[cur][pb][e]), facc[cb][pb], 0, 0, 0);
    } else {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          const i32x4 a4 = {(int)av[cur][cb].x, (int)av[cur][cb].y, (int)av[cur][cb].z, (int)av[cur][cb].w};
          const i32x4 b4 = {(int)bv[cur][pb].x, (int)bv[cur][pb].y, (int)bv[cur][pb].z, (int)bv[cur][pb].w};
          iacc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a4, b4, iacc[cb][pb], 0, 0, 0);
        }
    }
  }
}

// Register blocking per format: 2 x 2 blocks per wave (128-centroid tiles, 128
// points per workgroup), two workgroups per CU so that one's barrier and LDS
// refill hide under the other's MFMAs (measured faster than 4 x 2 blocks at one
// workgroup per CU).
template <int FMT>
struct Blocking {
  static constexpr int CB = 2;
  static constexpr int PB = 2;
  static constexpr int MINB = 2;
};

template <int FMT>
__global__ __launch_bounds__(kThreads, Blocking<FMT>::MINB) void assign_kernel(AssignArgs A) {
  constexpr int CB = Blocking<FMT>::CB, PB = Blocking<FMT>::PB;
  typedef Geo<CB, PB> G;
  __shared__ __align__(16) uint8_t lds[2 * G::STAGE];
  __shared__ __align__(16) float cparl[2][4 * G::TC];
  typedef typename std::conditional<Cfg<FMT>::kIntScore, int, float>::type score_t;

  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int wc = wave & 1, wp = wave >> 1;
  // With ngroups > 1 the ngroups workgroups of one point tile are consecutive
  // among the workgroups of one XCD (dispatch deals workgroup ids round-robin to
  // the 8 XCDs), so the re-reads of the point tile, one per centroid tile, are
  // served by that XCD's L2.
  const int NG = A.ngroups;
  int64_t pt = blockIdx.x;
  int g = 0;
  if (NG > 1) {
    const int64_t l = blockIdx.x >> 3;
    pt = (l / NG) * 8 + (blockIdx.x & 7);
    g = (int)(l % NG);
    if (pt >= A.n_ptiles) return;  // whole workgroup, before any barrier
  }
  const int64_t p0 = pt * G::TP;

  const int SF = Cfg<FMT>::kFp ? (A.df + 31) / 32 : 0;
  const int SI = Cfg<FMT>::kInt ? (A.di + kRowBytes - 1) / kRowBytes : 0;
  const int S = SF + SI;
  const int nct = (A.k + G::TC - 1) / G::TC;
  const int nmy = (nct - g + NG - 1) / NG;  // centroid tiles of this workgroup (>= 1: NG <= nct)
  const int total = nmy * S;

  float al[PB];
#pragma unroll
  for (int pb = 0; pb < PB; ++pb)
    al[pb] = Cfg<FMT>::kBits ? A.alpha[min<int64_t>(p0 + wp * 32 * PB + pb * 32 + r, A.n - 1)] : 0.f;

  score_t best[PB];
  int bidx[PB];
#pragma unroll
  for (int pb = 0; pb < PB; ++pb) {
    best[pb] = Cfg<FMT>::kIntScore ? (score_t)INT_MAX : (score_t)INFINITY;
    bidx[pb] = INT_MAX;
  }

  // Pipeline: at the start of step `it` the registers hold stage it+1 (loaded
  // during step it-1).  They are written to the free LDS buffer first (every wave
  // has finished reading it: barrier of step it-1), then reloaded with stage it+2,
  // then the MFMAs of stage `it` run from the other buffer.  Each global load thus
  // has a whole step to arrive.  q counts this workgroup's centroid tiles
  // (tile g + q * NG).
  StageRegs<CB, PB> R;
  load_stage<FMT, CB, PB>(A, 0, SI, (int64_t)g * G::TC, p0, R);
  store_stage<FMT, CB, PB>(A, 0, SI, R, lds, cparl[0]);
  if (total > 1) load_stage<FMT, CB, PB>(A, S > 1 ? 1 : 0, SI, (int64_t)(g + (S > 1 ? 0 : NG)) * G::TC, p0, R);
  __syncthreads();

  auto step = [&](int q, int s, auto fp_tag, auto &acc_f, auto &acc_i) {
    constexpr bool FPS = decltype(fp_tag)::value;
    const int it = q * S + s;
    const int s_n = (s + 1 == S) ? 0 : s + 1;
    const int q_n = (s + 1 == S) ? q + 1 : q;
    const int s_nn = (s_n + 1 == S) ? 0 : s_n + 1;
    const int q_nn = (s_n + 1 == S) ? q_n + 1 : q_n;
    if (it + 1 < total) store_stage<FMT, CB, PB>(A, s_n, SI, R, lds + ((it + 1) & 1) * G::STAGE, cparl[q_n & 1]);
    if (it + 2 < total) load_stage<FMT, CB, PB>(A, s_nn, SI, (int64_t)(g + q_nn * NG) * G::TC, p0, R);
    const uint8_t *buf = lds + (it & 1) * G::STAGE;
    __builtin_amdgcn_s_setprio(1);  // favour the wave that is feeding the matrix core
    mfma_stage<CB, PB, FPS>(buf, buf + G::CBYTES, wc, wp, r, h, acc_f, acc_i);
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();
  };

  for (int q = 0; q < nmy; ++q) {
    const int64_t c0 = (int64_t)(g + q * NG) * G::TC;
    const float *cp = cparl[q & 1];
    f32x16 facc[CB][PB];
    i32x16 iacc[CB][PB];
    if constexpr (Cfg<FMT>::kInt) {
#pragma unroll
      for (int a = 0; a < CB; ++a)
#pragma unroll
        for (int b = 0; b < PB; ++b)
#pragma unroll
          for (int i = 0; i < 16; ++i) iacc[a][b][i] = 0;
      for (int s = 0; s < SI; ++s) step(q, s, std::false_type{}, facc, iacc);
    }
    if constexpr (FMT == KM_HYBRID) {
      // the tail's exact 1-bit score ts becomes the starting value -ts/2 of the
      // fp32 accumulator, so -2 acc + ||c'||^2 = ||c'||^2 - 2<x',c'> + ts
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int crow = wc * 32 * CB + cb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          const int qs = __float_as_int(cp[G::TC + crow]);
          const float u = cp[2 * G::TC + crow];
          const float s2 = cp[3 * G::TC + crow];
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) {
            const int sd = 2 * iacc[cb][pb][i] - qs;
            const float ts = fmaf(-(al[pb] * s2), (float)sd, u);
            facc[cb][pb][i] = -0.5f * ts;
          }
        }
    } else if constexpr (FMT == KM_F32) {
#pragma unroll
      for (int a = 0; a < CB; ++a)
#pragma unroll
        for (int b = 0; b < PB; ++b)
#pragma unroll
          for (int i = 0; i < 16; ++i) facc[a][b][i] = 0.f;
    }
    if constexpr (Cfg<FMT>::kFp) {
      for (int s = SI; s < S; ++s) step(q, s, std::true_type{}, facc, iacc);
    }

    // epilogue for this centroid tile: scores and running argmin, lane-local.
    // fp formats: branch-free selects; lane rows ascend with (cb, i), so the strict
    // comparison keeps the smallest index among equal scores.
    if constexpr (FMT == KM_F32 || FMT == KM_HYBRID) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const int crow0 = wc * 32 * CB + cb * 32 + 4 * h;
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const f32x4 cn4 = *reinterpret_cast<const f32x4 *>(&cp[crow0 + 8 * i4]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = 4 * i4 + e;
            const int j = (int)c0 + crow0 + 8 * i4 + e;
#pragma unroll
            for (int pb = 0; pb < PB; ++pb) {
              const float sc = fmaf(-2.0f, facc[cb][pb][i], cn4[e]);  // tail score folded in for HYBRID
              const bool take = sc < best[pb];
              best[pb] = take ? sc : best[pb];
              bidx[pb] = take ? j : bidx[pb];
            }
          }
        }
      }
      // With one stage per tile, the next step already writes the constants of tile
      // q + 2 into cparl[q & 1]: every wave must be done reading them first.
      if (S == 1) __syncthreads();
      continue;
    }
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int crow = wc * 32 * CB + cb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
        const int64_t j = c0 + crow;
        const bool live = j < A.k;
        const float cn = cp[crow];
        const int qs = __float_as_int(cp[G::TC + crow]);
        const float u = cp[2 * G::TC + crow];
        const float s2 = cp[3 * G::TC + crow];
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          score_t sc;
          if constexpr (FMT == KM_F32) {
            sc = fmaf(-2.0f, facc[cb][pb][i], cn);
          } else if constexpr (FMT == KM_SQ8) {
            sc = qs - 2 * iacc[cb][pb][i];
          } else if constexpr (FMT == KM_SIGN1) {
            const int sd = 2 * iacc[cb][pb][i] - qs;
            const float v = al[pb] * s2;
            sc = fmaf(-v, (float)sd, u);
          } else {
            sc = fmaf(-2.0f, facc[cb][pb][i], cn);  // tail score already folded in
          }
          if (live && sc < best[pb]) {
            best[pb] = sc;
            bidx[pb] = (int)j;
          }
        }
      }
    }
  }

  // merge the two lane halves (rows 4h..), then the two centroid waves
#pragma unroll
  for (int pb = 0; pb < PB; ++pb) {
    score_t os = __shfl_xor(best[pb], 32);
    int oi = __shfl_xor(bidx[pb], 32);
    if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
      best[pb] = os;
      bidx[pb] = oi;
    }
  }
  score_t *ms = reinterpret_cast<score_t *>(lds);
  int *mi = reinterpret_cast<int *>(lds + G::TP * sizeof(score_t));
  if (wc == 1 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      ms[wp * 32 * PB + pb * 32 + r] = best[pb];
      mi[wp * 32 * PB + pb * 32 + r] = bidx[pb];
    }
  }
  __syncthreads();
  if (wc == 0 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int pc = wp * 32 * PB + pb * 32 + r;
      const score_t os = ms[pc];
      const int oi = mi[pc];
      if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
        best[pb] = os;
        bidx[pb] = oi;
      }
      const int64_t p = p0 + pc;
      if (p < A.n) {
        if (A.keys) {
          if constexpr (!Cfg<FMT>::kIntScore) atomicMin(A.keys + p, score_key(best[pb], bidx[pb]));
        } else {
          A.assign[p] = bidx[pb] + A.aoff;
          if (A.score) A.score[p] = (float)best[pb];
        }
      }
    }
  }
}

__global__ __launch_bounds__(256) void keys_init_kernel(unsigned long long *keys, int64_t n) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p < n) keys[p] = ~0ull;
}

template <bool INT>
__global__ __launch_bounds__(256) void keys_unpack_kernel(const unsigned long long *keys, int64_t n, int32_t *assign,
                                                          float *score, int aoff) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= n) return;
  const unsigned long long key = keys[p];
  assign[p] = (int32_t)(uint32_t)key + aoff;
  if (score) score[p] = INT ? (float)(int)((uint32_t)(key >> 32) ^ 0x80000000u) : key_score(key);
}

// ---- int8 assignment with 256 x 256 workgroup tiles ---------------------------
// Register-staged stages; the direct-copy kernels below replace it except for SQ8
// beyond 8192 dimensions and 1-bit points beyond 1280.  An int8 MFMA is 16-32x denser than
// the fp32 one, so operand bandwidth decides the tiling: the workgroup owns 256
// centroids x 256 points per stage (a quarter of the L2 bytes per MFMA of a 128
// tile) and each of its 8 waves 128 centroids x 64 points (4 x 2 blocks of
// 32 x 32, 0.75 LDS reads of 1 KB per MFMA).  128 accumulators per wave leave
// room for two waves per SIMD, so one wave's stage boundary (LDS writes, barrier)
// overlaps the other's matrix work.
constexpr int kT8 = 256;
constexpr int k8Threads = 512;                 // 8 waves: 2 centroid halves x 4 point quarters
constexpr int k8PB = 2;                        // 32-point blocks per wave
constexpr int kTileBytes8 = kT8 * kLdsStride;  // 36864
constexpr int kStageBytes8 = 2 * kTileBytes8;  // 73728

struct Stage8 {
  uint4 c[4];
  uint4 p[4];
  float cpar[4];
};

template <int FMT>
__device__ __forceinline__ void load_stage8(const AssignArgs &A, int s, int64_t c0, int64_t p0, Stage8 &R) {
  const int t = threadIdx.x;
  const int b0 = kRowBytes * s;
  // uniform tile bases + 32-bit per-thread offsets (rows clamped into the data)
  const int8_t *cbase = A.ci8 + c0 * A.cild;
  const int crmax = (int)min<int64_t>(A.k - 1 - c0, kT8 - 1);
  const uint8_t *pbase8 = A.pi8 + p0 * A.pild;
  const uint32_t *pbaseb = A.pbits + p0 * A.pbw + A.pbw0;
  const int prmax = (int)min<int64_t>(A.n - 1 - p0, kT8 - 1);
#pragma unroll
  for (int i = 0; i < 4; ++i) {  // 256 rows x 8 chunks of 16 bytes over 512 threads
    const int cidx = t + k8Threads * i;
    const int row = cidx >> 3, col = cidx & 7;
    const int b = b0 + 16 * col;
    const int bc = b < A.di ? b : 0;
    R.c[i] = *reinterpret_cast<const uint4 *>(cbase + (uint32_t)(min(row, crmax) * (int)A.cild + bc));
    if (FMT == KM_SQ8)
      R.p[i] = *reinterpret_cast<const uint4 *>(pbase8 + (uint32_t)(min(row, prmax) * (int)A.pild + bc));
  }
  if (FMT == KM_SIGN1 || FMT == KM_RABITQ) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {  // 256 rows x 4 words
      const int w = t + k8Threads * i;
      const int row = w >> 2, wi = w & 3;
      const int word = 4 * s + wi;
      R.p[i].x = pbaseb[(uint32_t)(min(row, prmax) * (int)A.pbw + (32 * word < A.di ? word : 0))];
    }
  }
  if (s == 0) {  // per-centroid constants: threads t < kT8 (the others load a valid duplicate)
    const int64_t j = min<int64_t>(c0 + (t & (kT8 - 1)), A.k - 1);
    R.cpar[1] = __int_as_float(A.cp.qsum[j]);
    if (FMT == KM_SIGN1 || FMT == KM_RABITQ) {
      R.cpar[2] = A.cp.u[j];
      R.cpar[3] = A.cp.sig2[j];
    }
    if (FMT == KM_RABITQ) R.cpar[0] = A.cp.cn[j];
  }
}

template <int FMT>
__device__ __forceinline__ void store_stage8(const AssignArgs &A, int s, const Stage8 &R, uint8_t *buf, float *cpar) {
  const int t = threadIdx.x;
  uint8_t *ct = buf;
  uint8_t *pt = buf + kTileBytes8;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int cidx = t + k8Threads * i;
    const int row = cidx >> 3, col = cidx & 7;
    const bool ok = kRowBytes * s + 16 * col < A.di;
    uint4 cv = R.c[i];
    if (FMT == KM_SQ8) cv = flip4(cv);
    *reinterpret_cast<uint4 *>(ct + row * kLdsStride + 16 * col) = mask4(cv, ok);
    if (FMT == KM_SQ8)
      *reinterpret_cast<uint4 *>(pt + row * kLdsStride + 16 * col) = mask4(flip4(R.p[i]), ok);
  }
  if (FMT == KM_SIGN1 || FMT == KM_RABITQ) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int w = t + k8Threads * i;
      const int row = w >> 2, wi = w & 3;
      const uint32_t bits = (32 * (4 * s + wi) < A.di) ? R.p[i].x : 0u;
      *reinterpret_cast<uint4 *>(pt + row * kLdsStride + 32 * wi) =
          make_uint4(spread4(bits & 15u), spread4((bits >> 4) & 15u), spread4((bits >> 8) & 15u),
                     spread4((bits >> 12) & 15u));
      *reinterpret_cast<uint4 *>(pt + row * kLdsStride + 32 * wi + 16) =
          make_uint4(spread4((bits >> 16) & 15u), spread4((bits >> 20) & 15u), spread4((bits >> 24) & 15u),
                     spread4(bits >> 28));
    }
  }
  if (s == 0 && t < kT8) {
#pragma unroll
    for (int q = (FMT == KM_RABITQ ? 0 : 1); q < 4; ++q) cpar[q * kT8 + t] = R.cpar[q];
  }
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// 16 bytes per lane are one operand of either matrix instruction: 16 int8 codes of
// v_mfma_i32_32x32x32_i8 or 8 bfloat16 values of v_mfma_f32_32x32x16_bf16.
template <bool BF>
using Acc8 = typename std::conditional<BF, f32x16, i32x16>::type;

__device__ __forceinline__ void mfma_stage8(const uint8_t *cbuf, const uint8_t *pbuf, int wc, int wp, int r, int h,
                                            i32x16 (&acc)[4][k8PB]) {
  uint4 av[2][4], bv[2][k8PB];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
    av[0][cb] = *reinterpret_cast<const uint4 *>(cbuf + (wc * 128 + cb * 32 + r) * kLdsStride + 16 * h);
#pragma unroll
  for (int pb = 0; pb < k8PB; ++pb)
    bv[0][pb] = *reinterpret_cast<const uint4 *>(pbuf + (wp * 32 * k8PB + pb * 32 + r) * kLdsStride + 16 * h);
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int cur = g & 1, nxt = cur ^ 1;
    if (g + 1 < 4) {
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        av[nxt][cb] = *reinterpret_cast<const uint4 *>(cbuf + (wc * 128 + cb * 32 + r) * kLdsStride + 32 * (g + 1) +
                                                       16 * h);
#pragma unroll
      for (int pb = 0; pb < k8PB; ++pb)
        bv[nxt][pb] = *reinterpret_cast<const uint4 *>(pbuf + (wp * 32 * k8PB + pb * 32 + r) * kLdsStride +
                                                       32 * (g + 1) + 16 * h);
    }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int pb = 0; pb < k8PB; ++pb) {
        const i32x4 a4 = {(int)av[cur][cb].x, (int)av[cur][cb].y, (int)av[cur][cb].z, (int)av[cur][cb].w};
        const i32x4 b4 = {(int)bv[cur][pb].x, (int)bv[cur][pb].y, (int)bv[cur][pb].z, (int)bv[cur][pb].w};
        acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a4, b4, acc[cb][pb], 0, 0, 0);
      }
  }
}

template <int FMT>
__global__ __launch_bounds__(k8Threads, 1) void assign_i8_kernel(AssignArgs A) {
  static_assert(FMT == KM_SQ8 || FMT == KM_SIGN1 || FMT == KM_RABITQ, "int8 formats beyond the direct-copy kernels");
  __shared__ __align__(16) uint8_t lds[2 * kStageBytes8];
  __shared__ __align__(16) float cparl[2][4 * kT8];
  typedef typename std::conditional<FMT == KM_SQ8, int, float>::type score_t;

  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int wc = wave & 1, wp = wave >> 1;
  const int64_t p0 = (int64_t)blockIdx.x * kT8;

  const int S = (A.di + kRowBytes - 1) / kRowBytes;
  const int nct = (A.k + kT8 - 1) / kT8;
  const int total = nct * S;

  float al[k8PB] = {};
  int pop[k8PB] = {};
  if (FMT == KM_SIGN1 || FMT == KM_RABITQ) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb) {
      const int64_t p = min<int64_t>(p0 + wp * 32 * k8PB + pb * 32 + r, A.n - 1);
      al[pb] = A.alpha[p];
      if (FMT == KM_RABITQ) {  // the point's number of set bits
        const uint32_t *row = A.pbits + p * A.pbw + A.pbw0;
        for (int w = 0; w < A.di / 32; ++w) pop[pb] += __popc(row[w]);
      }
    }
  }
  i32x16 acc[4][k8PB];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < k8PB; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0;

  score_t best[k8PB];
  int bidx[k8PB];
#pragma unroll
  for (int pb = 0; pb < k8PB; ++pb) {
    best[pb] = FMT == KM_SQ8 ? (score_t)INT_MAX : (score_t)INFINITY;
    bidx[pb] = INT_MAX;
  }

  Stage8 R;
  load_stage8<FMT>(A, 0, 0, p0, R);
  store_stage8<FMT>(A, 0, R, lds, cparl[0]);
  __syncthreads();

  for (int ct = 0; ct < nct; ++ct) {
    for (int s = 0; s < S; ++s) {
      const int it = ct * S + s;
      const bool has_next = it + 1 < total;
      const int s_n = (s + 1 == S) ? 0 : s + 1;
      const int ct_n = (s + 1 == S) ? ct + 1 : ct;
      if (has_next) load_stage8<FMT>(A, s_n, (int64_t)ct_n * kT8, p0, R);
      const uint8_t *buf = lds + (it & 1) * kStageBytes8;
      mfma_stage8(buf, buf + kTileBytes8, wc, wp, r, h, acc);
      if (has_next) store_stage8<FMT>(A, s_n, R, lds + ((it + 1) & 1) * kStageBytes8, cparl[ct_n & 1]);
      __syncthreads();
    }
    // epilogue: one 32-row block at a time (a scheduling barrier keeps the
    // compiler from pulling all 256 accumulators into VGPRs at once); per-row
    // constants read 4 at a time; branch-free selects.  Rows ascend with (cb, i)
    // in a lane, so the strict comparison keeps the smallest index among ties.
    const int c0 = ct * kT8;
    const float *cp = cparl[ct & 1];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int crow0 = wc * 128 + cb * 32 + 4 * h;
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int cr = crow0 + 8 * i4;
        const f32x4 q4 = *reinterpret_cast<const f32x4 *>(&cp[kT8 + cr]);
        f32x4 u4 = {0.f, 0.f, 0.f, 0.f}, s4 = {0.f, 0.f, 0.f, 0.f}, b4 = {0.f, 0.f, 0.f, 0.f};
        if constexpr (FMT == KM_SIGN1 || FMT == KM_RABITQ) {
          u4 = *reinterpret_cast<const f32x4 *>(&cp[2 * kT8 + cr]);
          s4 = *reinterpret_cast<const f32x4 *>(&cp[3 * kT8 + cr]);
        }
        if constexpr (FMT == KM_RABITQ) b4 = *reinterpret_cast<const f32x4 *>(&cp[cr]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * i4 + e;
          const int j = c0 + cr + e;
          const bool live = j < A.k;
#pragma unroll
          for (int pb = 0; pb < k8PB; ++pb) {
            score_t sc;
            if constexpr (FMT == KM_SQ8) {
              sc = -__float_as_int(q4[e]) - 2 * acc[cb][pb][i];  // the constant is -||c~||^2
            } else if constexpr (FMT == KM_RABITQ) {  // Eq. 4-5, fp32 in the oracle's order
              const int sd = 2 * acc[cb][pb][i] - __float_as_int(q4[e]);
              const float inner = fmaf(s4[e], (float)sd, b4[e] * (float)(2 * pop[pb] - A.di));
              sc = fmaf(-(2.0f * al[pb]), inner, u4[e]);
            } else {
              const int sd = 2 * acc[cb][pb][i] - __float_as_int(q4[e]);
              const float v = al[pb] * s4[e];
              sc = fmaf(-v, (float)sd, u4[e]);
            }
            const bool take = live && sc < best[pb];
            best[pb] = take ? sc : best[pb];
            bidx[pb] = take ? j : bidx[pb];
          }
        }
      }
#pragma unroll
      for (int pb = 0; pb < k8PB; ++pb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[cb][pb][i] = 0;
      __builtin_amdgcn_sched_barrier(0);
    }
    // the next tile's steps write tile ct + 2's constants into cparl[ct & 1]; with
    // one stage per tile no other barrier would order that after these reads.
    // (Unconditional: a branch here splits the loop and costs register spills.)
    __syncthreads();
  }

#pragma unroll
  for (int pb = 0; pb < k8PB; ++pb) {
    score_t os = __shfl_xor(best[pb], 32);
    int oi = __shfl_xor(bidx[pb], 32);
    if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
      best[pb] = os;
      bidx[pb] = oi;
    }
  }
  score_t *ms = reinterpret_cast<score_t *>(lds);
  int *mi = reinterpret_cast<int *>(lds + kT8 * sizeof(score_t));
  if (wc == 1 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb) {
      ms[wp * 32 * k8PB + pb * 32 + r] = best[pb];
      mi[wp * 32 * k8PB + pb * 32 + r] = bidx[pb];
    }
  }
  __syncthreads();
  if (wc == 0 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb) {
      const int pc = wp * 32 * k8PB + pb * 32 + r;
      const score_t os = ms[pc];
      const int oi = mi[pc];
      if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
        best[pb] = os;
        bidx[pb] = oi;
      }
      const int64_t p = p0 + pc;
      if (p < A.n) {
        A.assign[p] = bidx[pb] + A.aoff;
        if (A.score) A.score[p] = (float)best[pb];
      }
    }
  }
}

// ---- 1-bit assignment with the points' bits resident in LDS ----------------------
// A workgroup of NW waves owns 64 NW points.  Their code words are loaded once and
// kept in LDS transposed, word-major ([word][point]), so the 32 lanes of a wave that
// read the same word of 32 consecutive points hit 32 consecutive banks.  At load time
// the bits of each word are regrouped: bit 16h + 4q + j (dimension 4q + j of half h,
// i.e. byte j of operand register q for the lanes of half h) moves to bit 8j + 4h + q.
// Widening a half-word to 16 bytes then costs one shift and one mask per register
// instead of an extract, a multiply and a mask.  The centroids' int8 residual codes
// stream through LDS in stages of 128 centroids x 128 bytes, copied by direct
// global-to-LDS loads (no register staging): each load instruction of a wave fills
// 64 consecutive 16-byte slots, and the lane that fills slot p of row R fetches
// chunk p ^ ((R >> 1) & 7) of that row, so chunk c sits in slot c ^ ((R >> 1) & 7):
// the 16 lanes that an LDS cycle serves read 16 rows, and each half of them (even and
// odd rows, 64 banks apart by the 128-byte row) hits 8 different slots, so an MFMA
// operand read has no bank conflicts.  Every wave multiplies its
// 64 points by all 128 centroids of the tile (4 x 2 blocks of 32 x 32 x 32), so no
// cross-wave merge is needed.
//
// Two shapes: 4 waves and 256 points with up to 1024 resident dimensions (69 KB of
// LDS, two workgroups per CU, so one workgroup's epilogue runs under the other's
// MFMAs), and 8 waves and 512 points with up to 1280 dimensions (one per CU).
constexpr int kBTC = 128;  // centroids per tile
constexpr int kBStageBytes = kBTC * kRowBytes;
constexpr int kBWordsSmall = 32;  // 4-wave shape: d - d0 <= 1024
constexpr int kBWordsLarge = 40;  // 8-wave shape: d - d0 <= 1280

__device__ __forceinline__ uint32_t regroup_bits(uint32_t w) {
  uint32_t o = 0;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int q = 0; q < 4; ++q) o |= spread4((w >> (16 * h + 4 * q)) & 15u) << (4 * h + q);
  return o;
}

// x: a regrouped word shifted right by 4h.  Register q takes bit 8j + q of x as
// byte j with the value 0 or 2, so the products sum to 2D; seeded with -T the
// accumulator ends at 2D - T.
__device__ __forceinline__ i32x4 widen_regrouped2(uint32_t x) {
  constexpr uint32_t M2 = 0x02020202u;
  return i32x4{(int)((x << 1) & M2), (int)(x & M2), (int)((x >> 1) & M2), (int)((x >> 2) & M2)};
}

// Direct copy of 16 bytes per lane from global memory into LDS: the wave's 64 lanes
// fill 1 KB at LDS byte address lds (wave-uniform) in lane order.  Written as
// inline assembly so that the compiler, which cannot tell the destination from the
// LDS the MFMA loop reads, does not wait for the copy before every LDS read; the
// caller waits (vmcnt) before the barrier that publishes the data.  M0 is set and
// used inside the statement.
typedef __attribute__((address_space(3))) uint8_t lds_u8;

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_copy16(const void *src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory", "m0");
}
// the same from a wave-uniform base plus a 32-bit per-lane byte offset
__device__ __forceinline__ void lds_copy16(const void *base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// FMT: KM_SIGN1 (symmetric int8 centroid codes) or KM_RABITQ (SQ4 centroid codes
// with bias; the epilogue also needs each point's number of set bits).
template <int FMT, int NW, int MAXW>
__global__ __launch_bounds__(64 * NW, 8 / NW) void assign_bits_kernel(AssignArgs A) {
  constexpr int NT = 64 * NW;         // threads
  constexpr int TP = 64 * NW;         // points per workgroup
  constexpr int CPT = kBTC * 8 / NT;  // 16-byte centroid chunks per thread and stage
  static_assert(CPT * NT == kBTC * 8 && NT >= kBTC, "stage split");
  static_assert(MAXW % 4 == 0, "whole stages of resident words");
  __shared__ uint32_t bitsT[MAXW * TP];
  // two stage buffers as separate arrays: stage it reads one while the copies of
  // stage it + 1 fill the other, and each access names its array statically
  __shared__ __align__(16) uint8_t cst0[kBStageBytes];
  __shared__ __align__(16) uint8_t cst1[kBStageBytes];
  __shared__ __align__(16) float cparl[2][4 * kBTC];
  __shared__ int popl[TP];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int64_t p0 = (int64_t)blockIdx.x * TP;
  const int W = A.di / 32;  // words of the 1-bit part
  const int S = (A.di + kRowBytes - 1) / kRowBytes;
  const int nct = (A.k + kBTC - 1) / kBTC;
  const int total = nct * S;
  const int prmax = (int)min<int64_t>(A.n - 1 - p0, TP - 1);

  // resident codes: thread t loads point t's words, regroups them and counts set
  // bits; words past the last one up to the stage boundary are zero, so the chunks
  // that a partial last stage copies from past the dimensions contribute nothing
  {
    const uint32_t *row = A.pbits + (p0 + min(t, prmax)) * A.pbw + A.pbw0;
    int pc = 0;
    for (int w = 0; w < W; ++w) {
      const uint32_t v = row[w];
      bitsT[w * TP + t] = regroup_bits(v);
      pc += __popc(v);
    }
    for (int w = W; w < 4 * S; ++w) bitsT[w * TP + t] = 0u;
    popl[t] = pc;
  }
  float al[2];
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) al[pb] = A.alpha[p0 + min(wave * 64 + pb * 32 + r, prmax)];

  // centroid stage loads: 128 rows x 8 chunks of 16 B straight into LDS buffer dst.
  // A chunk past the last dimension repeats chunk 0 of its row: the resident point
  // words are zero there.  The tile constants hold the negated code sum and, past
  // the last centroid, u = +inf: such a score is +inf and never wins, so the
  // epilogue needs no bounds test.  Their loads go out before the copies, so that
  // waiting for them never waits for the copies.  Within a full stage of a full
  // tile a lane's source is a fixed offset (coff) from the stage's first byte.
  uint32_t coff[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int slot = (i * NW + wave) * 64 + lane;
    const int row = slot >> 3;
    coff[i] = (uint32_t)(row * (int)A.cild + 16 * ((slot & 7) ^ ((row >> 1) & 7)));
  }
  float cpv[4] = {0.f, 0.f, 0.f, 0.f};
  auto load = [&](int ct, int s, uint8_t *dst) {
    const int c0 = ct * kBTC;
    const int crmax = min(A.k - 1 - c0, kBTC - 1);
    if (s == 0 && t < kBTC) {
      const int j = c0 + min(t, crmax);
      cpv[0] = __int_as_float(-A.cp.qsum[j]);
      cpv[1] = t <= crmax ? A.cp.u[j] : INFINITY;
      cpv[2] = A.cp.sig2[j];
      if (FMT == KM_RABITQ) cpv[3] = A.cp.cn[j];
    }
    const int8_t *cbase = A.ci8 + (int64_t)c0 * A.cild;
    if (crmax == kBTC - 1 && kRowBytes * (s + 1) <= A.di) {
#pragma unroll
      for (int i = 0; i < CPT; ++i)
        lds_copy16(cbase + kRowBytes * s, coff[i],
                   (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t *)(dst + (i * NW + wave) * 1024));
    } else {
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int slot = (i * NW + wave) * 64 + lane;
        const int row = slot >> 3;
        const int b = kRowBytes * s + 16 * ((slot & 7) ^ ((row >> 1) & 7));
        lds_copy16(cbase + (uint32_t)(min(row, crmax) * (int)A.cild + (b < A.di ? b : 0)),
                   (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t *)(dst + (i * NW + wave) * 1024));
      }
    }
  };
  // completes a load: waits for this wave's copies (the barrier that follows makes
  // the whole stage visible) and stores the tile constants
  auto store = [&](int ct, int s) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (s == 0 && t < kBTC) {
#pragma unroll
      for (int q = 0; q < 4; ++q) cparl[ct & 1][q * kBTC + t] = cpv[q];
    }
  };

  float best[2] = {INFINITY, INFINITY};
  int bidx[2] = {INT_MAX, INT_MAX};

  load(0, 0, cst0);
  store(0, 0);
  __syncthreads();
  int pop[2] = {0, 0};
  if (FMT == KM_RABITQ) {
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) pop[pb] = popl[wave * 64 + pb * 32 + r];
  }
  const uint32_t hsh = 4u * (uint32_t)h;

  i32x16 acc[4][2];
  // one stage of MFMAs; in a tile's first stage the first products take their
  // accumulator seed, -T of the row, from the tile constants instead of acc
  auto mfma_stage = [&](int ct, int s, const uint8_t *buf, auto first) {
    constexpr bool kFirst = decltype(first)::value;
    i32x16 seed[4];
    if constexpr (kFirst) {
      const float *cp = cparl[ct & 1];
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const int4 v = *reinterpret_cast<const int4 *>(cp + cb * 32 + 8 * m + 4 * h);
          seed[cb][4 * m] = v.x;
          seed[cb][4 * m + 1] = v.y;
          seed[cb][4 * m + 2] = v.z;
          seed[cb][4 * m + 3] = v.w;
        }
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int w = 4 * s + g;
      i32x4 bv[2];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) bv[pb] = widen_regrouped2(bitsT[w * TP + wave * 64 + pb * 32 + r] >> hsh);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const uint4 av =
            *reinterpret_cast<const uint4 *>(buf + (cb * 32 + r) * kRowBytes + 16 * ((2 * g + h) ^ ((r >> 1) & 7)));
        const i32x4 a4 = {(int)av.x, (int)av.y, (int)av.z, (int)av.w};
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          if (kFirst && g == 0)
            acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a4, bv[pb], seed[cb], 0, 0, 0);
          else
            acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a4, bv[pb], acc[cb][pb], 0, 0, 0);
        }
      }
    }
  };

  // epilogue: acc holds the exact integer 2D - T; fp32 score in the fixed order of
  // Eq. 4.  Rows are visited in increasing order, so a strict < keeps the smaller
  // index on a tie; the tile-local row (without the half's offset 4h) is a constant.
  auto epilogue = [&](int ct) {
    const float *cp = cparl[ct & 1];
    int loc[2] = {-1, -1};
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        // the constants of 4 consecutive rows at a time
        const int row0 = cb * 32 + 8 * i4 + 4 * h;
        const f32x4 u4 = *reinterpret_cast<const f32x4 *>(cp + kBTC + row0);
        const f32x4 s24 = *reinterpret_cast<const f32x4 *>(cp + 2 * kBTC + row0);
        f32x4 bj4 = {0.f, 0.f, 0.f, 0.f};
        if constexpr (FMT == KM_RABITQ) bj4 = *reinterpret_cast<const f32x4 *>(cp + 3 * kBTC + row0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
        const int i = 4 * i4 + e;
        const int cl = cb * 32 + 8 * i4 + e;
        const float u = u4[e];
        const float s2 = s24[e];
        const float bj = bj4[e];
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          const int sd = acc[cb][pb][i];
          float sc;
          if constexpr (FMT == KM_RABITQ) {  // Eq. 4-5: fp32 in the oracle's order
            const float inner = fmaf(s2, (float)sd, bj * (float)(2 * pop[pb] - A.di));
            sc = fmaf(-(2.0f * al[pb]), inner, u);
          } else {
            const float v = al[pb] * s2;
            sc = fmaf(-v, (float)sd, u);
          }
          if (sc < best[pb]) {
            best[pb] = sc;
            loc[pb] = cl;
          }
        }
        }
      }
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
      if (loc[pb] >= 0) bidx[pb] = ct * kBTC + loc[pb] + 4 * h;
  };

  // stage s of tile ct reads buffer cur while the copies of the next stage fill nxt
  auto step = [&](int ct, int s, bool has_next, const uint8_t *cur, uint8_t *nxt) {
    const int s_n = (s + 1 == S) ? 0 : s + 1;
    const int ct_n = (s + 1 == S) ? ct + 1 : ct;
    if (has_next) load(ct_n, s_n, nxt);
    if (s == 0)
      mfma_stage(ct, s, cur, std::true_type{});
    else
      mfma_stage(ct, s, cur, std::false_type{});
    if (has_next) store(ct_n, s_n);
    __syncthreads();
    if (s == S - 1) {
      epilogue(ct);
      // the next tile's steps write tile ct + 2's constants into cparl[ct & 1]; with
      // one stage per tile no other barrier would order that after these reads
      __syncthreads();
    }
  };
  int cct = 0, cs = 0;  // tile and stage of the step about to run
  auto advance = [&]() {
    if (++cs == S) {
      cs = 0;
      ++cct;
    }
  };
  for (int it = 0; it < total; it += 2) {
    step(cct, cs, it + 1 < total, cst0, cst1);
    advance();
    if (it + 1 < total) {
      step(cct, cs, it + 2 < total, cst1, cst0);
      advance();
    }
  }
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) {
    const float os = __shfl_xor(best[pb], 32);
    const int oi = __shfl_xor(bidx[pb], 32);
    if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
      best[pb] = os;
      bidx[pb] = oi;
    }
    const int64_t p = p0 + wave * 64 + pb * 32 + r;
    if (h == 0 && p < A.n) {
      A.assign[p] = bidx[pb] + A.aoff;
      if (A.score) A.score[p] = best[pb];
    }
  }
}

// ---- SQ8 / bf16 / LVQ4 assignment with direct global-to-LDS stages ------------
// The same 256 x 256 workgroup tile and wave split as above (8 waves: 2 centroid
// halves x 4 point quarters, 128 centroids x 64 points each; bf16 uses 16 waves, NWC
// below), with the operand
// traffic moved off the vector units: every stage (256 centroid rows and 256 point
// rows of 128 bytes) is copied straight from global memory into LDS, 16 bytes per
// lane, with the XOR slot layout of the 1-bit kernel (chunk c of row R in slot
// c ^ ((R >> 1) & 7)), so nothing passes through registers and the MFMA operand
// reads are free of bank conflicts.  SQ8 centroid codes arrive already recentred to int8
// (code - 128, written by the centroid preparation); the point codes are recentred
// in registers after the LDS read (one XOR per register).  Chunks past the last
// dimension are zero-filled by ordinary LDS stores from the lanes that skip their
// copy.  Rows past the last centroid repeat the last centroid, codes and constant,
// so their scores tie with it exactly and lose on the index: the epilogue is
// branch-free and needs no bounds test.
//
// LVQ4 points stay packed (4 bits per dimension) through the copies, so a stage
// moves 64 bytes per point row; the MFMA operand is unpacked after the LDS read
// (low nibbles, then high nibbles of each word: two masks and a shift), and the
// centroid preparation writes the int8 centroid codes in that same order. The
// epilogue evaluates Eq. 2 per pair from the point's (s, b, A) and the centroid's
// (b, S, N, s).
//
// With ngroups > 1 the workgroup (pt, g) sweeps centroid tiles g, g + ngroups, ...
// of point tile pt; the ngroups workgroups of a point tile are consecutive among
// the workgroups of one XCD, so their concurrent reads of the point rows share that
// XCD's L2, and they merge through 64-bit (score, index) keys.
constexpr int kQT = 256;                            // points per workgroup (and centroids per tile, CB = 4)
constexpr int kQThreads = 512;                      // 8 waves
constexpr int kQWideThreads = 1024;                 // 16 waves (bf16, 256-centroid tiles)
constexpr int kQMaxDimSQ8 = 8192;                   // |2<x~,c~> - ||c~||^2| < 2^31
constexpr int kQPackMaxDim = 1024;                  // SQ8 packed selection keys (below)

// CB: 32 x 32 centroid blocks per wave, 4 (256-centroid tiles) or 2 (128-centroid
// tiles, for k <= 128, where a 256-centroid tile would be mostly padding)
//
// NWC: waves along the centroids.  2 is the shape above; 4 (bf16 only, with CB = 2)
// makes 16 waves of 64 centroids x 64 points on the same 256 x 256 tile.  A wave's
// direct copies complete one after another, so a stage's 64 copy instructions
// spread over 16 waves (4 each) take half the time they take over 8; the LDS
// operand reads grow by a third (each wave reads 4 operand blocks per step for 4
// MFMAs instead of 6 for 8).  Its 128-register budget leaves no room to keep the
// copy offsets, which are recomputed at each copy.  SQ8 spills at that budget and
// keeps the 8-wave shape.
//
// PK (SQ8 with d <= kQPackMaxDim): the key 2<x~,c~> - ||c~||^2 of every code pair
// lies in [-48896 d, 16384 d] (codes in [-128, 127]: the key is ||x~||^2 - ||x~ - c~||^2),
// so key + 16256 d lies within +-32640 d < 2^25 and leaves the low 6 bits of an int32
// for a row id that is unique among the 64 rows one lane scans per tile.  The
// centroid constant of a row becomes E = ((-||c~||^2 + 16256 d) << 6) + 63 - id, and
// the packed key of a pair, ((2<x~,c~> - ||c~||^2 + 16256 d) << 6) + 63 - id =
// (acc << 7) + E (modulo 2^32, exact since the result is in range), orders pairs by
// key and then by the smaller id: one shift-add and one max per pair select the
// tile's winner instead of a compare and two selects.
template <int FMT, bool SEG = false, int CB = 4, bool PK = false, int NWC = 2>
__global__ __launch_bounds__(256 * NWC, 1) void assign_q8_kernel(AssignArgs A0) {
  constexpr bool BF = FMT == KM_BF16;
  constexpr bool LV = FMT == KM_LVQ4;
  static_assert(CB == 2 || CB == 4, "64 or 128 centroids per wave");
  static_assert(NWC == 2 || NWC == 4, "2 or 4 waves along the centroids");
  constexpr int NW = 4 * NWC;                       // waves: NWC centroid groups x 4 point quarters
  constexpr int TC = 32 * CB * NWC;                 // centroids per tile
  constexpr int TP = kQT;                           // points per workgroup
  constexpr int PRB = LV ? kRowBytes / 2 : kRowBytes;  // point bytes per row and stage (LVQ4: packed)
  constexpr int NCC = TC / (8 * NW);                // centroid copies per thread and stage
  constexpr int NCOPY = NCC + TP * PRB / (1024 * NW);  // all copies per thread and stage
  constexpr int NCONST = LV ? 4 : 1;                // per-centroid constants of the epilogue
  static_assert(NWC == 2 || (BF && CB == 2), "16 waves: bf16 with 64 centroids per wave (SQ8 spills there)");
  static_assert(!LV || (!SEG && NWC == 2), "LVQ4: unsegmented, 8 waves");
  constexpr int STAGE = TC * kRowBytes + TP * PRB;  // centroid rows, then point rows
  // a segmented launch narrows the arguments to this workgroup's segment
  AssignArgs A = A0;
  int64_t seg_p0 = 0;  // first row of this workgroup's point tile (segmented launch)
  if constexpr (SEG) {
    const int2 ts = A0.tiles[blockIdx.x];
    const int4 sg = A0.segs[ts.x];
    seg_p0 = (int64_t)sg.x + (int64_t)ts.y * TP;
    A.n = (int64_t)sg.x + sg.y;
    A.k = sg.w;
    A.ci8 = A0.ci8 + (int64_t)sg.z * A0.cild;
    A.cp.cn = A0.cp.cn + sg.z;
    A.cp.qsum = A0.cp.qsum + sg.z;
    A.aoff = A0.aoff + sg.z;
    A.ngroups = 1;
  }
  static_assert(FMT == KM_SQ8 || FMT == KM_BF16 || LV, "SQ8, bf16 or LVQ4 points");
  static_assert(!PK || FMT == KM_SQ8, "packed keys are integer keys");
  // SQ8 maximises the key 2D - ||c~||^2 (= -score, exact in int32); bf16 and LVQ4
  // minimise their fp32 scores
  typedef typename std::conditional<BF || LV, float, int>::type key_t;
  // 128-centroid tiles of the 8-wave shape (k <= 128, and the hierarchical phases'
  // small centroid sets): a stage carries only ~1000 MFMA cycles per SIMD (SQ8)
  // against a copy latency of a microsecond or more, so three stage buffers (3 x 48
  // KB; LVQ4 3 x 32 KB) keep the copies two stages ahead; SQ8 17 % faster on a
  // 2M x 1024, k = 112 pass
  constexpr bool TRI = CB == 2 && NWC == 2;
  __shared__ __align__(16) uint8_t qst0[STAGE];
  __shared__ __align__(16) uint8_t qst1[STAGE];
  __shared__ __align__(16) uint8_t qst2[TRI ? STAGE : 16];
  __shared__ __align__(16) float cparl[2][NCONST * TC];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int wc = wave % NWC, wp = wave / NWC;
  const int NG = A.ngroups;
  int64_t pt = blockIdx.x;
  int g = 0;
  if (NG > 1) {
    const int64_t l = blockIdx.x >> 3;
    pt = (l / NG) * 8 + (blockIdx.x & 7);
    g = (int)(l % NG);
    if (pt >= A.n_ptiles) return;  // whole workgroup, before any barrier
  }
  const int64_t p0 = SEG ? seg_p0 : pt * TP;
  const int S = (A.di + kRowBytes - 1) / kRowBytes;
  const int nct = (A.k + TC - 1) / TC;
  const int nmy = (nct - g + NG - 1) / NG;  // centroid tiles of this workgroup (>= 1: NG <= nct)
  const int total = nmy * S;
  const int prmax = (int)min<int64_t>(A.n - 1 - p0, TP - 1);
  const uint8_t *pbase = A.pi8 + p0 * A.pild;
  const int pk_off = PK ? 16256 * A.di : 0;  // recentres the packed keys

  // copy i (0 .. NCOPY - 1) of a wave fills slots (NW i + wave) 64 .. + 63 of the
  // stage: rows 0 .. TC - 1 are centroids, the next TP rows points.  A lane's source is the stage's first
  // byte plus a 32-bit offset: point rows are clamped into the data once, centroid
  // rows only in a last, partial centroid tile.  In a partial last stage the lanes
  // whose chunk lies past the dimensions store zeros instead of copying.
  //
  // LVQ4 point rows hold a stage's 128 dimensions in 64 packed bytes (4 chunks of
  // 32 dimensions): chunk c of point row R sits in slot c ^ ((R >> 2) & 3), which
  // spreads the 16 rows that 16 lanes read over 16 distinct 16-byte bank groups if
  // an LDS cycle serves 16 lanes as it does for the 128-byte rows; the counters
  // still show two passes per read (a 2-way conflict on these reads only, worth
  // about 1 % of the kernel; other placements tried cost more in registers).
  auto point_slot = [&](int i, int &row, int &chunk) {  // LVQ4 point copies (i >= NCC)
    const int slot = ((i - NCC) * NW + wave) * 64 + lane;
    row = slot >> 2;
    chunk = (slot & 3) ^ ((row >> 2) & 3);
  };
  auto source_offset = [&](int i) {
    if (LV && i >= NCC) {
      int row, chunk;
      point_slot(i, row, chunk);
      return (uint32_t)(min(row, prmax) * (int)A.pild + 16 * chunk);
    }
    const int slot = (i * NW + wave) * 64 + lane;
    const int row = slot >> 3;
    const int chunk = (slot & 7) ^ ((row >> 1) & 7);
    return i < NCC ? (uint32_t)(row * (int)A.cild + 16 * chunk)
                   : (uint32_t)(min(row - TC, prmax) * (int)A.pild + 16 * chunk);
  };
  // 16 waves (and LVQ4, whose epilogue needs the point and centroid constants) have
  // no registers to spare: their offsets are recomputed at each copy (a few vector
  // instructions) and laundered so that the compiler keeps them there
  constexpr bool kKeepOffsets = NWC == 2 && !LV;
  uint32_t soff[kKeepOffsets ? NCOPY : 1];
  if constexpr (kKeepOffsets) {
#pragma unroll
    for (int i = 0; i < NCOPY; ++i) soff[i] = source_offset(i);
  }
  auto offset_of = [&](int i) {
    if constexpr (kKeepOffsets) {
      return soff[i];
    } else {
      uint32_t o = source_offset(i);
      asm volatile("" : "+v"(o));
      return o;
    }
  };
  float cpv = 0.f;
  float cpx[3] = {0.f, 0.f, 0.f};  // LVQ4: the other three constants of row t
  // the next stage's tile constant for row t (loaded with its tile's first stage)
  auto load_constant = [&](int ct) {
    const int c0 = (g + ct * NG) * TC;
    const int crmax = min(A.k - 1 - c0, TC - 1);
    if (t < TC) {
      const int j = c0 + min(t, crmax);
      cpv = BF ? A.cp.cn[j] : __int_as_float(A.cp.qsum[j]);  // SQ8: -||c~||^2
      if constexpr (LV) {  // b_y, S_y (the code sum as the float the epilogue multiplies), N_y, s_y
        cpv = A.cp.cn[j];
        cpx[0] = (float)A.cp.qsum[j];
        cpx[1] = A.cp.u[j];
        cpx[2] = A.cp.sig2[j];
      }
      if constexpr (PK) {
        const int rr = t & (32 * CB - 1);  // row within its wave's centroid group
        const int id = (rr >> 5) * 16 + ((rr >> 3) & 3) * 4 + (rr & 3);
        cpv = __int_as_float((int)(((uint32_t)(A.cp.qsum[j] + pk_off) << 6) + (uint32_t)(63 - id)));
      }
    }
  };
  // copy i of stage s of tile ct into buffer dst
  auto load_one = [&](int ct, int s, uint8_t *dst, int i) {
    const int c0 = (g + ct * NG) * TC;
    const int crmax = min(A.k - 1 - c0, TC - 1);
    const int8_t *cbase = A.ci8 + (int64_t)c0 * A.cild + kRowBytes * s;
    const uint8_t *psrc = pbase + PRB * s;
    const bool full_stage = kRowBytes * (s + 1) <= A.di;
    const int slot = (i * NW + wave) * 64 + lane;
    int row = slot >> 3;
    int chunk = (slot & 7) ^ ((row >> 1) & 7);
    // the chunk's first dimension (LVQ4 point chunks hold 32 dimensions)
    int dim0 = kRowBytes * s + 16 * chunk;
    if (LV && i >= NCC) {
      point_slot(i, row, chunk);
      dim0 = kRowBytes * s + 32 * chunk;
    }
    uint32_t off = offset_of(i);
    if (i < NCC && crmax < TC - 1) off = (uint32_t)(min(row, crmax) * (int)A.cild + 16 * chunk);
    const void *base = i < NCC ? (const void *)cbase : (const void *)psrc;
    lds_u8 *wdst = (lds_u8 *)dst + (i * NW + wave) * 1024;
    const uint32_t lds = (uint32_t)(size_t)wdst;
    if (full_stage) {
      lds_copy16(base, off, lds);
    } else if (dim0 < A.di) {
      lds_copy16(base, off, lds);
    } else {
      __attribute__((address_space(3))) uint32_t *z = (__attribute__((address_space(3))) uint32_t *)(wdst + 16 * lane);
      z[0] = z[1] = z[2] = z[3] = 0u;
    }
  };
  // The copies of one stage: its two source bases are computed once.  When the stage
  // lies wholly inside the dimensions and its centroid tile is full, every copy is
  // a plain one (a precomputed offset, no test); otherwise load_one handles the
  // clamped rows and the zero-filled chunks.  A stage's plan is (ct, s, dst, cb, pb,
  // plain), kept in scalar variables.
  auto plan_cb = [&](int ct, int s) { return A.ci8 + (int64_t)((g + ct * NG) * TC) * A.cild + kRowBytes * s; };
  auto plan_plain = [&](int ct, int s) { return kRowBytes * (s + 1) <= A.di && A.k - (g + ct * NG) * TC >= TC; };
  // copies i0 .. i1 - 1 of a stage (constants once the callers' loops are unrolled)
  auto copies = [&](int ct, int s, uint8_t *dst, const int8_t *cb, const uint8_t *pb, bool plain, int i0, int i1) {
    if (plain) {
#pragma unroll
      for (int i = i0; i < i1; ++i)
        lds_copy16(i < NCC ? (const void *)cb : (const void *)pb, offset_of(i),
                   (uint32_t)(size_t)((lds_u8 *)dst + (i * NW + wave) * 1024));
    } else {
#pragma unroll
      for (int i = i0; i < i1; ++i) load_one(ct, s, dst, i);
    }
  };
  auto load = [&](int ct, int s, uint8_t *dst) {
    if (s == 0) load_constant(ct);
    copies(ct, s, dst, plan_cb(ct, s), pbase + PRB * s, plan_plain(ct, s), 0, NCOPY);
  };
  auto store = [&](int ct, int s) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (s == 0 && t < TC) {
      cparl[ct & 1][t] = cpv;
      if constexpr (LV) {
#pragma unroll
        for (int q = 0; q < 3; ++q) cparl[ct & 1][(q + 1) * TC + t] = cpx[q];
      }
    }
  };

  // SQ8 with packed keys spreads the next stage's copies over the stage's four
  // steps (5 % faster at 1M x 768); unpacked SQ8 and LVQ4 issue them all before the
  // MFMAs (spreading them there spills: LVQ4 ran 15 % slower), and so does bf16
  // (spreading them gained nothing)
  constexpr bool SPREAD = PK;
  int sp_ct = 0, sp_s = 0;
  uint8_t *sp_dst = nullptr;
  const int8_t *sp_cb = nullptr;
  const uint8_t *sp_pb = nullptr;
  bool sp_on = false, sp_plain = false;

  Acc8<BF> acc[CB][k8PB];
  // one stage of 4 steps of 32 dimensions; a scheduling barrier per step keeps the
  // compiler from hoisting the 24 operand reads of the stage, which would spill the
  // accumulators (the other wave of the SIMD covers the read latency)
  auto mfma_stage = [&](const uint8_t *buf, auto first) {
    constexpr bool kFirst = decltype(first)::value;
    uint4 av[1][CB], bv[1][k8PB];
    // LVQ4: step g = 2j + e of a stage multiplies dimensions 16 (4j + 2h + e) .. + 15
    // in lane half h: packed point chunk 2j + h holds the point operands of steps 2j
    // and 2j + 1 (8 bytes each; each step reads it again, which keeps fewer registers
    // live than holding it across the pair), and the centroid operand is int8 chunk
    // 4j + 2h + e of its row
    auto read = [&](int g, int slot) {
      const int ca = LV ? 2 * g - (g & 1) + 2 * h : 2 * g + h;
      const int so = 16 * (ca ^ ((r >> 1) & 7));
      if constexpr (LV) {
        const int sp = 16 * (((g & ~1) + h) ^ ((r >> 2) & 3));
#pragma unroll
        for (int pb = 0; pb < k8PB; ++pb)
          bv[slot][pb] = *reinterpret_cast<const uint4 *>(buf + TC * kRowBytes + (wp * 32 * k8PB + pb * 32 + r) * PRB + sp);
      } else {
#pragma unroll
        for (int pb = 0; pb < k8PB; ++pb)
          bv[slot][pb] = *reinterpret_cast<const uint4 *>(buf + (TC + wp * 32 * k8PB + pb * 32 + r) * kRowBytes + so);
      }
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        av[slot][cb] = *reinterpret_cast<const uint4 *>(buf + (wc * 32 * CB + cb * 32 + r) * kRowBytes + so);
    };
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      constexpr int cur = 0;
      read(g, 0);
      if (SPREAD && sp_on)
        copies(sp_ct, sp_s, sp_dst, sp_cb, sp_pb, sp_plain, g * NCOPY / 4, (g + 1) * NCOPY / 4);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int pb = 0; pb < k8PB; ++pb) {
          Acc8<BF> cin;
          if (!BF && kFirst && g == 0) {
#pragma unroll
            for (int i = 0; i < 16; ++i) cin[i] = 0;
          } else {
            cin = acc[cb][pb];  // bf16: the tile's seeds -||c||^2 / 2 at its first step
          }
          if constexpr (BF) {
            acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, av[cur][cb]), __builtin_bit_cast(bf16x8, bv[cur][pb]), cin, 0, 0, 0);
          } else if constexpr (LV) {
            // 16 packed codes -> 16 bytes: the low nibbles of a word (even dimensions)
            // then its high nibbles (odd ones), the order of the centroid codes
            const uint32_t w0 = (g & 1) ? bv[cur][pb].z : bv[cur][pb].x;
            const uint32_t w1 = (g & 1) ? bv[cur][pb].w : bv[cur][pb].y;
            constexpr uint32_t M = 0x0F0F0F0Fu;
            const i32x4 a4 = {(int)av[cur][cb].x, (int)av[cur][cb].y, (int)av[cur][cb].z, (int)av[cur][cb].w};
            const i32x4 b4 = {(int)(w0 & M), (int)((w0 >> 4) & M), (int)(w1 & M), (int)((w1 >> 4) & M)};
            acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a4, b4, cin, 0, 0, 0);
          } else {
            const uint4 bq = flip4(bv[cur][pb]);  // point codes recentred to int8
            const i32x4 a4 = {(int)av[cur][cb].x, (int)av[cur][cb].y, (int)av[cur][cb].z, (int)av[cur][cb].w};
            const i32x4 b4 = {(int)bq.x, (int)bq.y, (int)bq.z, (int)bq.w};
            acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a4, b4, cin, 0, 0, 0);
          }
        }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  key_t best[k8PB];
  int bidx[k8PB];
#pragma unroll
  for (int pb = 0; pb < k8PB; ++pb) {
    best[pb] = LV ? (key_t)INFINITY : BF ? (key_t)-INFINITY : (key_t)INT_MIN;
    bidx[pb] = INT_MAX;
  }
  f32x4 vp[k8PB] = {};  // LVQ4: (s, b, A, N) of the lane's points
  if constexpr (LV) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb)
      vp[pb] = *reinterpret_cast<const f32x4 *>(A.vparams + 4 * (p0 + min(wp * 32 * k8PB + pb * 32 + r, prmax)));
  }
  // rows ascend with (cb, i) in a lane, so the strict comparison keeps the smallest
  // index among ties; the tile-local row without the wave's and half's offsets is a
  // constant here
  auto epilogue = [&](int ct) {
    const float *cp = cparl[ct & 1];
    if constexpr (LV) {  // Eq. 2 without N_x, fp32 in the oracle's order
      int loc[k8PB] = {-1, -1};
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int cr = wc * 32 * CB + cb * 32 + 8 * i4 + 4 * h;
          const f32x4 b4 = *reinterpret_cast<const f32x4 *>(cp + cr);           // b_y
          const f32x4 q4 = *reinterpret_cast<const f32x4 *>(cp + TC + cr);      // S_y
          const f32x4 u4 = *reinterpret_cast<const f32x4 *>(cp + 2 * TC + cr);  // N_y
          const f32x4 s4 = *reinterpret_cast<const f32x4 *>(cp + 3 * TC + cr);  // s_y
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = 4 * i4 + e;
            const int cl = cb * 32 + 8 * i4 + e;
#pragma unroll
            for (int pb = 0; pb < k8PB; ++pb) {
              const float sy = s4[e];
              const float tt =
                  fmaf(vp[pb][1] * sy, q4[e], fmaf(b4[e], vp[pb][2], (vp[pb][0] * sy) * (float)acc[cb][pb][i]));
              const float sc = fmaf(-2.0f, tt, u4[e]);
              if (sc < best[pb]) {
                best[pb] = sc;
                loc[pb] = cl;
              }
            }
          }
          // four rows at a time: their 16 constants, not a block's 64, in registers
          __builtin_amdgcn_sched_barrier(0);
        }
      }
#pragma unroll
      for (int pb = 0; pb < k8PB; ++pb)
        if (loc[pb] >= 0) bidx[pb] = (g + ct * NG) * TC + wc * 32 * CB + loc[pb] + 4 * h;
      return;
    }
    if constexpr (PK) {
      int tk[k8PB] = {INT_MIN, INT_MIN};  // the tile's best packed key per point block
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const f32x4 e4 = *reinterpret_cast<const f32x4 *>(cp + wc * 32 * CB + cb * 32 + 8 * i4 + 4 * h);
#pragma unroll
          for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int pb = 0; pb < k8PB; ++pb)
              tk[pb] = max(tk[pb], (int)(((uint32_t)acc[cb][pb][4 * i4 + e] << 7) + (uint32_t)__float_as_int(e4[e])));
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // tiles ascend, so the strict comparison keeps the earlier tile on ties
#pragma unroll
      for (int pb = 0; pb < k8PB; ++pb) {
        const int ks = tk[pb] >> 6;  // key + 16256 d
        if (ks > best[pb]) {
          const int id = 63 - (tk[pb] & 63);
          best[pb] = ks;
          bidx[pb] = (g + ct * NG) * TC + wc * 32 * CB + (id >> 4) * 32 + ((id >> 2) & 3) * 8 + 4 * h + (id & 3);
        }
      }
      return;
    }
    int loc[k8PB] = {-1, -1};
    // one 32-row block at a time (a scheduling barrier per block keeps the compiler
    // from loading every constant and accumulator at once); constants 4 at a time
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const f32x4 cq4 = *reinterpret_cast<const f32x4 *>(cp + wc * 32 * CB + cb * 32 + 8 * i4 + 4 * h);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * i4 + e;
          const int cl = cb * 32 + 8 * i4 + e;
#pragma unroll
          for (int pb = 0; pb < k8PB; ++pb) {
            if constexpr (BF) {
              const float sc = acc[cb][pb][i];  // <x,c> - ||c||^2 / 2 = -(||c||^2 - 2<x,c>) / 2
              if (sc > best[pb]) {
                best[pb] = sc;
                loc[pb] = cl;
              }
            } else {
              const int key = 2 * acc[cb][pb][i] + __float_as_int(cq4[e]);  // 2<x~,c~> - ||c~||^2
              if (key > best[pb]) {
                best[pb] = key;
                loc[pb] = cl;
              }
            }
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb)
      if (loc[pb] >= 0) bidx[pb] = (g + ct * NG) * TC + wc * 32 * CB + loc[pb] + 4 * h;
  };

  // bf16: the accumulators start at -||c||^2 / 2 of their row (exact halving), so
  // they end at <x,c> - ||c||^2 / 2 and the epilogue only keeps the largest
  auto seed = [&](int ct) {
    const float *cp = cparl[ct & 1];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(cp + wc * 32 * CB + cb * 32 + 8 * m + 4 * h);
#pragma unroll
        for (int pb = 0; pb < k8PB; ++pb)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[cb][pb][4 * m + e] = -0.5f * v[e];
      }
  };
  if constexpr (TRI) {
    // stage j (tile j / S, stage j % S) lives in buffer j % 3.  Step it issues the
    // copies of stage it + 2, then waits until at most NCOPY of its own copies are in
    // flight (they complete in issue order: stage it + 1's are done), and the barrier
    // publishes stage it + 1.  The buffer refilled at step it was last read at step
    // it - 1, before that step's barrier.  A tile's constants are loaded after the
    // previous tile's epilogue, draining the copies in flight once per tile.
    auto buf_of = [&](int j) { const int m = j % 3; return m == 0 ? qst0 : m == 1 ? qst1 : qst2; };
    auto issue = [&](int j) {
      const int ct_j = j / S, s_j = j % S;
      copies(ct_j, s_j, buf_of(j), plan_cb(ct_j, s_j), pbase + PRB * s_j, plan_plain(ct_j, s_j), 0, NCOPY);
    };
    auto set_constants = [&](int ct) {
      load_constant(ct);
      store(ct, 0);  // waits for every copy in flight, then writes the tile's constants
    };
    set_constants(0);
    issue(0);
    if (total > 1) {
      issue(1);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NCOPY) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    __syncthreads();
    for (int it = 0; it < total; ++it) {
      const int ct = it / S, s = it % S;
      if (it + 2 < total) issue(it + 2);
      if (BF && s == 0) seed(ct);
      if (s == 0)
        mfma_stage(buf_of(it), std::true_type{});
      else
        mfma_stage(buf_of(it), std::false_type{});
      if (it + 2 < total)
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NCOPY) : "memory");
      else
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (s == S - 1) {
        epilogue(ct);
        if (ct + 1 < nmy) set_constants(ct + 1);
        __syncthreads();
      }
    }
  } else {
  load(0, 0, qst0);
  store(0, 0);
  __syncthreads();
  // stage s of tile ct reads buffer cur while the copies of the next stage fill nxt
  auto step = [&](int ct, int s, bool has_next, const uint8_t *cur, uint8_t *nxt) {
    const int s_n = (s + 1 == S) ? 0 : s + 1;
    const int ct_n = (s + 1 == S) ? ct + 1 : ct;
    if constexpr (SPREAD) {
      sp_on = has_next;
      sp_ct = ct_n;
      sp_s = s_n;
      sp_dst = nxt;
      sp_cb = plan_cb(ct_n, s_n);
      sp_pb = pbase + PRB * s_n;
      sp_plain = plan_plain(ct_n, s_n);
      if (has_next && s_n == 0) load_constant(ct_n);
    } else {
      if (has_next) load(ct_n, s_n, nxt);
    }
    if (BF && s == 0) seed(ct);
    if (s == 0)
      mfma_stage(cur, std::true_type{});
    else
      mfma_stage(cur, std::false_type{});
    if (has_next) store(ct_n, s_n);
    __syncthreads();
    if (s == S - 1) {
      epilogue(ct);
      // the next tile's steps write tile ct + 2's constants into cparl[ct & 1]
      __syncthreads();
    }
  };
  int cct = 0, cs = 0;  // tile and stage of the step about to run
  auto advance = [&]() {
    if (++cs == S) {
      cs = 0;
      ++cct;
    }
  };
  for (int it = 0; it < total; it += 2) {
    step(cct, cs, it + 1 < total, qst0, qst1);
    advance();
    if (it + 1 < total) {
      step(cct, cs, it + 2 < total, qst1, qst0);
      advance();
    }
  }
  }
  if constexpr (PK) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb) best[pb] -= pk_off;  // back to 2<x~,c~> - ||c~||^2
  }
  if constexpr (BF) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb) best[pb] = -2.0f * best[pb];  // the score ||c||^2 - 2<x,c>
  }

  // merges in the key order (SQ8: exact integers), smaller index on ties; the
  // stored score is the key for bf16 and LVQ4 and the negated key (||c~||^2 - 2<x~,c~>)
  // for SQ8
  auto better = [](key_t o, int oi, key_t b, int bi) {
    return (BF || LV ? o < b : o > b) || (o == b && oi < bi);
  };
#pragma unroll
  for (int pb = 0; pb < k8PB; ++pb) {
    const key_t os = __shfl_xor(best[pb], 32);
    const int oi = __shfl_xor(bidx[pb], 32);
    if (better(os, oi, best[pb], bidx[pb])) {
      best[pb] = os;
      bidx[pb] = oi;
    }
  }
  // centroid groups 1 .. NWC - 1 hand their per-point winners to group 0 through LDS
  key_t *ms = reinterpret_cast<key_t *>(qst0);
  int *mi = reinterpret_cast<int *>(qst0 + (NWC - 1) * TP * sizeof(key_t));
  if (wc > 0 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb) {
      ms[(wc - 1) * TP + wp * 32 * k8PB + pb * 32 + r] = best[pb];
      mi[(wc - 1) * TP + wp * 32 * k8PB + pb * 32 + r] = bidx[pb];
    }
  }
  __syncthreads();
  if (wc == 0 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < k8PB; ++pb) {
      const int pc = wp * 32 * k8PB + pb * 32 + r;
#pragma unroll
      for (int o = 0; o < NWC - 1; ++o) {
        const key_t os = ms[o * TP + pc];
        const int oi = mi[o * TP + pc];
        if (better(os, oi, best[pb], bidx[pb])) {
          best[pb] = os;
          bidx[pb] = oi;
        }
      }
      const int64_t p = p0 + pc;
      if (p < A.n) {
        if (A.keys) {
          atomicMin(A.keys + p,
                    BF || LV ? score_key((float)best[pb], bidx[pb]) : int_score_key(-(int)best[pb], bidx[pb]));
        } else {
          A.assign[p] = bidx[pb] + A.aoff;
          if (A.score) A.score[p] = BF || LV ? (float)best[pb] : (float)(-(int)best[pb]);
        }
      }
    }
  }
}

// ---- fp32 assignment with direct global-to-LDS stages -------------------------
// The SQ8 / bf16 kernel's workgroup shape on fp32 rows: 8 waves, a 256-point tile
// against centroid tiles of TC = 64 CB (256, or 128 when k <= 128), each wave
// CB x 2 blocks of v_mfma_f32_32x32x2_f32 (128 centroids x 64 points for CB = 4),
// stages of 32 dimensions (128 bytes of every row) copied straight from global
// memory into LDS in the conflict-free slot layout (chunk c of row R in slot
// c ^ ((R >> 1) & 7)), two stage buffers, one workgroup per CU.  Per flop it moves
// half the stage bytes of a 128 x 128 tile, and moving stage bytes (by any route)
// is what costs matrix-core time here.  The copies of stage it+1 are spread over
// stage it's four 8-dimension steps, between the operand reads (double-buffered)
// and the MFMAs; full stages take a branch-free path, and in the last, partial
// stage of a tile the lanes whose chunk lies past the dimensions store zeros
// instead of copying (rows hold d % 4 == 0 floats, so a chunk is wholly in or out).
// Rows past the last centroid read the last centroid's row (clamped) with an
// infinite norm, so they never win.  Groups (ngroups > 1) and the per-point merge
// are those of the other kernels: (score, index) keys through a 64-bit atomicMin.
template <bool SEG = false, int CB = 4>
__global__ __launch_bounds__(kQThreads, 1) void assign_f32_kernel(AssignArgs A0) {
  static_assert(CB == 2 || CB == 4, "128- or 256-centroid tiles");
  constexpr int TC = 64 * CB, TP = kQT, PB = k8PB;
  constexpr int NCC = TC / 64;           // centroid copies per thread and stage
  constexpr int NCOPY = (TC + TP) / 64;  // all copies per thread and stage
  constexpr int STAGE = (TC + TP) * kRowBytes;
  AssignArgs A = A0;
  int64_t seg_p0 = 0;  // first row of this workgroup's point tile (segmented launch)
  if constexpr (SEG) {
    const int2 ts = A0.tiles[blockIdx.x];
    const int4 sg = A0.segs[ts.x];
    seg_p0 = (int64_t)sg.x + (int64_t)ts.y * TP;
    A.n = (int64_t)sg.x + sg.y;
    A.k = sg.w;
    A.cf = A0.cf + (int64_t)sg.z * A0.cfld;
    A.cp.cn = A0.cp.cn + sg.z;
    A.aoff = A0.aoff + sg.z;
    A.ngroups = 1;
  }
  __shared__ __align__(16) uint8_t fst0[STAGE];
  __shared__ __align__(16) uint8_t fst1[STAGE];
  __shared__ __align__(16) float cnl[2][TC];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int wc = wave & 1, wp = wave >> 1;
  const int NG = A.ngroups;
  int64_t pt = blockIdx.x;
  int g = 0;
  if (NG > 1) {
    const int64_t l = blockIdx.x >> 3;
    pt = (l / NG) * 8 + (blockIdx.x & 7);
    g = (int)(l % NG);
    if (pt >= A.n_ptiles) return;  // whole workgroup, before any barrier
  }
  const int64_t p0 = SEG ? seg_p0 : pt * TP;
  const int S = (A.df + 31) / 32;
  const int nct = (A.k + TC - 1) / TC;
  const int nmy = (nct - g + NG - 1) / NG;  // centroid tiles of this workgroup (>= 1: NG <= nct)
  const int total = nmy * S;
  const int prmax = (int)min<int64_t>(A.n - 1 - p0, TP - 1);
  const float *pbase = A.pf + p0 * A.pfld;

  // copy i of a wave fills slots (8 i + wave) 64 .. + 63 of the stage: rows 0 .. TC - 1
  // are centroids, the next TP rows points.  Byte offsets from the stage's first
  // float: point rows clamped into the data once, centroid rows of a full tile here
  // and of a last, partial tile at copy time.
  uint32_t soff[NCOPY];
#pragma unroll
  for (int i = 0; i < NCOPY; ++i) {
    const int slot = (i * 8 + wave) * 64 + lane;
    const int row = slot >> 3;
    const int chunk = (slot & 7) ^ ((row >> 1) & 7);
    soff[i] = i < NCC ? (uint32_t)(row * (int)A.cfld * 4 + 16 * chunk)
                      : (uint32_t)(min(row - TC, prmax) * (int)A.pfld * 4 + 16 * chunk);
  }
  // the stage being copied: tile c0, stage cs, into buffer cdst
  int c0c = 0, crmax = 0, cs = 0;
  bool cfull = true;
  uint8_t *cdst = fst0;
  float cnv = 0.f;  // the next tile's norm for row t, stored once the copies have landed
  auto begin_copies = [&](int ct, int s, uint8_t *dst) {
    c0c = (g + ct * NG) * TC;
    crmax = min(A.k - 1 - c0c, TC - 1);
    cs = s;
    cdst = dst;
    cfull = 32 * (s + 1) <= A.df;
    if (s == 0 && t < TC) cnv = t <= crmax ? A.cp.cn[c0c + t] : INFINITY;
  };
  auto copy = [&](int i) {
    const int slot = (i * 8 + wave) * 64 + lane;
    const int row = slot >> 3;
    const int chunk = (slot & 7) ^ ((row >> 1) & 7);
    uint32_t off = soff[i];
    if (i < NCC && crmax < TC - 1) off = (uint32_t)(min(row, crmax) * (int)A.cfld * 4 + 16 * chunk);
    const void *base = i < NCC ? (const void *)(A.cf + (int64_t)c0c * A.cfld + 32 * cs) : (const void *)(pbase + 32 * cs);
    lds_u8 *wdst = (lds_u8 *)cdst + (i * 8 + wave) * 1024;
    if (cfull) {
      lds_copy16(base, off, (uint32_t)(size_t)wdst);
    } else if (32 * cs + 4 * chunk < A.df) {
      lds_copy16(base, off, (uint32_t)(size_t)wdst);
    } else {
      __attribute__((address_space(3))) uint32_t *z = (__attribute__((address_space(3))) uint32_t *)(wdst + 16 * lane);
      z[0] = z[1] = z[2] = z[3] = 0u;
    }
  };
  auto land = [&](int ct, int s) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (s == 0 && t < TC) cnl[ct & 1][t] = cnv;
  };

  f32x16 acc[CB][PB];
  // one stage: four steps of 8 dimensions (4 k-pairs per MFMA block); the operand
  // reads of step gg+1 and the copies of the next stage go out before step gg's MFMAs
  auto mfma_stage = [&](const uint8_t *buf, bool copying) {
    uint4 av[2][CB], bv[2][PB];
    auto read = [&](int gg, int set) {
      const int so = 16 * ((2 * gg + h) ^ ((r >> 1) & 7));
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
        bv[set][pb] = *reinterpret_cast<const uint4 *>(buf + (TC + wp * 32 * PB + pb * 32 + r) * kRowBytes + so);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        av[set][cb] = *reinterpret_cast<const uint4 *>(buf + (wc * 32 * CB + cb * 32 + r) * kRowBytes + so);
    };
    read(0, 0);
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      const int cur = gg & 1;
      if (gg + 1 < 4) read(gg + 1, cur ^ 1);
      __builtin_amdgcn_sched_barrier(0);
      if (copying) {
#pragma unroll
        for (int i = gg * NCOPY / 4; i < (gg + 1) * NCOPY / 4; ++i) copy(i);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int pb = 0; pb < PB; ++pb)
            acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(av[cur][cb][e]),
                                                              __uint_as_float(bv[cur][pb][e]), acc[cb][pb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // scores ||c||^2 - 2<x,c> and running argmin, lane-local and branch-free; rows
  // ascend with (cb, i) in a lane, so the strict comparison keeps the smallest
  // index among equal scores
  float best[PB];
  int bidx[PB];
#pragma unroll
  for (int pb = 0; pb < PB; ++pb) {
    best[pb] = INFINITY;
    bidx[pb] = INT_MAX;
  }
  auto epilogue = [&](int ct) {
    const float *cp = cnl[ct & 1];
    const int c0 = (g + ct * NG) * TC;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int crow0 = wc * 32 * CB + cb * 32 + 4 * h;
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const f32x4 cn4 = *reinterpret_cast<const f32x4 *>(&cp[crow0 + 8 * i4]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = c0 + crow0 + 8 * i4 + e;
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) {
            const float sc = fmaf(-2.0f, acc[cb][pb][4 * i4 + e], cn4[e]);
            const bool take = sc < best[pb];
            best[pb] = take ? sc : best[pb];
            bidx[pb] = take ? j : bidx[pb];
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  begin_copies(0, 0, fst0);
#pragma unroll
  for (int i = 0; i < NCOPY; ++i) copy(i);
  land(0, 0);
  __syncthreads();
  // stage s of tile ct reads buffer cur while the copies of the next stage fill nxt
  auto step = [&](int ct, int s, bool has_next, const uint8_t *cur, uint8_t *nxt) {
    const int s_n = (s + 1 == S) ? 0 : s + 1;
    const int ct_n = (s + 1 == S) ? ct + 1 : ct;
    if (s == 0) {
#pragma unroll
      for (int a = 0; a < CB; ++a)
#pragma unroll
        for (int b = 0; b < PB; ++b)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;
    }
    if (has_next) begin_copies(ct_n, s_n, nxt);
    mfma_stage(cur, has_next);
    if (has_next) land(ct_n, s_n);
    __syncthreads();
    if (s == S - 1) {
      epilogue(ct);
      // the next tile's steps write tile ct + 2's norms into cnl[ct & 1]
      __syncthreads();
    }
  };
  int cur_t = 0, cur_s = 0;  // tile and stage of the step about to run
  auto advance = [&]() {
    if (++cur_s == S) {
      cur_s = 0;
      ++cur_t;
    }
  };
  for (int it = 0; it < total; it += 2) {
    step(cur_t, cur_s, it + 1 < total, fst0, fst1);
    advance();
    if (it + 1 < total) {
      step(cur_t, cur_s, it + 2 < total, fst1, fst0);
      advance();
    }
  }

  // merge the two lane halves (rows 4h..), then the two centroid halves
#pragma unroll
  for (int pb = 0; pb < PB; ++pb) {
    const float os = __shfl_xor(best[pb], 32);
    const int oi = __shfl_xor(bidx[pb], 32);
    if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
      best[pb] = os;
      bidx[pb] = oi;
    }
  }
  float *ms = reinterpret_cast<float *>(fst0);
  int *mi = reinterpret_cast<int *>(fst0 + TP * sizeof(float));
  if (wc == 1 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      ms[wp * 32 * PB + pb * 32 + r] = best[pb];
      mi[wp * 32 * PB + pb * 32 + r] = bidx[pb];
    }
  }
  __syncthreads();
  if (wc == 0 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int pc = wp * 32 * PB + pb * 32 + r;
      const float os = ms[pc];
      const int oi = mi[pc];
      if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
        best[pb] = os;
        bidx[pb] = oi;
      }
      const int64_t p = p0 + pc;
      if (p < A.n) {
        if (A.keys) {
          atomicMin(A.keys + p, score_key(best[pb], bidx[pb]));
        } else {
          A.assign[p] = bidx[pb] + A.aoff;
          if (A.score) A.score[p] = best[pb];
        }
      }
    }
  }
}

// ---- hybrid assignment (fp32 front + 1-bit tail) with direct global-to-LDS stages ---
// The fp32 kernel's shape (8 waves, a 256-point tile against 256-centroid tiles,
// 4 x 2 blocks per wave, one workgroup per CU) on the segment decomposition of the
// squared distance (Sec. 3.1 SuperKMeans).  Per centroid tile the tail comes first:
// int8 stages of the centroids' residual codes (128 bytes of every row per stage,
// copied straight into LDS in the conflict-free slot layout) against the points'
// tail bits, which stay resident in LDS for the whole workgroup, regrouped at load
// so that widening a half-word to {0, 2} bytes costs a shift and a mask per
// register.  Seeded with -T the integer accumulators end at 2D - T; that becomes the
// 1-bit score ts = fmaf(-(alpha 2 sigma), 2D - T, sigma^2 Q) in fp32 (Eq. 4, the
// order the oracle uses), the same registers then start the fp32 front at -ts/2, and
// the front's fp32 stages follow, so the epilogue's ||c'||^2 - 2 acc is
// ||c'||^2 - 2<x',c'> + ts.  The copies of the next stage, of either kind, are spread
// over the current stage's four steps.
constexpr int kHybMaxTW = 20;  // resident tail words per point (640 tail dims)

template <int CB = 4>
__global__ __launch_bounds__(kQThreads, 1) void assign_hyb_kernel(AssignArgs A) {
  static_assert(CB == 2 || CB == 4, "128- or 256-centroid tiles");
  constexpr int TC = 64 * CB, TP = kQT, PB = k8PB;
  constexpr int NCC = TC / 64;           // centroid copies per thread and stage
  constexpr int NCOPY = (TC + TP) / 64;  // all copies per thread of a front stage
  constexpr int STAGE = (TC + TP) * kRowBytes;
  __shared__ __align__(16) uint8_t fst0[STAGE];
  __shared__ __align__(16) uint8_t fst1[STAGE];
  __shared__ __align__(16) float cnl[2][4][TC];  // per tile: ||c'||^2, -T (int bits), sigma^2 Q, 2 sigma
  __shared__ uint32_t bitsT[kHybMaxTW * TP];
  __shared__ float alp[TP];  // the points' alpha
  const int t = threadIdx.x;
  const int lane = t & 63, wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int wc = wave & 1, wp = wave >> 1;
  const int NG = A.ngroups;
  int64_t pt = blockIdx.x;
  int g = 0;
  if (NG > 1) {
    const int64_t l = blockIdx.x >> 3;
    pt = (l / NG) * 8 + (blockIdx.x & 7);
    g = (int)(l % NG);
    if (pt >= A.n_ptiles) return;  // whole workgroup, before any barrier
  }
  const int64_t p0 = pt * TP;
  const int SI = (A.di + kRowBytes - 1) / kRowBytes;  // tail stages
  const int SF = (A.df + 31) / 32;                    // front stages
  const int S = SI + SF;
  const int nct = (A.k + TC - 1) / TC;
  const int nmy = (nct - g + NG - 1) / NG;
  const int total = nmy * S;
  const int prmax = (int)min<int64_t>(A.n - 1 - p0, TP - 1);
  const float *pbase = A.pf + p0 * A.pfld;

  // resident tail bits, word-major, regrouped; words past the tail up to the last
  // stage's end are zero (the codes there are zero-filled too)
  {
    const int TW = A.di / 32;
    for (int e = t; e < 4 * SI * TP; e += kQThreads) {
      const int w = e / TP, pp = e - w * TP;
      uint32_t v = 0u;
      if (w < TW) v = regroup_bits(A.pbits[(p0 + min(pp, prmax)) * A.pbw + A.pbw0 + w]);
      bitsT[w * TP + pp] = v;
    }
  }
  if (t < TP) alp[t] = A.alpha[p0 + min(t, prmax)];

  // the stage being copied: tile c0c, stage cs of the tile, into buffer cdst
  int c0c = 0, crmax = 0, cs = 0;
  bool cfull = true, ctail = true;
  uint8_t *cdst = fst0;
  auto begin_copies = [&](int ct, int s, uint8_t *dst) {
    c0c = (g + ct * NG) * TC;
    crmax = min(A.k - 1 - c0c, TC - 1);
    cs = s;
    cdst = dst;
    ctail = s < SI;
    cfull = ctail ? kRowBytes * (s + 1) <= A.di : 32 * (s - SI + 1) <= A.df;
  };
  // copy i of a wave fills slots (8 i + wave) 64 .. + 63 of the stage: in a tail
  // stage rows 0 .. TC - 1 of centroid codes, in a front stage TC fp32 centroid rows
  // and then TP point rows; rows past the last centroid or point are clamped
  auto copy = [&](int i) {
    if (ctail && i >= NCC) return;  // a tail stage copies centroid codes only
    const int slot = (i * 8 + wave) * 64 + lane;
    const int row = slot >> 3;
    const int chunk = (slot & 7) ^ ((row >> 1) & 7);
    uint32_t off;
    const void *base;
    bool inside;
    if (ctail) {
      off = (uint32_t)(min(row, crmax) * (int)A.cild + 16 * chunk);
      base = A.ci8 + (int64_t)c0c * A.cild + kRowBytes * cs;
      inside = kRowBytes * cs + 16 * chunk < A.di;
    } else {
      const int sf = cs - SI;
      if (i < NCC) {
        off = (uint32_t)(min(row, crmax) * (int)A.cfld * 4 + 16 * chunk);
        base = A.cf + (int64_t)c0c * A.cfld + 32 * sf;
      } else {
        off = (uint32_t)(min(row - TC, prmax) * (int)A.pfld * 4 + 16 * chunk);
        base = pbase + 32 * sf;
      }
      inside = 32 * sf + 4 * chunk < A.df;
    }
    lds_u8 *wdst = (lds_u8 *)cdst + (i * 8 + wave) * 1024;
    if (cfull || inside) {
      lds_copy16(base, off, (uint32_t)(size_t)wdst);
    } else {
      __attribute__((address_space(3))) uint32_t *z = (__attribute__((address_space(3))) uint32_t *)(wdst + 16 * lane);
      z[0] = z[1] = z[2] = z[3] = 0u;
    }
  };
  auto land = [&]() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };
  // a tile's constants for row t: loaded during the first (tail) stage of the tile
  // before (the prologue for the first tile), where few registers are live, and
  // stored once that stage's copies have landed
  float cv[4] = {0.f, 0.f, 0.f, 0.f};
  auto load_consts = [&](int ct) {
    if (t < TC) {
      const int c0 = (g + ct * NG) * TC;
      const int j = c0 + min(t, A.k - 1 - c0);
      cv[0] = t <= A.k - 1 - c0 ? A.cp.cn[j] : INFINITY;
      cv[1] = __int_as_float(-A.cp.qsum[j]);
      cv[2] = A.cp.u[j];
      cv[3] = A.cp.sig2[j];
    }
  };
  auto store_consts = [&](int ct) {
    if (t < TC) {
#pragma unroll
      for (int q = 0; q < 4; ++q) cnl[ct & 1][q][t] = cv[q];
    }
  };

  f32x16 acc[CB][PB];  // the tail's int32 2D - T (bit patterns), then the fp32 front
  // one tail stage: four steps of 32 dims (one int8 MFMA per block and step)
  // a tile's accumulators start at -T of their row
  auto seed = [&](int ct) {
    const float *cp = cnl[ct & 1][1];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(cp + wc * 32 * CB + cb * 32 + 8 * m + 4 * h);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) acc[cb][pb][4 * m + e] = v[e];
      }
  };
  auto tail_stage = [&](int s, const uint8_t *buf, bool copying) {
    const uint32_t hsh = 4u * (uint32_t)h;
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      uint4 av[CB];
      i32x4 bv[PB];
      const int so = 16 * ((2 * gg + h) ^ ((r >> 1) & 7));
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        av[cb] = *reinterpret_cast<const uint4 *>(buf + (wc * 32 * CB + cb * 32 + r) * kRowBytes + so);
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) bv[pb] = widen_regrouped2(bitsT[(4 * s + gg) * TP + wp * 64 + pb * 32 + r] >> hsh);
      __builtin_amdgcn_sched_barrier(0);
      if (copying) {
#pragma unroll
        for (int i = gg * NCOPY / 4; i < (gg + 1) * NCOPY / 4; ++i) copy(i);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const i32x4 a4 = {(int)av[cb].x, (int)av[cb].y, (int)av[cb].z, (int)av[cb].w};
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
          acc[cb][pb] = __builtin_bit_cast(
              f32x16, __builtin_amdgcn_mfma_i32_32x32x32_i8(a4, bv[pb], __builtin_bit_cast(i32x16, acc[cb][pb]), 0, 0, 0));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // the tail's 2D - T to the fp32 seed -ts/2 of the front
  auto fold_tail = [&](int ct) {
    const float *cu = cnl[ct & 1][2];
    const float *c2 = cnl[ct & 1][3];
    float al[PB];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) al[pb] = alp[wp * 64 + pb * 32 + r];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int row0 = wc * 32 * CB + cb * 32 + 8 * m + 4 * h;
        const f32x4 u4 = *reinterpret_cast<const f32x4 *>(cu + row0);
        const f32x4 s4 = *reinterpret_cast<const f32x4 *>(c2 + row0);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) {
            const int sd = __float_as_int(acc[cb][pb][4 * m + e]);
            const float ts = fmaf(-(al[pb] * s4[e]), (float)sd, u4[e]);
            acc[cb][pb][4 * m + e] = -0.5f * ts;
          }
      }
  };
  // one front stage: four steps of 8 dims (4 k-pairs per MFMA block), operand reads
  // double-buffered
  auto front_stage = [&](const uint8_t *buf, bool copying) {
    uint4 av[2][CB], bv[2][PB];
    auto read = [&](int gg, int set) {
      const int so = 16 * ((2 * gg + h) ^ ((r >> 1) & 7));
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
        bv[set][pb] = *reinterpret_cast<const uint4 *>(buf + (TC + wp * 32 * PB + pb * 32 + r) * kRowBytes + so);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        av[set][cb] = *reinterpret_cast<const uint4 *>(buf + (wc * 32 * CB + cb * 32 + r) * kRowBytes + so);
    };
    read(0, 0);
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      const int cur = gg & 1;
      if (gg + 1 < 4) read(gg + 1, cur ^ 1);
      __builtin_amdgcn_sched_barrier(0);
      if (copying) {
#pragma unroll
        for (int i = gg * NCOPY / 4; i < (gg + 1) * NCOPY / 4; ++i) copy(i);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int pb = 0; pb < PB; ++pb)
            acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(av[cur][cb][e]),
                                                              __uint_as_float(bv[cur][pb][e]), acc[cb][pb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  float best[PB];
  int bidx[PB];
#pragma unroll
  for (int pb = 0; pb < PB; ++pb) {
    best[pb] = INFINITY;
    bidx[pb] = INT_MAX;
  }
  auto epilogue = [&](int ct) {
    const float *cp = cnl[ct & 1][0];
    const int c0 = (g + ct * NG) * TC;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int crow0 = wc * 32 * CB + cb * 32 + 4 * h;
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const f32x4 cn4 = *reinterpret_cast<const f32x4 *>(&cp[crow0 + 8 * i4]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = c0 + crow0 + 8 * i4 + e;
#pragma unroll
          for (int pb = 0; pb < PB; ++pb) {
            const float sc = fmaf(-2.0f, acc[cb][pb][4 * i4 + e], cn4[e]);
            const bool take = sc < best[pb];
            best[pb] = take ? sc : best[pb];
            bidx[pb] = take ? j : bidx[pb];
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  load_consts(0);
  begin_copies(0, 0, fst0);
#pragma unroll
  for (int i = 0; i < NCOPY; ++i) copy(i);
  land();
  store_consts(0);
  __syncthreads();  // also publishes the resident bits and alpha
  // Per tile: the tail stages, the fold, the front stages, the scores.  Stage gi of
  // the workgroup's sequence reads buffer gi & 1 while the copies of stage gi + 1
  // fill the other one.  The tail and front stages run in loops of their own (one
  // loop with a branch between the two kinds of MFMA stage makes the register
  // allocator keep a second copy of the accumulators).  A tile's first stage is a
  // tail stage and never the last stage (S >= 2): its copies land and the next
  // tile's constants wait with them.
  int gi = 0;
  for (int ct = 0; ct < nmy; ++ct) {
    seed(ct);
    for (int s = 0; s < SI; ++s, ++gi) {
      const uint8_t *cur = (gi & 1) ? fst1 : fst0;
      uint8_t *nxt = (gi & 1) ? fst0 : fst1;
      begin_copies(ct, s + 1, nxt);  // s + 1 <= SI < S
      const bool consts = s == 0 && ct + 1 < nmy;
      if (consts) load_consts(ct + 1);
      tail_stage(s, cur, true);
      land();
      // cnl[(ct + 1) & 1] held tile ct - 1's constants, last read before the barrier
      // that closed that tile
      if (consts) store_consts(ct + 1);
      __syncthreads();
    }
    fold_tail(ct);
    for (int s = SI; s < S; ++s, ++gi) {
      const uint8_t *cur = (gi & 1) ? fst1 : fst0;
      uint8_t *nxt = (gi & 1) ? fst0 : fst1;
      const bool has_next = gi + 1 < total;
      if (has_next) begin_copies(s + 1 == S ? ct + 1 : ct, s + 1 == S ? 0 : s + 1, nxt);
      front_stage(cur, has_next);
      if (has_next) land();
      __syncthreads();
    }
    epilogue(ct);
    // the next tile's first stage writes tile ct + 2's constants into cnl[ct & 1]
    __syncthreads();
  }

  // merge the two lane halves (rows 4h..), then the two centroid halves
#pragma unroll
  for (int pb = 0; pb < PB; ++pb) {
    const float os = __shfl_xor(best[pb], 32);
    const int oi = __shfl_xor(bidx[pb], 32);
    if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
      best[pb] = os;
      bidx[pb] = oi;
    }
  }
  float *ms = reinterpret_cast<float *>(fst0);
  int *mi = reinterpret_cast<int *>(fst0 + TP * sizeof(float));
  if (wc == 1 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      ms[wp * 32 * PB + pb * 32 + r] = best[pb];
      mi[wp * 32 * PB + pb * 32 + r] = bidx[pb];
    }
  }
  __syncthreads();
  if (wc == 0 && h == 0) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int pc = wp * 32 * PB + pb * 32 + r;
      const float os = ms[pc];
      const int oi = mi[pc];
      if (os < best[pb] || (os == best[pb] && oi < bidx[pb])) {
        best[pb] = os;
        bidx[pb] = oi;
      }
      const int64_t p = p0 + pc;
      if (p < A.n) {
        if (A.keys) {
          atomicMin(A.keys + p, score_key(best[pb], bidx[pb]));
        } else {
          A.assign[p] = bidx[pb] + A.aoff;
          if (A.score) A.score[p] = best[pb];
        }
      }
    }
  }
}

// ---- centroid preparation: one workgroup per centroid ----------------------

template <int FMT>
__global__ __launch_bounds__(256) void prep_kernel(const void *Cv, int k, int d, int d0, const float *m,
                                                   float *cn, int *qsum, float *u, float *sig2, int8_t *q,
                                                   uint16_t *cb) {
  __shared__ double shd[256];
  __shared__ float shf[256];
  __shared__ int shi[256];
  const int j = blockIdx.x;
  const int t = threadIdx.x;
  if (FMT == KM_F32 || FMT == KM_HYBRID) {
    const float *c = static_cast<const float *>(Cv) + (int64_t)j * d;
    const int dd = FMT == KM_F32 ? d : d0;
    double s = 0.0;
    for (int i = t; i < dd; i += 256) s += (double)c[i] * (double)c[i];
    s = block_sum_f64(s, shd);
    if (t == 0) cn[j] = (float)s;
  }
  if (FMT == KM_BF16) {  // round the fp32 centroid to bfloat16; ||c||^2 of the rounded values
    const float *c = static_cast<const float *>(Cv) + (int64_t)j * d;
    double s = 0.0;
    for (int i = t; i < d; i += 256) {
      const uint32_t b = bf16_bits(c[i]);
      cb[(int64_t)j * d + i] = (uint16_t)b;
      const double v = bf16_value(b);
      s += v * v;
    }
    s = block_sum_f64(s, shd);
    if (t == 0) cn[j] = (float)s;
  }
  if (FMT == KM_SQ8) {  // recentred int8 codes (code - 128) and their squared norm
    const uint8_t *c = static_cast<const uint8_t *>(Cv) + (int64_t)j * d;
    int s = 0;
    for (int i = t; i < d; i += 256) {
      const int v = (int)c[i] - 128;
      q[(int64_t)j * d + i] = (int8_t)v;
      s += v * v;
    }
    shi[t] = s;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shi[t] += shi[t + st];
      __syncthreads();
    }
    if (t == 0) qsum[j] = -shi[0];  // negated: the assignment maximises 2<x~,c~> - ||c~||^2
  }
  if (FMT == KM_LVQ4) {  // LVQ4 of the centroid (Sec. 3.1 LVQ): b = min, s = range / 15, S, Q, N
    const float *c = static_cast<const float *>(Cv) + (int64_t)j * d;
    float lo = INFINITY, hi = -INFINITY;
    for (int i = t; i < d; i += 256) {
      lo = fminf(lo, c[i]);
      hi = fmaxf(hi, c[i]);
    }
    shf[t] = lo;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shf[t] = fminf(shf[t], shf[t + st]);
      __syncthreads();
    }
    lo = shf[0];
    __syncthreads();
    shf[t] = hi;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shf[t] = fmaxf(shf[t], shf[t + st]);
      __syncthreads();
    }
    hi = shf[0];
    const float sc = hi > lo ? (hi - lo) / 15.0f : 1.0f;
    int ts = 0, tq = 0;
    for (int i = t; i < d; i += 256) {
      const int v = (int)fminf(fmaxf(rintf((c[i] - lo) / sc), 0.f), 15.f);
      // within each 8 dimensions the even ones first, then the odd ones: the byte
      // order in which the assignment unpacks the points' packed codes
      q[(int64_t)j * d + (i & ~7) + ((i & 1) << 2) + ((i >> 1) & 3)] = (int8_t)v;
      ts += v;
      tq += v * v;
    }
    __syncthreads();
    shi[t] = ts;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shi[t] += shi[t + st];
      __syncthreads();
    }
    const int S = shi[0];
    __syncthreads();
    shi[t] = tq;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shi[t] += shi[t + st];
      __syncthreads();
    }
    if (t == 0) {
      const int Q = shi[0];
      const float db = (float)d * lo;
      qsum[j] = S;
      u[j] = fmaf(sc * sc, (float)Q, fmaf(2.0f * lo * sc, (float)S, db * lo));
      sig2[j] = sc;
      cn[j] = lo;
    }
  }
  if (FMT == KM_RABITQ) {  // per-centroid SQ4 of the residual (Eq. 5): b = min, s = range / 15
    const float *c = static_cast<const float *>(Cv) + (int64_t)j * d;
    float lo = INFINITY, hi = -INFINITY;
    double nn = 0.0;
    for (int i = t; i < d; i += 256) {
      lo = fminf(lo, c[i]);
      hi = fmaxf(hi, c[i]);
      nn += (double)c[i] * (double)c[i];
    }
    nn = block_sum_f64(nn, shd);
    shf[t] = lo;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shf[t] = fminf(shf[t], shf[t + st]);
      __syncthreads();
    }
    lo = shf[0];
    __syncthreads();
    shf[t] = hi;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shf[t] = fmaxf(shf[t], shf[t + st]);
      __syncthreads();
    }
    hi = shf[0];
    const float sc = hi > lo ? (hi - lo) / 15.0f : 1.0f;
    int ts = 0;
    for (int i = t; i < d; i += 256) {
      const float v = fminf(fmaxf(rintf((c[i] - lo) / sc), 0.f), 15.f);
      q[(int64_t)j * d + i] = (int8_t)(int)v;
      ts += (int)v;
    }
    __syncthreads();
    shi[t] = ts;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shi[t] += shi[t + st];
      __syncthreads();
    }
    if (t == 0) {
      qsum[j] = shi[0];
      u[j] = (float)nn;
      sig2[j] = sc;
      cn[j] = lo;
    }
  }
  if (FMT == KM_SIGN1 || FMT == KM_HYBRID) {
    const float *c = static_cast<const float *>(Cv) + (int64_t)j * d;
    const int dt = d - d0;
    float mx = 0.f;
    for (int i = d0 + t; i < d; i += 256) mx = fmaxf(mx, fabsf(c[i] - m[i]));
    shf[t] = mx;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shf[t] = fmaxf(shf[t], shf[t + st]);
      __syncthreads();
    }
    mx = shf[0];
    const float sg = mx > 0.f ? mx / 127.0f : 1.0f;
    int ts = 0, qq = 0;
    for (int i = d0 + t; i < d; i += 256) {
      float v = mx > 0.f ? rintf((c[i] - m[i]) / sg) : 0.f;
      v = fminf(fmaxf(v, -127.f), 127.f);
      const int qi = (int)v;
      q[(int64_t)j * dt + (i - d0)] = (int8_t)qi;
      ts += qi;
      qq += qi * qi;
    }
    __syncthreads();
    shi[t] = ts;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shi[t] += shi[t + st];
      __syncthreads();
    }
    const int T = shi[0];
    __syncthreads();
    shi[t] = qq;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) shi[t] += shi[t + st];
      __syncthreads();
    }
    if (t == 0) {
      const int Q = shi[0];
      qsum[j] = T;
      u[j] = (sg * sg) * (float)Q;
      sig2[j] = 2.0f * sg;
    }
  }
}

// ---- point-only terms of the in-space distance ------------------------------
// F32, BF16: ||x||^2 ; SQ8: ||code-128||^2 ; SIGN1: alpha^2 d ; HYBRID: ||x'||^2 + alpha^2 (d - d0)
// One wave per point, 16-byte loads.
template <int FMT>
__global__ __launch_bounds__(256) void xconst_kernel(Points P, float *xc) {
  const int lane = threadIdx.x & 63;
  const int64_t p = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (p >= P.n) return;
  double s = 0.0;
  if (FMT == KM_F32 || FMT == KM_HYBRID) {
    const float *x = FMT == KM_F32 ? static_cast<const float *>(P.data) + p * P.ld : P.front + p * P.d_front;
    const int dd = FMT == KM_F32 ? P.d : P.d_front;
    for (int i = 4 * lane; i < dd; i += 256) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(x + i);
      s += (double)v.x * v.x + (double)v.y * v.y + (double)v.z * v.z + (double)v.w * v.w;
    }
  } else if (FMT == KM_LVQ4) {
    if (lane == 0) s = P.vparams[4 * p + 3];  // N_x (only lane 0's value is kept)
  } else if (FMT == KM_BF16) {
    const uint16_t *x = static_cast<const uint16_t *>(P.data) + p * P.ld;
    for (int i = 8 * lane; i < P.d; i += 512) {
      const uint4 w = *reinterpret_cast<const uint4 *>(x + i);
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const double lo = bf16_value(ws[q] & 0xffffu), hi = bf16_value(ws[q] >> 16);
        s += lo * lo + hi * hi;
      }
    }
  } else if (FMT == KM_SQ8) {
    const uint8_t *x = static_cast<const uint8_t *>(P.data) + p * P.ld;
    int acc = 0;
    for (int i = 16 * lane; i < P.d; i += 1024) {
      const uint4 w = *reinterpret_cast<const uint4 *>(x + i);
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int v = (int)((ws[q] >> (8 * e)) & 255u) - 128;
          acc += v * v;
        }
    }
    s = (double)acc;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) {
    if (is_bits_fmt(FMT)) {
      const double a = P.alpha[p];
      s += a * a * (double)(P.d - (FMT == KM_HYBRID ? P.d_front : 0));
    }
    xc[p] = (float)s;
  }
}

// ---- objective: sum of (point term + score), deterministic two-level sum ----
__global__ __launch_bounds__(256) void objective_partial_kernel(const float *xc, const float *score, int64_t n,
                                                                double *partials) {
  __shared__ double sh[256];
  double s = 0.0;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < n; p += stride)
    s += (double)xc[p] + (double)score[p];
  s = block_sum_f64(s, sh);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void sum_partials_kernel(const double *partials, int np, double *out) {
  __shared__ double sh[256];
  double s = 0.0;
  for (int i = threadIdx.x; i < np; i += 256) s += partials[i];
  s = block_sum_f64(s, sh);
  if (threadIdx.x == 0) *out = s;
}

// ---- STEP 1: gather the sampled points as initial centroids -----------------
template <int FMT>
__global__ __launch_bounds__(256) void gather_kernel(Points P, const int64_t *idx, void *Cv) {
  const int j = blockIdx.x;
  const int64_t row = idx[j];  // validated on the host
  const int d = P.d;
  if (FMT == KM_F32) {
    const float *x = static_cast<const float *>(P.data) + row * P.ld;
    float *c = static_cast<float *>(Cv) + (int64_t)j * d;
    for (int i = threadIdx.x; i < d; i += 256) c[i] = x[i];
  } else if (FMT == KM_LVQ4) {
    const uint8_t *x = static_cast<const uint8_t *>(P.data) + row * P.ld;
    const float sx = P.vparams[4 * row], bx = P.vparams[4 * row + 1];
    float *c = static_cast<float *>(Cv) + (int64_t)j * d;
    for (int i = threadIdx.x; i < d; i += 256) c[i] = fmaf(sx, (float)((x[i >> 1] >> (4 * (i & 1))) & 15u), bx);
  } else if (FMT == KM_BF16) {
    const uint16_t *x = static_cast<const uint16_t *>(P.data) + row * P.ld;
    float *c = static_cast<float *>(Cv) + (int64_t)j * d;
    for (int i = threadIdx.x; i < d; i += 256) c[i] = bf16_value(x[i]);
  } else if (FMT == KM_SQ8) {
    const uint8_t *x = static_cast<const uint8_t *>(P.data) + row * P.ld;
    uint8_t *c = static_cast<uint8_t *>(Cv) + (int64_t)j * d;
    for (int i = threadIdx.x; i < d; i += 256) c[i] = x[i];
  } else {
    const int d0 = FMT == KM_HYBRID ? P.d_front : 0;
    const uint32_t *b = static_cast<const uint32_t *>(P.data) + row * (d / 32);
    const float a = P.alpha[row];
    float *c = static_cast<float *>(Cv) + (int64_t)j * d;
    for (int i = threadIdx.x; i < d; i += 256) {
      if (i < d0) {
        c[i] = P.front[row * d0 + i];
      } else {
        const float sg = ((b[i >> 5] >> (i & 31)) & 1u) ? a : -a;
        c[i] = (P.center ? P.center[i] : 0.0f) + sg;  // decoded point m + alpha (2b - 1)
      }
    }
  }
}

// ---- full-precision cost of a partition: sum ||x - c_a||^2 in fp64 ----------
// One wave per point at a time, 16-byte loads of the point and its centroid row.
// Rows whose length is not a multiple of 4 fall back to scalar loads.
__global__ __launch_bounds__(256) void cost_kernel(const float *X, int64_t n, int d, int64_t ldx, const float *C,
                                                   int k, const int32_t *assign, double *partials) {
  __shared__ double sh[256];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const bool vec = (d % 4 == 0) && (ldx % 4 == 0) &&
                   (((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(C)) & 15u) == 0);
  double s = 0.0;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t p = (int64_t)blockIdx.x * 4 + wv; p < n; p += stride) {
    const int a = assign[p];
    if (a < 0 || a >= k) continue;
    const float *x = X + p * ldx;
    const float *c = C + (int64_t)a * d;
    if (vec) {
      for (int i = 4 * lane; i < d; i += 256) {
        const f32x4 xv = *reinterpret_cast<const f32x4 *>(x + i);
        const f32x4 cv = *reinterpret_cast<const f32x4 *>(c + i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double t = (double)xv[e] - (double)cv[e];
          s += t * t;
        }
      }
    } else {
      for (int i = lane; i < d; i += 64) {
        const double t = (double)x[i] - (double)c[i];
        s += t * t;
      }
    }
  }
  s = block_sum_f64(s, sh);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

constexpr int kObjBlocks = 1024;

// Centroid-tile groups of the hybrid kernel: up to 8 workgroups share a point
// tile, each scanning every 8th centroid tile.
// centroids per tile of the 8-wave kernels (fp32, SQ8, bf16): 128 when k fits, else 256
static int q8_tile_centroids(int k) { return k <= 128 ? 128 : 256; }

// Centroid-tile groups of the 8-wave kernels (one workgroup per CU, long-lived
// workgroups): the group count g that minimises the rounds of workgroups over the
// CUs times the centroid tiles of the busiest group, ceil(npt g / CUs) ceil(nct / g).
// This fills the GPU when the point tiles alone do not, and shortens the partly
// filled last round (1M points: 3907 point tiles = 15.3 rounds alone, 30.5 with
// g = 2); the smallest such g, since each group adds a key merge.
static int tile_groups(int64_t n, int k) {
  const int64_t npt = cdiv(n, kQT);
  const int nct = (int)cdiv(k, q8_tile_centroids(k));
  const int64_t cus = cu_count();
  int best_g = 1;
  int64_t best = -1;
  for (int g = 1; g <= std::min(8, nct); ++g) {
    const int64_t cost = cdiv(npt * g, cus) * cdiv(nct, g);
    if (best < 0 || cost < best) {
      best = cost;
      best_g = g;
    }
  }
  return best_g;
}

// hybrid points whose tail words fit the direct-copy kernel's resident LDS array
static bool hyb_direct(const Points &P) { return P.fmt == KM_HYBRID && P.d - P.d_front <= 32 * kHybMaxTW; }

int assign_groups(const Points &P, int k) {
  if (P.fmt == KM_F32 || hyb_direct(P)) return tile_groups(P.n, k);
  if (P.fmt == KM_HYBRID) {
    constexpr int TC = Geo<Blocking<KM_F32>::CB, Blocking<KM_F32>::PB>::TC;
    return (int)std::min<int64_t>(8, cdiv(k, TC));
  }
  if (P.fmt == KM_BF16 || P.fmt == KM_LVQ4 || (P.fmt == KM_SQ8 && P.d <= kQMaxDimSQ8)) return tile_groups(P.n, k);
  return 1;
}

template <int FMT>
km_status launch_assign_t(const Points &P, const void *C, const CentroidPrep &cp, int k, int32_t *assign,
                          float *score, hipStream_t s, int aoff) {
  AssignArgs A{};
  A.aoff = aoff;
  A.ngroups = 1;
  A.n = P.n;
  A.k = k;
  A.assign = assign;
  A.score = score;
  A.cp = cp;
  A.alpha = P.alpha;
  if (FMT == KM_F32) {
    A.pf = static_cast<const float *>(P.data);
    A.pfld = P.ld;
    A.cf = static_cast<const float *>(C);
    A.cfld = P.d;
    A.df = P.d;
  } else if (FMT == KM_SQ8) {  // recentred centroid codes for the direct-copy kernel
    A.pi8 = static_cast<const uint8_t *>(P.data);
    A.pild = P.ld;
    A.ci8 = P.d <= kQMaxDimSQ8 ? cp.q : static_cast<const int8_t *>(C);
    A.cild = P.d;
    A.di = P.d;
  } else if (FMT == KM_LVQ4) {  // packed 4-bit point codes, unpacked centroid codes
    A.pi8 = static_cast<const uint8_t *>(P.data);
    A.pild = P.ld;
    A.ci8 = cp.q;
    A.cild = P.d;
    A.di = P.d;
    A.vparams = P.vparams;
  } else if (FMT == KM_BF16) {  // byte-addressed rows of 16-bit values
    A.pi8 = static_cast<const uint8_t *>(P.data);
    A.pild = 2 * P.ld;
    A.ci8 = reinterpret_cast<const int8_t *>(cp.cb);
    A.cild = 2 * (int64_t)P.d;
    A.di = 2 * P.d;
  } else {
    const int d0 = FMT == KM_HYBRID ? P.d_front : 0;
    if (FMT == KM_HYBRID) {
      A.pf = P.front;
      A.pfld = d0;
      A.cf = static_cast<const float *>(C);
      A.cfld = P.d;
      A.df = d0;
    }
    A.pbits = static_cast<const uint32_t *>(P.data);
    A.pbw = P.d / 32;
    A.pbw0 = d0 / 32;
    A.ci8 = cp.q;
    A.cild = P.d - d0;
    A.di = P.d - d0;
  }
  if constexpr (FMT == KM_SIGN1 || FMT == KM_RABITQ) {
    if (P.d <= 32 * kBWordsSmall) {
      hipLaunchKernelGGL((assign_bits_kernel<FMT, 4, kBWordsSmall>), dim3((unsigned)cdiv(P.n, 256)), dim3(256), 0, s, A);
    } else if (P.d <= 32 * kBWordsLarge) {
      hipLaunchKernelGGL((assign_bits_kernel<FMT, 8, kBWordsLarge>), dim3((unsigned)cdiv(P.n, 512)), dim3(512), 0, s, A);
    } else {
      hipLaunchKernelGGL(assign_i8_kernel<FMT>, dim3((unsigned)cdiv(P.n, kT8)), dim3(k8Threads), 0, s, A);
    }
  } else if constexpr (FMT == KM_SQ8 || FMT == KM_BF16 || FMT == KM_LVQ4) {
    if (FMT != KM_SQ8 || P.d <= kQMaxDimSQ8) {
      const int64_t npt = cdiv(P.n, kQT);
      const int ng = assign_groups(P, k);
      A.n_ptiles = npt;
      if (ng > 1) {
        const dim3 gp((unsigned)cdiv(P.n, 256));
        A.ngroups = ng;
        A.keys = cp.keys;
        hipLaunchKernelGGL(keys_init_kernel, gp, dim3(256), 0, s, cp.keys, P.n);
      }
      const dim3 grid((unsigned)(ng > 1 ? cdiv(npt, 8) * 8 * ng : npt));
      const bool pk = FMT == KM_SQ8 && P.d <= kQPackMaxDim;
      if (q8_tile_centroids(k) == 128) {
        if (pk)
          hipLaunchKernelGGL((assign_q8_kernel<FMT, false, 2, FMT == KM_SQ8>), grid, dim3(kQThreads), 0, s, A);
        else
          hipLaunchKernelGGL((assign_q8_kernel<FMT, false, 2>), grid, dim3(kQThreads), 0, s, A);
      } else if constexpr (FMT == KM_BF16) {
        // 16 waves of 64 x 64: half the direct copies per wave of the 8-wave shape
        hipLaunchKernelGGL((assign_q8_kernel<FMT, false, 2, false, 4>), grid, dim3(kQWideThreads), 0, s, A);
      } else {
        if (pk)
          hipLaunchKernelGGL((assign_q8_kernel<FMT, false, 4, FMT == KM_SQ8>), grid, dim3(kQThreads), 0, s, A);
        else
          hipLaunchKernelGGL((assign_q8_kernel<FMT, false, 4>), grid, dim3(kQThreads), 0, s, A);
      }
      if (ng > 1) {
        const dim3 gp((unsigned)cdiv(P.n, 256));
        hipLaunchKernelGGL(keys_unpack_kernel<FMT == KM_SQ8>, gp, dim3(256), 0, s, cp.keys, P.n, assign, score, aoff);
      }
    } else if constexpr (FMT == KM_SQ8) {
      hipLaunchKernelGGL(assign_i8_kernel<FMT>, dim3((unsigned)cdiv(P.n, kT8)), dim3(k8Threads), 0, s, A);
    }
  } else if constexpr (FMT == KM_F32) {
    const int64_t npt = cdiv(P.n, kQT);
    const int ng = assign_groups(P, k);
    A.n_ptiles = npt;
    if (ng > 1) {
      const dim3 gp((unsigned)cdiv(P.n, 256));
      A.ngroups = ng;
      A.keys = cp.keys;
      hipLaunchKernelGGL(keys_init_kernel, gp, dim3(256), 0, s, cp.keys, P.n);
    }
    const dim3 grid((unsigned)(ng > 1 ? cdiv(npt, 8) * 8 * ng : npt));
    if (q8_tile_centroids(k) == 128)
      hipLaunchKernelGGL((assign_f32_kernel<false, 2>), grid, dim3(kQThreads), 0, s, A);
    else
      hipLaunchKernelGGL((assign_f32_kernel<false, 4>), grid, dim3(kQThreads), 0, s, A);
    if (ng > 1) {
      const dim3 gp((unsigned)cdiv(P.n, 256));
      hipLaunchKernelGGL(keys_unpack_kernel<false>, gp, dim3(256), 0, s, cp.keys, P.n, assign, score, aoff);
    }
  } else if (FMT == KM_HYBRID && hyb_direct(P)) {
    const int64_t npt = cdiv(P.n, kQT);
    const int ng = assign_groups(P, k);
    A.n_ptiles = npt;
    if (ng > 1) {
      const dim3 gp((unsigned)cdiv(P.n, 256));
      A.ngroups = ng;
      A.keys = cp.keys;
      hipLaunchKernelGGL(keys_init_kernel, gp, dim3(256), 0, s, cp.keys, P.n);
    }
    const dim3 grid((unsigned)(ng > 1 ? cdiv(npt, 8) * 8 * ng : npt));
    if (q8_tile_centroids(k) == 128)
      hipLaunchKernelGGL((assign_hyb_kernel<2>), grid, dim3(kQThreads), 0, s, A);
    else
      hipLaunchKernelGGL((assign_hyb_kernel<4>), grid, dim3(kQThreads), 0, s, A);
    if (ng > 1) {
      const dim3 gp((unsigned)cdiv(P.n, 256));
      hipLaunchKernelGGL(keys_unpack_kernel<false>, gp, dim3(256), 0, s, cp.keys, P.n, assign, score, aoff);
    }
  } else {
    constexpr int TP = Geo<Blocking<FMT>::CB, Blocking<FMT>::PB>::TP;
    const int64_t npt = cdiv(P.n, TP);
    const int ng = assign_groups(P, k);
    const dim3 gp((unsigned)cdiv(P.n, 256));
    A.n_ptiles = npt;
    if (ng > 1) {
      A.ngroups = ng;
      A.keys = cp.keys;
      hipLaunchKernelGGL(keys_init_kernel, gp, dim3(256), 0, s, cp.keys, P.n);
      hipLaunchKernelGGL(assign_kernel<FMT>, dim3((unsigned)(cdiv(npt, 8) * 8 * ng)), dim3(kThreads), 0, s, A);
      hipLaunchKernelGGL(keys_unpack_kernel<false>, gp, dim3(256), 0, s, cp.keys, P.n, assign, score, aoff);
    } else {
      hipLaunchKernelGGL(assign_kernel<FMT>, dim3((unsigned)npt), dim3(kThreads), 0, s, A);
    }
  }
  KMQ_LAUNCH_CHECK("assign_kernel");
  return KM_OK;
}

}  // namespace

// prep workspace: cn, qsum, u, sig2 (k each) | residual codes or bf16 rows | keys (n)
static size_t prep_codes_bytes(const Points &P, int k) {
  const int d0 = P.fmt == KM_HYBRID ? P.d_front : 0;
  if (is_bits_fmt(P.fmt)) return (size_t)k * (size_t)(P.d - d0);
  if (P.fmt == KM_LVQ4 || P.fmt == KM_SQ8) return (size_t)k * (size_t)P.d;
  if (P.fmt == KM_BF16) return 2 * (size_t)k * (size_t)P.d;
  return 0;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t prep_bytes(const Points &P, int k) {
  size_t b = align256(16 * (size_t)k) + align256(prep_codes_bytes(P, k));
  if (assign_groups(P, k) > 1) b += align256(8 * (size_t)P.n);
  return b;
}

km_status launch_prep(const Points &P, const void *C, int k, void *ws, CentroidPrep *out, hipStream_t s) {
  uint8_t *w = static_cast<uint8_t *>(ws);
  float *cn = reinterpret_cast<float *>(w);
  int *qsum = reinterpret_cast<int *>(w + (size_t)k * 4);
  float *u = reinterpret_cast<float *>(w + (size_t)k * 8);
  float *sig2 = reinterpret_cast<float *>(w + (size_t)k * 12);
  int8_t *q = reinterpret_cast<int8_t *>(w + align256(16 * (size_t)k));
  uint16_t *cb = reinterpret_cast<uint16_t *>(q);  // BF16 uses the same region for its rows
  out->keys = assign_groups(P, k) > 1 ? reinterpret_cast<unsigned long long *>(
                                            w + align256(16 * (size_t)k) + align256(prep_codes_bytes(P, k)))
                                      : nullptr;
  out->cn = cn;
  out->qsum = qsum;
  out->u = u;
  out->sig2 = sig2;
  out->q = q;
  out->cb = cb;
  const int d0 = P.fmt == KM_HYBRID ? P.d_front : 0;
  switch (P.fmt) {
    case KM_F32:
      hipLaunchKernelGGL(prep_kernel<KM_F32>, dim3(k), dim3(256), 0, s, C, k, P.d, 0, nullptr, cn, qsum, u, sig2, q, cb);
      break;
    case KM_BF16:
      hipLaunchKernelGGL(prep_kernel<KM_BF16>, dim3(k), dim3(256), 0, s, C, k, P.d, 0, nullptr, cn, qsum, u, sig2, q,
                         cb);
      break;
    case KM_SQ8:
      hipLaunchKernelGGL(prep_kernel<KM_SQ8>, dim3(k), dim3(256), 0, s, C, k, P.d, 0, nullptr, cn, qsum, u, sig2, q, cb);
      break;
    case KM_SIGN1:
      hipLaunchKernelGGL(prep_kernel<KM_SIGN1>, dim3(k), dim3(256), 0, s, C, k, P.d, 0, P.center, cn, qsum, u, sig2,
                         q, cb);
      break;
    case KM_LVQ4:
      hipLaunchKernelGGL(prep_kernel<KM_LVQ4>, dim3(k), dim3(256), 0, s, C, k, P.d, 0, nullptr, cn, qsum, u, sig2, q,
                         cb);
      break;
    case KM_RABITQ:
      hipLaunchKernelGGL(prep_kernel<KM_RABITQ>, dim3(k), dim3(256), 0, s, C, k, P.d, 0, nullptr, cn, qsum, u, sig2, q,
                         cb);
      break;
    case KM_HYBRID:
      hipLaunchKernelGGL(prep_kernel<KM_HYBRID>, dim3(k), dim3(256), 0, s, C, k, P.d, d0, P.center, cn, qsum, u,
                         sig2, q, cb);
      break;
    default:
      return KM_EUNSUPPORTED;
  }
  KMQ_LAUNCH_CHECK("prep_kernel");
  return KM_OK;
}

km_status launch_assign(const Points &P, const void *C, const CentroidPrep &cp, int k, int32_t *assign,
                        float *score, hipStream_t s, int aoff) {
  switch (P.fmt) {
    case KM_F32: return launch_assign_t<KM_F32>(P, C, cp, k, assign, score, s, aoff);
    case KM_BF16: return launch_assign_t<KM_BF16>(P, C, cp, k, assign, score, s, aoff);
    case KM_SQ8: return launch_assign_t<KM_SQ8>(P, C, cp, k, assign, score, s, aoff);
    case KM_SIGN1: return launch_assign_t<KM_SIGN1>(P, C, cp, k, assign, score, s, aoff);
    case KM_HYBRID: return launch_assign_t<KM_HYBRID>(P, C, cp, k, assign, score, s, aoff);
    case KM_RABITQ: return launch_assign_t<KM_RABITQ>(P, C, cp, k, assign, score, s, aoff);
    case KM_LVQ4: return launch_assign_t<KM_LVQ4>(P, C, cp, k, assign, score, s, aoff);
    default: return KM_EUNSUPPORTED;
  }
}

int segment_tile_centroids(int k_seg) { return k_seg <= 128 ? 128 : 256; }

int assign_segment_rows(const Points &P) {
  if (P.fmt == KM_F32) return kQT;
  if (P.fmt == KM_BF16 || (P.fmt == KM_SQ8 && P.d <= kQMaxDimSQ8)) return kQT;
  return 0;
}

km_status launch_assign_segments(const Points &P, const void *C, const CentroidPrep &cp, const int4 *segs,
                                 const int2 *tiles, int64_t ntiles, int tile_c, int32_t *assign, float *score,
                                 hipStream_t s) {
  if (assign_segment_rows(P) == 0) return KM_EUNSUPPORTED;
  if (ntiles == 0) return KM_OK;
  AssignArgs A{};
  A.ngroups = 1;
  A.n = P.n;
  A.assign = assign;
  A.score = score;
  A.cp = cp;
  A.segs = segs;
  A.tiles = tiles;
  if (P.fmt == KM_F32) {
    A.pf = static_cast<const float *>(P.data);
    A.pfld = P.ld;
    A.cf = static_cast<const float *>(C);
    A.cfld = P.d;
    A.df = P.d;
    if (tile_c == 128)
      hipLaunchKernelGGL((assign_f32_kernel<true, 2>), dim3((unsigned)ntiles), dim3(kQThreads), 0, s, A);
    else
      hipLaunchKernelGGL((assign_f32_kernel<true, 4>), dim3((unsigned)ntiles), dim3(kQThreads), 0, s, A);
  } else if (P.fmt == KM_SQ8) {  // recentred centroid codes from the preparation
    A.pi8 = static_cast<const uint8_t *>(P.data);
    A.pild = P.ld;
    A.ci8 = cp.q;
    A.cild = P.d;
    A.di = P.d;
    const dim3 grid((unsigned)ntiles);
    const bool pk = P.d <= kQPackMaxDim;
    if (tile_c == 128) {
      if (pk)
        hipLaunchKernelGGL((assign_q8_kernel<KM_SQ8, true, 2, true>), grid, dim3(kQThreads), 0, s, A);
      else
        hipLaunchKernelGGL((assign_q8_kernel<KM_SQ8, true, 2>), grid, dim3(kQThreads), 0, s, A);
    } else {
      if (pk)
        hipLaunchKernelGGL((assign_q8_kernel<KM_SQ8, true, 4, true>), grid, dim3(kQThreads), 0, s, A);
      else
        hipLaunchKernelGGL((assign_q8_kernel<KM_SQ8, true, 4>), grid, dim3(kQThreads), 0, s, A);
    }
  } else {  // bfloat16 rows as bytes
    A.pi8 = static_cast<const uint8_t *>(P.data);
    A.pild = 2 * P.ld;
    A.ci8 = reinterpret_cast<const int8_t *>(cp.cb);
    A.cild = 2 * (int64_t)P.d;
    A.di = 2 * P.d;
    if (tile_c == 128)
      hipLaunchKernelGGL((assign_q8_kernel<KM_BF16, true, 2>), dim3((unsigned)ntiles), dim3(kQThreads), 0, s, A);
    else
      hipLaunchKernelGGL((assign_q8_kernel<KM_BF16, true, 2, false, 4>), dim3((unsigned)ntiles), dim3(kQWideThreads), 0,
                         s, A);
  }
  KMQ_LAUNCH_CHECK("assign kernel (segments)");
  return KM_OK;
}

CentroidPrep prep_slice(const Points &P, const CentroidPrep &cp, int off, int64_t pstart) {
  CentroidPrep r = cp;
  r.cn = cp.cn + off;
  r.qsum = cp.qsum + off;
  r.u = cp.u + off;
  r.sig2 = cp.sig2 + off;
  const int d0 = P.fmt == KM_HYBRID ? P.d_front : 0;
  if (is_bits_fmt(P.fmt)) r.q = cp.q + (int64_t)off * (P.d - d0);
  if (P.fmt == KM_LVQ4 || P.fmt == KM_SQ8) r.q = cp.q + (int64_t)off * P.d;
  if (P.fmt == KM_BF16) {
    r.cb = cp.cb + (int64_t)off * P.d;
    r.q = reinterpret_cast<const int8_t *>(r.cb);
  }
  if (cp.keys) r.keys = cp.keys + pstart;
  return r;
}

km_status launch_xconst(const Points &P, float *xc, hipStream_t s) {
  const dim3 g((unsigned)cdiv(P.n, 4));
  switch (P.fmt) {
    case KM_F32: hipLaunchKernelGGL(xconst_kernel<KM_F32>, g, dim3(256), 0, s, P, xc); break;
    case KM_BF16: hipLaunchKernelGGL(xconst_kernel<KM_BF16>, g, dim3(256), 0, s, P, xc); break;
    case KM_SQ8: hipLaunchKernelGGL(xconst_kernel<KM_SQ8>, g, dim3(256), 0, s, P, xc); break;
    case KM_SIGN1: hipLaunchKernelGGL(xconst_kernel<KM_SIGN1>, g, dim3(256), 0, s, P, xc); break;
    case KM_HYBRID: hipLaunchKernelGGL(xconst_kernel<KM_HYBRID>, g, dim3(256), 0, s, P, xc); break;
    case KM_RABITQ: hipLaunchKernelGGL(xconst_kernel<KM_RABITQ>, g, dim3(256), 0, s, P, xc); break;
    case KM_LVQ4: hipLaunchKernelGGL(xconst_kernel<KM_LVQ4>, g, dim3(256), 0, s, P, xc); break;
    default: return KM_EUNSUPPORTED;
  }
  KMQ_LAUNCH_CHECK("xconst_kernel");
  return KM_OK;
}

int objective_blocks(int64_t n) { return (int)std::min<int64_t>(kObjBlocks, std::max<int64_t>(1, cdiv(n, 256))); }

km_status launch_objective(const Points &P, const float *xc, const float *score, int64_t n, double *out,
                           double *partials, int nblk_max, hipStream_t s) {
  (void)P;
  const int nb = std::min(nblk_max, objective_blocks(n));
  hipLaunchKernelGGL(objective_partial_kernel, dim3(nb), dim3(256), 0, s, xc, score, n, partials);
  hipLaunchKernelGGL(sum_partials_kernel, dim3(1), dim3(256), 0, s, partials, nb, out);
  KMQ_LAUNCH_CHECK("objective");
  return KM_OK;
}

km_status launch_gather_init(const Points &P, const int64_t *idx, int k, void *C, hipStream_t s) {
  switch (P.fmt) {
    case KM_F32: hipLaunchKernelGGL(gather_kernel<KM_F32>, dim3(k), dim3(256), 0, s, P, idx, C); break;
    case KM_BF16: hipLaunchKernelGGL(gather_kernel<KM_BF16>, dim3(k), dim3(256), 0, s, P, idx, C); break;
    case KM_SQ8: hipLaunchKernelGGL(gather_kernel<KM_SQ8>, dim3(k), dim3(256), 0, s, P, idx, C); break;
    case KM_SIGN1: hipLaunchKernelGGL(gather_kernel<KM_SIGN1>, dim3(k), dim3(256), 0, s, P, idx, C); break;
    case KM_HYBRID: hipLaunchKernelGGL(gather_kernel<KM_HYBRID>, dim3(k), dim3(256), 0, s, P, idx, C); break;
    case KM_RABITQ: hipLaunchKernelGGL(gather_kernel<KM_RABITQ>, dim3(k), dim3(256), 0, s, P, idx, C); break;
    case KM_LVQ4: hipLaunchKernelGGL(gather_kernel<KM_LVQ4>, dim3(k), dim3(256), 0, s, P, idx, C); break;
    default: return KM_EUNSUPPORTED;
  }
  KMQ_LAUNCH_CHECK("gather_kernel");
  return KM_OK;
}

km_status launch_cost(const float *X, int64_t n, int d, int64_t ldx, const float *C, int k, const int32_t *assign,
                      double *out, double *partials, hipStream_t s) {
  const int nb = (int)std::min<int64_t>(kObjBlocks, std::max<int64_t>(1, cdiv(n, 4)));
  hipLaunchKernelGGL(cost_kernel, dim3(nb), dim3(256), 0, s, X, n, d, ldx, C, k, assign, partials);
  hipLaunchKernelGGL(sum_partials_kernel, dim3(1), dim3(256), 0, s, partials, nb, out);
  KMQ_LAUNCH_CHECK("cost_kernel");
  return KM_OK;
}

}  // namespace kmq
