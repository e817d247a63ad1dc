// STEP 3 (Sec. 2.3): centroid update as a deterministic segmented sum.
//
//   1. hist     per block of points (about 1024 blocks), member counts of every cluster
//               (LDS-privatised histogram), stored cluster-major [k][nblk].
//   2. scan     exclusive scan of that table (block sums, then each block's
//               scan plus the sum of the blocks before it): entry (j, b) is where
//               block b's first member of cluster j goes in the cluster-sorted
//               order; one workgroup then derives every cluster's count, start
//               and chunk offset.
//   3. scatter  stable counting sort: points are ranked inside each wave among
//               the lanes with the same cluster id (found with one ballot per
//               id bit) and the four waves take their slots in order, so
//               members stay in point order.
//   4. segsum   fixed-size chunks (<= 512 members, never crossing a cluster)
//               are summed by one workgroup per (chunk, column slice): each
//               wave adds every 4th member's slice of the row (coalesced
//               1 KiB reads of fp32 rows, 256 B of codes, 128 B of bits); the
//               four wave sums are combined in LDS in a fixed order.
//               1-bit members are decoded on the fly: alpha_x (2b - 1) (fused
//               decode-averaging, Sec. 3.1 RabitQ); SQ8 codes are summed as
//               exact integers (averaging in the quantised domain, Sec. 3.1).
//   5. finalize per cluster, chunk sums in chunk order in fp64, divided by
//               the count: fp32 mean / 1-bit residual mean / rounded code mean.
//   6. split    empty clusters in ascending order take a split of the cluster
//               with the largest current count (one workgroup, sequential);
//               with segments given (hierarchical fine phase), the donor is
//               searched among the empty cluster's own segment of centroids.
//   7. compose  write the new centroids (1-bit dims: m + residual).
// Every sum has a fixed order, so results are bit-identical run to run.
#include <algorithm>

#include "common.hpp"

namespace kmq {
namespace {

constexpr int kHistBlocks = 512;   // target number of histogram / scatter blocks
constexpr int kChunk = 512;        // members per segmented-sum chunk
constexpr int kLdsCursorMax = 16384;
constexpr int kScanSeg = 4096;     // elements per scan block (256 threads x 16)

struct UpdWs {
  int ppb;       // points per histogram / scatter block (multiple of 256)
  int nblk;      // histogram blocks
  int64_t L;     // k * nblk
  int nsb;       // scan blocks
  int maxchunks;
  int dp;        // row length of partial sums / Z (F32: d, SQ8: d, SIGN1/HYBRID: d)
  int *offs;     // [L]
  int *bsum;     // [nsb + 1]
  int *total;    // [4]
  int *cnt;      // [k]
  int *cstart;   // [k]
  int *choff;    // [k + 1]
  int *perm;     // [n]
  void *partial; // [maxchunks * dp] float or int
  uint32_t *partialA; // [maxchunks] 1-bit formats: sum of the scaled alphas per chunk
  float *partialM;    // [maxchunks] 1-bit formats: largest alpha per chunk; LVQ4: largest scale
  double *partialB;   // [maxchunks] LVQ4: sum of the biases per chunk
  void *Z;       // [k * dp] float or uint8
  uint8_t *fresh;  // [k]
  int64_t *cntw;   // [k]
  int *empties;    // [k]
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

UpdWs carve(const Points &P, int k, void *base, size_t *bytes_out) {
  UpdWs w{};
  w.ppb = (int)std::max<int64_t>(256, cdiv(cdiv(P.n, kHistBlocks), 256) * 256);
  w.nblk = (int)cdiv(P.n, w.ppb);
  w.L = (int64_t)k * w.nblk;
  w.nsb = (int)cdiv(w.L, kScanSeg);
  w.maxchunks = (int)(cdiv(P.n, kChunk) + k);
  w.dp = P.d;
  uint8_t *b = static_cast<uint8_t *>(base);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    void *p = b ? b + o : nullptr;
    o += align256(bytes);
    return p;
  };
  w.offs = (int *)take(sizeof(int) * (size_t)w.L);
  w.bsum = (int *)take(sizeof(int) * (size_t)(w.nsb + 1));
  w.total = (int *)take(sizeof(int) * 4);
  w.cnt = (int *)take(sizeof(int) * (size_t)k);
  w.cstart = (int *)take(sizeof(int) * (size_t)k);
  w.choff = (int *)take(sizeof(int) * (size_t)(k + 1));
  w.perm = (int *)take(sizeof(int) * (size_t)P.n);
  w.partial = take(sizeof(float) * (size_t)w.maxchunks * (size_t)w.dp);
  w.partialA = (uint32_t *)take(sizeof(uint32_t) * (size_t)w.maxchunks);
  w.partialM = (float *)take(sizeof(float) * (size_t)w.maxchunks);
  w.partialB = (double *)take(sizeof(double) * (size_t)w.maxchunks);
  w.Z = take(sizeof(float) * (size_t)k * (size_t)w.dp);
  w.fresh = (uint8_t *)take((size_t)k);
  w.cntw = (int64_t *)take(sizeof(int64_t) * (size_t)k);
  w.empties = (int *)take(sizeof(int) * (size_t)k);
  if (bytes_out) *bytes_out = o;
  return w;
}

// ---- 1. histogram ------------------------------------------------------------
__global__ __launch_bounds__(256) void hist_kernel(const int32_t *assign, int64_t n, int k, int nblk, int ppb,
                                                   int *offs, int use_lds) {
  extern __shared__ int lc[];
  const int b = blockIdx.x, t = threadIdx.x;
  const int64_t lo = (int64_t)b * ppb;
  const int64_t hi = min<int64_t>(n, lo + ppb);
  if (use_lds) {
    for (int j = t; j < k; j += 256) lc[j] = 0;
    __syncthreads();
    for (int64_t p = lo + t; p < hi; p += 256) {
      const int a = assign[p];
      if (a >= 0 && a < k) atomicAdd(&lc[a], 1);
    }
    __syncthreads();
    for (int j = t; j < k; j += 256) offs[(int64_t)j * nblk + b] = lc[j];
  } else {
    for (int64_t p = lo + t; p < hi; p += 256) {
      const int a = assign[p];
      if (a >= 0 && a < k) atomicAdd(&offs[(int64_t)a * nblk + b], 1);
    }
  }
}

__global__ void fill_int_kernel(int *p, int64_t n, int v) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = v;
}

// ---- 2. scan -----------------------------------------------------------------
__device__ __forceinline__ int block_excl_scan_int(int v, int *sh, int *total) {
  // Hillis-Steele inclusive scan over 256 thread values, returned exclusive.
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    int add = t >= off ? sh[t - off] : 0;
    __syncthreads();
    sh[t] += add;
    __syncthreads();
  }
  const int incl = sh[t];
  if (total) *total = sh[255];
  __syncthreads();
  return incl - v;
}

__global__ __launch_bounds__(256) void scan_reduce_kernel(const int *x, int64_t L, int *bsum) {
  __shared__ int sh[256];
  const int64_t base = (int64_t)blockIdx.x * kScanSeg;
  int s = 0;
  for (int i = threadIdx.x; i < kScanSeg; i += 256) {
    const int64_t g = base + i;
    if (g < L) s += x[g];
  }
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (threadIdx.x < st) sh[threadIdx.x] += sh[threadIdx.x + st];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = sh[0];
}

// Exclusive scan of block b's segment plus the sum of the segments before it, which
// the block adds up itself from the segment sums (a few thousand at most); the last
// block also writes the grand total.
__global__ __launch_bounds__(256) void scan_down_kernel(int *x, int64_t L, const int *bsum, int *total) {
  __shared__ int sh[256];
  __shared__ int pre[4];
  const int b = blockIdx.x, t = threadIdx.x;
  int ps = 0;
  for (int i = t; i < b; i += 256) ps += bsum[i];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ps += __shfl_xor(ps, o);
  if ((t & 63) == 0) pre[t >> 6] = ps;
  const int64_t base = (int64_t)b * kScanSeg + (int64_t)t * 16;
  int v[16];
  int s = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    v[e] = base + e < L ? x[base + e] : 0;
    s += v[e];
  }
  int tot;
  int run = block_excl_scan_int(s, sh, &tot);  // its barriers also publish pre[]
  const int prefix = pre[0] + pre[1] + pre[2] + pre[3];
  run += prefix;
  if (t == 0 && b == gridDim.x - 1) *total = prefix + tot;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    if (base + e < L) x[base + e] = run;
    run += v[e];
  }
}

// counts and start offsets of each cluster from the scanned table, and the exclusive
// scan of their chunk counts ceil(cnt / kChunk) (one workgroup; choff[k] = all chunks)
__global__ __launch_bounds__(256) void counts_kernel(const int *offs, int nblk, int k, const int *total, int *cnt,
                                                     int *cstart, int *choff) {
  __shared__ int sh[256];
  const int t = threadIdx.x;
  const int per = (k + 255) / 256;
  const int lo = min(k, t * per), hi = min(k, lo + per);
  int sum = 0;
  for (int j = lo; j < hi; ++j) {
    const int s0 = offs[(int64_t)j * nblk];
    const int e0 = j + 1 < k ? offs[(int64_t)(j + 1) * nblk] : total[0];
    cnt[j] = e0 - s0;
    cstart[j] = s0;
    sum += (e0 - s0 + kChunk - 1) / kChunk;
  }
  int tot;
  int run = block_excl_scan_int(sum, sh, &tot);
  for (int j = lo; j < hi; ++j) {
    choff[j] = run;
    run += (cnt[j] + kChunk - 1) / kChunk;
  }
  if (t == 0) choff[k] = tot;
}

// ---- 3. stable scatter -------------------------------------------------------
__global__ __launch_bounds__(256) void scatter_kernel(const int32_t *assign, int64_t n, int k, int nblk, int ppb,
                                                      int *offs, int use_lds, int *perm) {
  extern __shared__ int cur[];
  const int b = blockIdx.x, t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int64_t lo = (int64_t)b * ppb;
  const int64_t hi = min<int64_t>(n, lo + ppb);
  if (use_lds) {
    for (int j = t; j < k; j += 256) cur[j] = offs[(int64_t)j * nblk + b];
    __syncthreads();
  }
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int nbits = k > 1 ? 32 - __clz(k - 1) : 0;  // bits of a cluster id
  for (int64_t base = lo; base < hi; base += 256) {
    const int64_t p = base + t;
    int a = p < hi ? assign[p] : -1;
    const bool valid = a >= 0 && a < k;
    // lanes holding the same id: one ballot per id bit; then the rank among them
    // (lanes below), their number and their first lane
    uint64_t peers = __ballot(valid);
    for (int ib = 0; ib < nbits; ++ib) {
      const bool bit = (a >> ib) & 1;
      const uint64_t ones = __ballot(valid && bit);
      peers &= bit ? ones : ~ones;
    }
    int rank = 0, cnt = 0, leader = 0;
    if (valid) {
      rank = __popcll(peers & lt_mask);
      cnt = __popcll(peers);
      leader = __ffsll((unsigned long long)peers) - 1;
    }
    for (int w = 0; w < 4; ++w) {
      __syncthreads();
      if (wave == w) {
        int old = 0;
        if (valid && lane == leader) {
          old = use_lds ? atomicAdd(&cur[a], cnt) : atomicAdd(&offs[(int64_t)a * nblk + b], cnt);
        }
        const int basepos = __shfl(old, leader);
        if (valid) perm[basepos + rank] = (int)p;
      }
    }
  }
}

// ---- 4. chunked segmented sums ----------------------------------------------
__device__ __forceinline__ int find_cluster(const int *choff, int k, int c) {
  // largest j with choff[j] <= c (clusters with no chunks have equal neighbours)
  int lo = 0, hi = k;  // invariant: choff[lo] <= c < choff[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (choff[mid] <= c) lo = mid; else hi = mid;
  }
  return lo;
}

// fp32 rows: one slice of 256 columns per workgroup
__global__ __launch_bounds__(256) void segsum_f32_kernel(const float *X, int64_t ld, int df, const int *perm,
                                                         const int *cnt, const int *cstart, const int *choff, int k,
                                                         float *partial, int dp) {
  __shared__ f32x4 red[4][64];
  const int c = blockIdx.x;
  if (c >= choff[k]) return;
  const int j = find_cluster(choff, k, c);
  const int ci = c - choff[j];
  const int m0 = cstart[j] + ci * kChunk;
  const int m1 = cstart[j] + min(cnt[j], (ci + 1) * kChunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.y * 256 + 4 * lane;
  const bool ok = col < df;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  int m = m0 + wave;
  for (; m + 28 < m1; m += 32) {
    int pp[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pp[e] = perm[m + 4 * e];
    if (ok) {
      f32x4 v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const f32x4 *>(X + (int64_t)pp[e] * ld + col);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc += v[e];
    }
  }
  for (; m < m1; m += 4) {
    const int p = perm[m];
    if (ok) acc += *reinterpret_cast<const f32x4 *>(X + (int64_t)p * ld + col);
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && ok) {
    f32x4 s = red[0][lane];
    s += red[1][lane];
    s += red[2][lane];
    s += red[3][lane];
    *reinterpret_cast<f32x4 *>(partial + (int64_t)c * dp + col) = s;
  }
}

// bfloat16 rows: one slice of 512 columns per workgroup; lane = 8 values (16 bytes),
// decoded to fp32 and summed in fp32 within a chunk (as for fp32 rows)
__global__ __launch_bounds__(256) void segsum_bf16_kernel(const uint16_t *X, int64_t ld, int d, const int *perm,
                                                          const int *cnt, const int *cstart, const int *choff, int k,
                                                          float *partial, int dp) {
  __shared__ f32x4 red[4][2][64];
  const int c = blockIdx.x;
  if (c >= choff[k]) return;
  const int j = find_cluster(choff, k, c);
  const int ci = c - choff[j];
  const int m0 = cstart[j] + ci * kChunk;
  const int m1 = cstart[j] + min(cnt[j], (ci + 1) * kChunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.y * 512 + 8 * lane;
  const bool ok = col < d;
  f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
  auto add = [&](uint4 w) {
    lo += f32x4{bf16_value(w.x & 0xffffu), bf16_value(w.x >> 16), bf16_value(w.y & 0xffffu), bf16_value(w.y >> 16)};
    hi += f32x4{bf16_value(w.z & 0xffffu), bf16_value(w.z >> 16), bf16_value(w.w & 0xffffu), bf16_value(w.w >> 16)};
  };
  int m = m0 + wave;
  for (; m + 28 < m1; m += 32) {
    int pp[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pp[e] = perm[m + 4 * e];
    if (ok) {
      uint4 v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const uint4 *>(X + (int64_t)pp[e] * ld + col);
#pragma unroll
      for (int e = 0; e < 8; ++e) add(v[e]);
    }
  }
  for (; m < m1; m += 4) {
    const int p = perm[m];
    if (ok) add(*reinterpret_cast<const uint4 *>(X + (int64_t)p * ld + col));
  }
  red[wave][0][lane] = lo;
  red[wave][1][lane] = hi;
  __syncthreads();
  if (wave == 0 && ok) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      f32x4 t = red[0][hh][lane];
      t += red[1][hh][lane];
      t += red[2][hh][lane];
      t += red[3][hh][lane];
      *reinterpret_cast<f32x4 *>(partial + (int64_t)c * dp + col + 4 * hh) = t;
    }
  }
}

// 1-bit rows: one slice of 1024 tail dims per workgroup; lane = 16 dims (half a
// word).  Only W = sum of alpha over the members whose bit is set is accumulated
// per dim (finalize forms the mean decoded residual (2W - A)/n with A = sum of
// alpha), and in exact integers: the chunk's alphas are first scaled to 23-bit
// integers q = rint(alpha / s), s = (largest alpha of the chunk) / (2^23 - 1), so
// one member costs a bit extract and a 24-bit multiply-add per dim, and every sum
// is exact (at most 128 members per lane: < 2^30; four waves: < 2^32).
constexpr double kAlphaSteps = 8388607.0;  // 2^23 - 1

// d = a * b + c on the low 24 bits of a and b (one vector instruction; it writes
// no scalar register, flag or mask)
__device__ __forceinline__ uint32_t mad_u24(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t d;
  asm("v_mad_u32_u24 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
  return d;
}

__global__ __launch_bounds__(256) void segsum_bits_kernel(const uint32_t *bits, int64_t wpr, int w0, int dt,
                                                          const float *alpha, const int *perm, const int *cnt,
                                                          const int *cstart, const int *choff, int k,
                                                          uint32_t *partial, uint32_t *partialA, float *partialM,
                                                          int dp, int coff) {
  __shared__ int sperm[kChunk];
  __shared__ uint32_t sq[kChunk];
  __shared__ uint32_t red[4][64 * 17];
  __shared__ float smax[4];
  __shared__ uint32_t ssum[4];
  const int c = blockIdx.x;
  if (c >= choff[k]) return;
  const int j = find_cluster(choff, k, c);
  const int ci = c - choff[j];
  const int m0 = cstart[j] + ci * kChunk;
  const int len = min(cnt[j], (ci + 1) * kChunk) - ci * kChunk;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  // the chunk's member ids and alphas (two per thread), and its largest alpha
  float av[2] = {0.f, 0.f};
  float mx = 0.f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = t + 256 * h;
    if (i < len) {
      const int p = perm[m0 + i];
      sperm[i] = p;
      av[h] = alpha[p];
      mx = fmaxf(mx, av[h]);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if (lane == 0) smax[wave] = mx;
  __syncthreads();
  const float amax = fmaxf(fmaxf(smax[0], smax[1]), fmaxf(smax[2], smax[3]));
  const double inv_s = amax > 0.f ? kAlphaSteps / (double)amax : 0.0;
  uint32_t qs = 0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = t + 256 * h;
    if (i < len) {
      const uint32_t q = (uint32_t)rint((double)av[h] * inv_s);
      sq[i] = q;
      qs += q;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) qs += __shfl_xor(qs, o);
  if (lane == 0) ssum[wave] = qs;
  __syncthreads();
  if (t == 0 && blockIdx.y == 0) {
    partialA[c] = ssum[0] + ssum[1] + ssum[2] + ssum[3];  // < 512 (2^23 - 1) < 2^32
    partialM[c] = amax;
  }
  const int hw = blockIdx.y * 64 + lane;  // half-word index within the tail
  const bool ok = 16 * hw < dt;
  const int wo = w0 + ((ok ? hw : 0) >> 1);  // clamped: every load is valid
  const int sh = 16 * (hw & 1);
  uint32_t acc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0u;
  auto add = [&](uint32_t q, uint32_t w) {
    const uint32_t hb = ok ? (w >> sh) : 0u;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = mad_u24(__builtin_amdgcn_ubfe(hb, e, 1), q, acc[e]);
  };
  // 8 members in flight per wave (their loads issued together); each lane adds
  // the members m, m + 4, m + 8, ... of the chunk
  int m = wave;
  for (; m + 28 < len; m += 32) {
    uint32_t qq[8], ww[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      qq[e] = sq[m + 4 * e];
      ww[e] = bits[(int64_t)sperm[m + 4 * e] * wpr + wo];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) add(qq[e], ww[e]);
  }
  for (; m < len; m += 4) add(sq[m], bits[(int64_t)sperm[m] * wpr + wo]);
#pragma unroll
  for (int e = 0; e < 16; ++e) red[wave][lane * 17 + e] = acc[e];
  __syncthreads();
  if (wave == 0 && ok) {
    uint32_t *out = partial + (int64_t)c * dp + coff + 16 * hw;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      out[e] = red[0][lane * 17 + e] + red[1][lane * 17 + e] + red[2][lane * 17 + e] + red[3][lane * 17 + e];
  }
}

// LVQ4 rows: one slice of 1024 dims (512 packed bytes) per workgroup; lane = 16
// dims from 8 packed bytes.  A member decodes to s x + b per dim (x its 4-bit
// code); the bias part is summed once per member (B = sum of b, in fp64) and the
// scaled codes in exact integers, as for the 1-bit rows: the chunk's scales become
// 19-bit integers q = rint(s / u), u = (largest scale of the chunk) / (2^19 - 1), so
// a dim costs a bit-field extract and a 24-bit multiply-add, and no sum can wrap
// (at most 512 members: 512 * 15 * (2^19 - 1) < 2^32).  The fold forms
// sum over chunks of u W + B in fp64.
constexpr double kLvqSteps = 524287.0;  // 2^19 - 1

__global__ __launch_bounds__(256) void segsum_lvq4_kernel(const uint8_t *codes, int64_t ld, const float *vparams,
                                                          int d, const int *perm, const int *cnt, const int *cstart,
                                                          const int *choff, int k, uint32_t *partial, float *partialM,
                                                          double *partialB, int dp) {
  __shared__ int sperm[kChunk];
  __shared__ uint32_t sq[kChunk];
  __shared__ uint32_t red[4][64 * 17];
  __shared__ float smax[4];
  __shared__ double sbias[4];
  const int c = blockIdx.x;
  if (c >= choff[k]) return;
  const int j = find_cluster(choff, k, c);
  const int ci = c - choff[j];
  const int m0 = cstart[j] + ci * kChunk;
  const int len = min(cnt[j], (ci + 1) * kChunk) - ci * kChunk;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  // the chunk's member ids and scales (two per thread), its largest scale and its
  // bias sum (fixed-order reductions)
  float sv[2] = {0.f, 0.f};
  float mx = 0.f;
  double bs = 0.0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = t + 256 * h;
    if (i < len) {
      const int p = perm[m0 + i];
      sperm[i] = p;
      const float2 sb = *reinterpret_cast<const float2 *>(vparams + 4 * (int64_t)p);
      sv[h] = sb.x;
      mx = fmaxf(mx, sb.x);
      bs += (double)sb.y;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o));
    bs += __shfl_xor(bs, o);
  }
  if (lane == 0) {
    smax[wave] = mx;
    sbias[wave] = bs;
  }
  __syncthreads();
  const float smx = fmaxf(fmaxf(smax[0], smax[1]), fmaxf(smax[2], smax[3]));
  const double inv_u = smx > 0.f ? kLvqSteps / (double)smx : 0.0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = t + 256 * h;
    if (i < len) sq[i] = (uint32_t)rint((double)sv[h] * inv_u);
  }
  if (t == 0 && blockIdx.y == 0) {
    partialM[c] = smx;
    partialB[c] = ((sbias[0] + sbias[1]) + sbias[2]) + sbias[3];
  }
  __syncthreads();
  const int col = blockIdx.y * 1024 + 16 * lane;
  const bool ok = col < d;  // d % 32 == 0: 16 dims are wholly in or out
  const int bo = (ok ? col : 0) / 2;
  uint32_t acc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0u;
  // nibble 2e of the lane's 8 bytes is dim col + 2e (low nibble first)
  auto add = [&](uint32_t q, uint2 w) {
#pragma unroll
    for (int e = 0; e < 16; ++e)
      acc[e] = mad_u24(__builtin_amdgcn_ubfe(e < 8 ? w.x : w.y, 4 * (e & 7), 4), q, acc[e]);
  };
  // lane adds the members m, m + 4, m + 8, ... of the chunk, 8 at a time, with the
  // next 8 rows' loads in flight while the current ones are added (the last
  // round's look-ahead rereads the chunk's last row and is not used)
  uint32_t qq[8];
  uint2 ww[8];
  auto fetch = [&](int mb) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = min(mb + 4 * e, len - 1);
      qq[e] = sq[i];
      ww[e] = *reinterpret_cast<const uint2 *>(codes + (int64_t)sperm[i] * ld + bo);
    }
  };
  const int rounds = len - 28 > wave ? (len - 28 - wave + 31) / 32 : 0;  // m + 28 < len
  if (rounds > 0) fetch(wave);
  for (int r = 0; r < rounds; ++r) {
    uint32_t q0[8];
    uint2 w0[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      q0[e] = qq[e];
      w0[e] = ww[e];
    }
    fetch(wave + 32 * (r + 1));
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int e = 0; e < 8; ++e) add(q0[e], w0[e]);
  }
  for (int m = wave + 32 * rounds; m < len; m += 4)
    add(sq[m], *reinterpret_cast<const uint2 *>(codes + (int64_t)sperm[m] * ld + bo));
#pragma unroll
  for (int e = 0; e < 16; ++e) red[wave][lane * 17 + e] = acc[e];
  __syncthreads();
  if (wave == 0 && ok) {
    uint32_t *out = partial + (int64_t)c * dp + col;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      out[e] = red[0][lane * 17 + e] + red[1][lane * 17 + e] + red[2][lane * 17 + e] + red[3][lane * 17 + e];
  }
}

// SQ8 codes: one slice of 1024 bytes (16 per lane) per workgroup, exact int32 sums
__global__ __launch_bounds__(256) void segsum_sq8_kernel(const uint8_t *codes, int64_t ld, int d, const int *perm,
                                                         const int *cnt, const int *cstart, const int *choff, int k,
                                                         int *partial) {
  __shared__ int red[4][64 * 17];
  const int c = blockIdx.x;
  if (c >= choff[k]) return;
  const int j = find_cluster(choff, k, c);
  const int ci = c - choff[j];
  const int m0 = cstart[j] + ci * kChunk;
  const int m1 = cstart[j] + min(cnt[j], (ci + 1) * kChunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.y * 1024 + 16 * lane;
  const bool ok = col < d;
  int acc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0;
  int m = m0 + wave;
  for (; m + 28 < m1; m += 32) {
    int pp[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pp[e] = perm[m + 4 * e];
    if (ok) {
      uint4 v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const uint4 *>(codes + (int64_t)pp[e] * ld + col);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t ws[4] = {v[e].x, v[e].y, v[e].z, v[e].w};
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[4 * q + b] += (int)((ws[q] >> (8 * b)) & 255u);
      }
    }
  }
  for (; m < m1; m += 4) {
    const int p = perm[m];
    if (ok) {
      const uint4 v = *reinterpret_cast<const uint4 *>(codes + (int64_t)p * ld + col);
      const uint32_t ws[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[4 * q + b] += (int)((ws[q] >> (8 * b)) & 255u);
    }
  }
#pragma unroll
  for (int e = 0; e < 16; ++e) red[wave][lane * 17 + e] = acc[e];
  __syncthreads();
  if (wave == 0 && ok) {
#pragma unroll
    for (int e = 0; e < 16; ++e)
      partial[(int64_t)c * d + col + e] =
          red[0][lane * 17 + e] + red[1][lane * 17 + e] + red[2][lane * 17 + e] + red[3][lane * 17 + e];
  }
}

// ---- 5. finalize (and compose) ---------------------------------------------------
// The new centroid in the original space from its clustering-space value z: on the
// 1-bit dims (col >= d_bits of a 1-bit format) m + z, the centre m being NULL (0)
// for RabitQ's residual space; elsewhere z.
struct Compose {
  float *C;
  const float *m;
  int d_bits;
  int bits;
  int64_t *counts;
  __device__ float operator()(int col, float z) const {
    return bits && col >= d_bits ? (m ? m[col] : 0.0f) + z : z;
  }
};

// Columns from d_bits on hold, per chunk, W as an exact integer sum of the scaled
// alphas q over the set bits; partialA the chunk's sum of q and partialM its
// largest alpha, which fixes the scale s = partialM / (2^23 - 1).  The mean decoded
// residual is (2W - A)/n with W and A scaled back by each chunk's s.  LVQ4
// (partialB set): W is the chunk's exact sum of its scaled scales times the codes,
// partialM its largest scale and partialB its bias sum; the mean is the sum over
// chunks of (partialM / (2^19 - 1)) W + partialB, over n.
__global__ __launch_bounds__(256) void finalize_f32_kernel(const float *partial, int dp, const int *cnt,
                                                           const int *choff, float *Z, uint8_t *fresh,
                                                           const uint32_t *partialA, const float *partialM,
                                                           const double *partialB, int d_bits, Compose cm) {
  const int j = blockIdx.x;
  const int col = blockIdx.y * 256 + threadIdx.x;
  const int nj = cnt[j];
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    fresh[j] = nj > 0;
    if (cm.counts) cm.counts[j] = nj;
  }
  if (nj == 0 || col >= dp) return;
  double s = 0.0;
  if (partialA && col >= d_bits) {
    const uint32_t *pu = reinterpret_cast<const uint32_t *>(partial);
    double a = 0.0;
    for (int c = choff[j]; c < choff[j + 1]; ++c) {
      const double sc = (double)partialM[c] / kAlphaSteps;
      s += sc * (double)pu[(int64_t)c * dp + col];
      a += sc * (double)partialA[c];
    }
    s = 2.0 * s - a;
  } else if (partialB) {
    const uint32_t *pu = reinterpret_cast<const uint32_t *>(partial);
    for (int c = choff[j]; c < choff[j + 1]; ++c)
      s += (double)partialM[c] / kLvqSteps * (double)pu[(int64_t)c * dp + col] + partialB[c];
  } else {
    for (int c = choff[j]; c < choff[j + 1]; ++c) s += (double)partial[(int64_t)c * dp + col];
  }
  const float z = (float)(s / (double)nj);
  Z[(int64_t)j * dp + col] = z;
  cm.C[(int64_t)j * dp + col] = cm(col, z);
}

__global__ __launch_bounds__(256) void finalize_sq8_kernel(const int *partial, int d, const int *cnt,
                                                           const int *choff, uint8_t *Z, uint8_t *fresh, uint8_t *C,
                                                           int64_t *counts) {
  const int j = blockIdx.x;
  const int col = blockIdx.y * 256 + threadIdx.x;
  const int nj = cnt[j];
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    fresh[j] = nj > 0;
    if (counts) counts[j] = nj;
  }
  if (nj == 0 || col >= d) return;
  int64_t S = 0;
  for (int c = choff[j]; c < choff[j + 1]; ++c) S += partial[(int64_t)c * d + col];
  // mean of the codes rounded half up: floor((2S + n) / (2n))
  const uint8_t z = (uint8_t)((2 * S + nj) / (2 * (int64_t)nj));
  Z[(int64_t)j * d + col] = z;
  C[(int64_t)j * d + col] = z;
}

// ---- 6. empty-cluster split (one workgroup) -----------------------------------
// The empty clusters are first listed in ascending order (block scan over the
// counts); the split itself is inherently sequential (each donor choice sees the
// counts left by the previous split) and runs over that list only.
template <bool CODES>
__global__ __launch_bounds__(256) void split_kernel(void *Zv, int k, int dp, const int *cnt, int64_t *cntw,
                                                    uint8_t *fresh, int *empties, const int *seg_lo,
                                                    const int *seg_hi, Compose cm) {
  __shared__ int64_t sv[256];
  __shared__ int si[256];
  __shared__ int shs[256];
  __shared__ int n_empty;
  const int t = threadIdx.x;
  const int per = (k + 255) / 256;
  const int lo = min(k, t * per), hi = min(k, lo + per);
  int mine = 0;
  for (int j = lo; j < hi; ++j) mine += cnt[j] == 0;
  int tot;
  int pos = block_excl_scan_int(mine, shs, &tot);
  for (int j = lo; j < hi; ++j)
    if (cnt[j] == 0) empties[pos++] = j;
  if (t == 0) n_empty = tot;
  __syncthreads();
  const int ne = n_empty;
  if (ne == 0) return;
  for (int j = t; j < k; j += 256) cntw[j] = cnt[j];
  __syncthreads();
  const float up = 1.0f + 0x1p-10f, dn = 1.0f - 0x1p-10f;
  for (int e = 0; e < ne; ++e) {
    const int j = empties[e];
    const int slo = seg_lo ? seg_lo[j] : 0, shi = seg_hi ? seg_hi[j] : k;  // donor candidates
    int64_t bv = -1;
    int bi = slo;
    for (int i = slo + t; i < shi; i += 256) {
      const int64_t v = cntw[i];
      if (v > bv) {
        bv = v;
        bi = i;
      }
    }
    sv[t] = bv;
    si[t] = bi;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (t < st) {
        const int64_t ov = sv[t + st];
        const int oi = si[t + st];
        if (ov > sv[t] || (ov == sv[t] && oi < si[t])) {
          sv[t] = ov;
          si[t] = oi;
        }
      }
      __syncthreads();
    }
    const int b = si[0];
    const int64_t nb = sv[0];
    __syncthreads();
    if (nb < 2) continue;  // uniform
    // the two rows change in Z and, composed, in C (finalize composed the others)
    if (CODES) {
      uint8_t *Z = static_cast<uint8_t *>(Zv);
      uint8_t *C = reinterpret_cast<uint8_t *>(cm.C);
      for (int i = t; i < dp; i += 256) {
        const int v = Z[(int64_t)b * dp + i];
        const int p = (i & 1) ? -1 : 1;
        const uint8_t zj = (uint8_t)min(255, max(0, v + p)), zb = (uint8_t)min(255, max(0, v - p));
        Z[(int64_t)j * dp + i] = zj;
        Z[(int64_t)b * dp + i] = zb;
        C[(int64_t)j * dp + i] = zj;
        C[(int64_t)b * dp + i] = zb;
      }
    } else {
      float *Z = static_cast<float *>(Zv);
      for (int i = t; i < dp; i += 256) {
        const float v = Z[(int64_t)b * dp + i];
        const bool even = (i & 1) == 0;
        const float zj = v * (even ? up : dn), zb = v * (even ? dn : up);
        Z[(int64_t)j * dp + i] = zj;
        Z[(int64_t)b * dp + i] = zb;
        cm.C[(int64_t)j * dp + i] = cm(i, zj);
        cm.C[(int64_t)b * dp + i] = cm(i, zb);
      }
    }
    __syncthreads();
    if (t == 0) {
      const int64_t half = nb / 2;
      cntw[j] = half;
      cntw[b] = nb - half;
      fresh[j] = 1;
    }
    __syncthreads();
  }
}

}  // namespace

size_t update_bytes(const Points &P, int k) {
  size_t b = 0;
  carve(P, k, nullptr, &b);
  return b;
}

// steps 1-3: counts, starts and the stable cluster-sorted order of the points
static km_status launch_sort(const int32_t *assign, int64_t n, int k, const UpdWs &w, hipStream_t s) {
  const bool lds = k <= kLdsCursorMax;
  const size_t lds_bytes = lds ? sizeof(int) * (size_t)k : 0;
  if (!lds) hipLaunchKernelGGL(fill_int_kernel, dim3(1024), dim3(256), 0, s, w.offs, w.L, 0);
  hipLaunchKernelGGL(hist_kernel, dim3(w.nblk), dim3(256), lds_bytes, s, assign, n, k, w.nblk, w.ppb, w.offs,
                     (int)lds);
  hipLaunchKernelGGL(scan_reduce_kernel, dim3(w.nsb), dim3(256), 0, s, w.offs, w.L, w.bsum);
  hipLaunchKernelGGL(scan_down_kernel, dim3(w.nsb), dim3(256), 0, s, w.offs, w.L, w.bsum, w.total);
  hipLaunchKernelGGL(counts_kernel, dim3(1), dim3(256), 0, s, w.offs, w.nblk, k, w.total, w.cnt, w.cstart, w.choff);
  hipLaunchKernelGGL(scatter_kernel, dim3(w.nblk), dim3(256), lds_bytes, s, assign, n, k, w.nblk, w.ppb, w.offs,
                     (int)lds, w.perm);
  KMQ_LAUNCH_CHECK("update: sort");
  return KM_OK;
}

static Points sort_only_points(int64_t n) {  // the sort's workspace does not depend on the format
  Points q{};
  q.n = n;
  q.d = 4;
  return q;
}

size_t sort_bytes(int64_t n, int k) {
  size_t b = 0;
  carve(sort_only_points(n), k, nullptr, &b);
  return b;
}

km_status launch_cluster_sort(const int32_t *assign, int64_t n, int k, void *ws, SortOut *out, hipStream_t s) {
  UpdWs w = carve(sort_only_points(n), k, ws, nullptr);
  out->perm = w.perm;
  out->cnt = w.cnt;
  out->cstart = w.cstart;
  return launch_sort(assign, n, k, w, s);
}

km_status launch_update(const Points &P, const int32_t *assign, int k, void *C, int64_t *counts, int policy,
                        void *ws, hipStream_t s, const int *seg_lo, const int *seg_hi) {
  UpdWs w = carve(P, k, ws, nullptr);
  km_status sst = launch_sort(assign, P.n, k, w, s);
  if (sst != KM_OK) return sst;

  const int d = P.d;
  Compose cm;
  cm.C = static_cast<float *>(C);
  cm.m = P.center;
  cm.d_bits = P.fmt == KM_HYBRID ? P.d_front : 0;
  cm.bits = is_bits_fmt(P.fmt);
  cm.counts = counts;
  if (P.fmt == KM_SQ8) {
    hipLaunchKernelGGL(segsum_sq8_kernel, dim3(w.maxchunks, (unsigned)cdiv(d, 1024)), dim3(256), 0, s,
                       static_cast<const uint8_t *>(P.data), P.ld, d, w.perm, w.cnt, w.cstart, w.choff, k,
                       static_cast<int *>(w.partial));
    hipLaunchKernelGGL(finalize_sq8_kernel, dim3(k, (unsigned)cdiv(d, 256)), dim3(256), 0, s,
                       static_cast<const int *>(w.partial), d, w.cnt, w.choff, static_cast<uint8_t *>(w.Z), w.fresh,
                       static_cast<uint8_t *>(C), counts);
  } else {
    int df = 0;
    const float *F = nullptr;
    int64_t fld = 0;
    if (P.fmt == KM_F32) {
      df = d;
      F = static_cast<const float *>(P.data);
      fld = P.ld;
    } else if (P.fmt == KM_HYBRID) {
      df = P.d_front;
      F = P.front;
      fld = P.d_front;
    }
    if (P.fmt == KM_LVQ4)
      hipLaunchKernelGGL(segsum_lvq4_kernel, dim3(w.maxchunks, (unsigned)cdiv(d, 1024)), dim3(256), 0, s,
                         static_cast<const uint8_t *>(P.data), P.ld, P.vparams, d, w.perm, w.cnt, w.cstart, w.choff,
                         k, static_cast<uint32_t *>(w.partial), w.partialM, w.partialB, w.dp);
    if (P.fmt == KM_BF16)
      hipLaunchKernelGGL(segsum_bf16_kernel, dim3(w.maxchunks, (unsigned)cdiv(d, 512)), dim3(256), 0, s,
                         static_cast<const uint16_t *>(P.data), P.ld, d, w.perm, w.cnt, w.cstart, w.choff, k,
                         static_cast<float *>(w.partial), w.dp);
    if (df > 0)
      hipLaunchKernelGGL(segsum_f32_kernel, dim3(w.maxchunks, (unsigned)cdiv(df, 256)), dim3(256), 0, s, F, fld, df,
                         w.perm, w.cnt, w.cstart, w.choff, k, static_cast<float *>(w.partial), w.dp);
    const int d_bits = P.fmt == KM_HYBRID ? P.d_front : 0;
    if (is_bits_fmt(P.fmt)) {
      const int dt = d - d_bits;
      hipLaunchKernelGGL(segsum_bits_kernel, dim3(w.maxchunks, (unsigned)cdiv(dt, 1024)), dim3(256), 0, s,
                         static_cast<const uint32_t *>(P.data), (int64_t)(d / 32), d_bits / 32, dt, P.alpha, w.perm,
                         w.cnt, w.cstart, w.choff, k, static_cast<uint32_t *>(w.partial), w.partialA, w.partialM,
                         w.dp, d_bits);
    }
    hipLaunchKernelGGL(finalize_f32_kernel, dim3(k, (unsigned)cdiv(w.dp, 256)), dim3(256), 0, s,
                       static_cast<const float *>(w.partial), w.dp, w.cnt, w.choff, static_cast<float *>(w.Z),
                       w.fresh, is_bits_fmt(P.fmt) ? w.partialA : nullptr, w.partialM,
                       P.fmt == KM_LVQ4 ? w.partialB : nullptr, d_bits, cm);
  }
  KMQ_LAUNCH_CHECK("update: segmented sums");

  if (policy == KM_EMPTY_SPLIT) {
    if (P.fmt == KM_SQ8)
      hipLaunchKernelGGL(split_kernel<true>, dim3(1), dim3(256), 0, s, w.Z, k, w.dp, w.cnt, w.cntw, w.fresh,
                         w.empties, seg_lo, seg_hi, cm);
    else
      hipLaunchKernelGGL(split_kernel<false>, dim3(1), dim3(256), 0, s, w.Z, k, w.dp, w.cnt, w.cntw, w.fresh,
                         w.empties, seg_lo, seg_hi, cm);
  }
  KMQ_LAUNCH_CHECK("update: split/compose");
  return KM_OK;
}

}  // namespace kmq
