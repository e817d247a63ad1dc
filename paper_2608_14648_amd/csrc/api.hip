// C ABI entry points of libkmq: argument validation (host only, before any HIP
// call), stream-ordered scratch memory, and the Lloyd loop of Sec. 2.3.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <new>
#include <vector>

#include "common.hpp"

namespace kmq {

static thread_local char g_err[512] = "";

void set_error(const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}

km_status hip_fail(hipError_t e, const char *what) {
  set_error("%s: %s", what, hipGetErrorString(e));
  return KM_EDEVICE;
}

#define KMQ_CHECK(cond, code, ...) \
  do {                             \
    if (!(cond)) {                 \
      set_error(__VA_ARGS__);      \
      return (code);               \
    }                              \
  } while (0)

static bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Keep freed scratch in each device's default pool instead of returning it to
// the driver after every synchronisation.
static km_status prepare_pool() {
  static std::mutex mu;
  static bool done[64] = {false};
  int dev = 0;
  KMQ_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> g(mu);
  if (dev >= 0 && dev < 64 && !done[dev]) {
    hipMemPool_t pool;
    KMQ_HIP(hipDeviceGetDefaultMemPool(&pool, dev));
    uint64_t thr = ~0ull;
    KMQ_HIP(hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr));
    done[dev] = true;
  }
  return KM_OK;
}

// Scratch taken from the stream-ordered pool and handed back on the same stream.
class Scratch {
 public:
  explicit Scratch(hipStream_t s) : s_(s) {}
  ~Scratch() {
    if (p_) (void)hipFreeAsync(p_, s_);
  }
  km_status alloc(size_t bytes) {
    // KMQ_FAIL_ALLOC=1 makes every scratch allocation fail before any HIP call:
    // the failure path can be exercised on a machine without a GPU
    const char *fail = getenv("KMQ_FAIL_ALLOC");
    if (fail && fail[0] == '1') {
      set_error("scratch allocation of %zu bytes failed: refused (KMQ_FAIL_ALLOC=1)", bytes);
      return KM_ENOMEM;
    }
    km_status st = prepare_pool();
    if (st != KM_OK) return st;
    hipError_t e = hipMallocAsync(&p_, std::max<size_t>(bytes, 256), s_);
    if (e == hipErrorOutOfMemory) {
      p_ = nullptr;
      set_error("scratch allocation of %zu bytes failed: %s", bytes, hipGetErrorString(e));
      return KM_ENOMEM;
    }
    if (e != hipSuccess) {
      p_ = nullptr;
      return hip_fail(e, "hipMallocAsync");
    }
    return KM_OK;
  }
  uint8_t *get() const { return static_cast<uint8_t *>(p_); }

 private:
  void *p_ = nullptr;
  hipStream_t s_;
};

static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

// Scratch of kmeans_assign_noalloc: one file-scope array per device, for the
// life of the process.  Its name is a host-side stand-in in host code; the
// device address is taken once per device with hipGetSymbolAddress and only
// that address is handed to kernels.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

static km_status static_scratch(uint8_t **out) {
  static std::mutex mu;
  static void *addr[64] = {nullptr};
  int dev = 0;
  KMQ_HIP(hipGetDevice(&dev));
  KMQ_CHECK(dev >= 0 && dev < 64, KM_EDEVICE, "device index %d outside [0, 64)", dev);
  std::lock_guard<std::mutex> g(mu);
  if (addr[dev] == nullptr) {
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    addr[dev] = p;
  }
  *out = static_cast<uint8_t *>(addr[dev]);
  return KM_OK;
}

static km_status check_points(const km_points *P, Points *out) {
  KMQ_CHECK(P != nullptr, KM_EINVAL, "points descriptor is NULL");
  const int fmt = P->fmt;
  KMQ_CHECK(fmt == KM_F32 || fmt == KM_BF16 || fmt == KM_SQ8 || fmt == KM_SIGN1 || fmt == KM_HYBRID ||
                fmt == KM_RABITQ || fmt == KM_LVQ4,
            KM_EUNSUPPORTED, "unknown point format %d", fmt);
  KMQ_CHECK(P->reserved == 0, KM_EINVAL, "reserved field must be 0");
  KMQ_CHECK(P->n >= 1 && P->n < (int64_t)INT32_MAX, KM_EINVAL, "n = %lld outside [1, 2^31)", (long long)P->n);
  KMQ_CHECK(P->d >= 1, KM_EINVAL, "d = %d must be >= 1", P->d);
  KMQ_CHECK(P->data != nullptr, KM_EINVAL, "points data is NULL");
  KMQ_CHECK(aligned16(P->data), KM_EINVAL, "points data must be 16-byte aligned");
  Points p{};
  p.fmt = fmt;
  p.d = P->d;
  p.n = P->n;
  p.data = P->data;
  p.ld = P->ld;
  p.alpha = P->alpha;
  p.center = P->center;
  p.front = P->front;
  p.d_front = P->d_front;
  p.raw = P->raw;
  p.raw_ld = P->raw_ld;
  p.vparams = P->vparams;
  KMQ_CHECK((fmt == KM_LVQ4) == (P->vparams != nullptr), KM_EINVAL,
            "vparams must be given for LVQ4 points and only for them");
  if (fmt == KM_F32 || fmt == KM_BF16 || fmt == KM_SQ8 || fmt == KM_LVQ4) {
    // the assignment kernels address a tile of 256 rows with 32-bit offsets
    const int64_t elem = fmt == KM_F32 ? 4 : fmt == KM_BF16 ? 2 : 1;
    KMQ_CHECK(P->ld >= 0 && P->ld <= ((int64_t)1 << 31) / (256 * elem) - 1, KM_EINVAL,
              "ld = %lld too large: 256 rows of ld elements must span less than 2^31 bytes", (long long)P->ld);
  }
  if (P->raw) {
    KMQ_CHECK(fmt != KM_SQ8, KM_EINVAL, "raw rows are not allowed for SQ8 points (their centroids are codes)");
    KMQ_CHECK(P->d % 4 == 0 && P->raw_ld >= P->d && P->raw_ld % 4 == 0 && aligned16(P->raw), KM_EINVAL,
              "raw rows need d %% 4 == 0, raw_ld >= d, raw_ld %% 4 == 0 and 16-byte alignment");
  }
  if (fmt == KM_F32) {
    KMQ_CHECK(P->d % 4 == 0, KM_EINVAL, "fp32 points need d %% 4 == 0 (d = %d)", P->d);
    KMQ_CHECK(P->ld >= P->d && P->ld % 4 == 0, KM_EINVAL, "fp32 points need ld >= d and ld %% 4 == 0");
    KMQ_CHECK(P->d_front == 0, KM_EINVAL, "d_front must be 0 for this format");
  } else if (fmt == KM_BF16) {
    KMQ_CHECK(P->d % 8 == 0, KM_EINVAL, "bfloat16 points need d %% 8 == 0 (d = %d)", P->d);
    KMQ_CHECK(P->ld >= P->d && P->ld % 8 == 0, KM_EINVAL, "bfloat16 points need ld >= d and ld %% 8 == 0");
    KMQ_CHECK(P->d_front == 0, KM_EINVAL, "d_front must be 0 for this format");
  } else if (fmt == KM_SQ8) {
    KMQ_CHECK(P->d % 16 == 0, KM_EINVAL, "SQ8 codes need d %% 16 == 0 (d = %d)", P->d);
    KMQ_CHECK(P->ld >= P->d && P->ld % 16 == 0, KM_EINVAL, "SQ8 codes need ld >= d and ld %% 16 == 0");
    KMQ_CHECK(P->d_front == 0, KM_EINVAL, "d_front must be 0 for this format");
  } else if (fmt == KM_LVQ4) {
    KMQ_CHECK(P->d % 32 == 0, KM_EINVAL, "LVQ4 codes need d %% 32 == 0 (d = %d)", P->d);
    KMQ_CHECK(P->ld >= P->d / 2 && P->ld % 16 == 0, KM_EINVAL, "LVQ4 codes need ld >= d/2 and ld %% 16 == 0");
    KMQ_CHECK(P->d_front == 0 && P->center == nullptr, KM_EINVAL, "LVQ4 points take no front and no center");
    KMQ_CHECK(aligned16(P->vparams), KM_EINVAL, "vparams must be 16-byte aligned");
  } else {
    KMQ_CHECK(P->d % 32 == 0, KM_EINVAL, "1-bit codes need d %% 32 == 0 (d = %d)", P->d);
    KMQ_CHECK(P->alpha != nullptr, KM_EINVAL, "alpha is NULL");
    if (fmt == KM_RABITQ)
      KMQ_CHECK(P->center == nullptr, KM_EINVAL, "RabitQ codes are of the rotated residual: center must be NULL");
    else
      KMQ_CHECK(P->center != nullptr, KM_EINVAL, "center is NULL");
    p.ld = P->d / 32;
    if (fmt == KM_HYBRID) {
      KMQ_CHECK(P->d_front > 0 && P->d_front < P->d && P->d_front % 32 == 0, KM_EINVAL,
                "hybrid needs 0 < d_front < d and d_front %% 32 == 0 (d_front = %d)", P->d_front);
      KMQ_CHECK(P->front != nullptr && aligned16(P->front), KM_EINVAL, "hybrid front must be a 16-byte aligned pointer");
    } else {
      KMQ_CHECK(P->d_front == 0, KM_EINVAL, "d_front must be 0 for this format");
    }
  }
  *out = p;
  return KM_OK;
}

static km_status check_centroids(const Points &p, const void *C, int k) {
  KMQ_CHECK(k >= 1, KM_EINVAL, "k = %d must be >= 1", k);
  KMQ_CHECK(C != nullptr, KM_EINVAL, "centroids pointer is NULL");
  KMQ_CHECK(aligned16(C), KM_EINVAL, "centroids must be 16-byte aligned");
  (void)p;
  return KM_OK;
}

// The raw rows of p as fp32 points (the last update of a fit).
static Points raw_points(const Points &p) {
  Points r{};
  r.fmt = KM_F32;
  r.d = p.d;
  r.n = p.n;
  r.data = p.raw;
  r.ld = p.raw_ld;
  return r;
}

static size_t centroid_bytes(const Points &p, int k) {  // BF16 centroids are fp32
  return (size_t)k * p.d * (p.fmt == KM_SQ8 ? 1 : sizeof(float));
}

}  // namespace kmq

using namespace kmq;

extern "C" {

const char *km_last_error(void) { return g_err; }

km_status km_release(void) {
  int dev = 0;
  KMQ_HIP(hipGetDevice(&dev));
  hipMemPool_t pool;
  KMQ_HIP(hipDeviceGetDefaultMemPool(&pool, dev));
  KMQ_HIP(hipMemPoolTrimTo(pool, 0));
  return KM_OK;
}

km_status quantize(const float *X, int64_t n, int32_t d, int64_t ldx, int32_t fmt, void *codes, float *params,
                   float *alpha, int32_t d_front, float *front, int32_t flags, km_stream stream) {
  g_err[0] = 0;
  KMQ_CHECK(fmt == KM_SQ8 || fmt == KM_SIGN1 || fmt == KM_BF16 || fmt == KM_LVQ4, KM_EUNSUPPORTED,
            "quantize supports SQ8, SIGN1, BF16 and LVQ4 (fmt = %d)", fmt);
  KMQ_CHECK(X != nullptr && codes != nullptr && (params != nullptr || fmt == KM_BF16), KM_EINVAL, "NULL argument");
  KMQ_CHECK(n >= 1 && n < (int64_t)INT32_MAX, KM_EINVAL, "n = %lld outside [1, 2^31)", (long long)n);
  KMQ_CHECK(d >= 1 && ldx >= d && ldx % 4 == 0, KM_EINVAL, "need d >= 1, ldx >= d, ldx %% 4 == 0");
  KMQ_CHECK(aligned16(X) && aligned16(codes), KM_EINVAL, "X and codes must be 16-byte aligned");
  KMQ_CHECK((flags & ~KM_Q_FIT_PARAMS) == 0, KM_EINVAL, "unknown flags 0x%x", flags);
  if (fmt == KM_SQ8) {
    KMQ_CHECK(d % 16 == 0, KM_EINVAL, "SQ8 needs d %% 16 == 0 (d = %d)", d);
    KMQ_CHECK(d_front == 0 && front == nullptr, KM_EINVAL, "d_front/front are for 1-bit codes only");
  } else if (fmt == KM_BF16) {
    KMQ_CHECK(d % 8 == 0, KM_EINVAL, "BF16 needs d %% 8 == 0 (d = %d)", d);
    KMQ_CHECK(d_front == 0 && front == nullptr, KM_EINVAL, "d_front/front are for 1-bit codes only");
  } else if (fmt == KM_LVQ4) {
    KMQ_CHECK(d % 32 == 0, KM_EINVAL, "LVQ4 needs d %% 32 == 0 (d = %d)", d);
    KMQ_CHECK(d_front == 0 && front == nullptr, KM_EINVAL, "d_front/front are for 1-bit codes only");
    KMQ_CHECK(aligned16(params), KM_EINVAL, "params must be 16-byte aligned");
  } else {
    KMQ_CHECK(d % 32 == 0, KM_EINVAL, "1-bit codes need d %% 32 == 0 (d = %d)", d);
    KMQ_CHECK(alpha != nullptr, KM_EINVAL, "alpha is NULL");
    KMQ_CHECK(d_front >= 0 && d_front < d && d_front % 32 == 0, KM_EINVAL,
              "need 0 <= d_front < d and d_front %% 32 == 0 (d_front = %d)", d_front);
    KMQ_CHECK(front == nullptr || d_front > 0, KM_EINVAL, "front copy needs d_front > 0");
    KMQ_CHECK(aligned16(params) && (front == nullptr || aligned16(front)), KM_EINVAL,
              "params and front must be 16-byte aligned");
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Scratch ws(s);
  km_status st = ws.alloc(quantize_bytes(n, d, fmt));
  if (st != KM_OK) return st;
  return launch_quantize(X, n, d, ldx, fmt, codes, params, alpha, d_front, front, flags, ws.get(), s);
}

km_status pca_fit_cov(const float *X, int64_t n, int32_t d, float *mean, float *cov, km_stream stream) {
  g_err[0] = 0;
  KMQ_CHECK(X != nullptr && mean != nullptr && cov != nullptr, KM_EINVAL, "NULL argument");
  KMQ_CHECK(n >= 1 && n < (int64_t)INT32_MAX, KM_EINVAL, "n = %lld outside [1, 2^31)", (long long)n);
  KMQ_CHECK(d >= 1 && d % 4 == 0, KM_EINVAL, "pca_fit_cov needs d %% 4 == 0 (d = %d)", d);
  KMQ_CHECK(aligned16(X) && aligned16(mean), KM_EINVAL, "X and mean must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Scratch ws(s);
  km_status st = ws.alloc(pca_cov_bytes(n, d));
  if (st != KM_OK) return st;
  return launch_pca_cov(X, n, d, mean, cov, ws.get(), s);
}

km_status pca_project(const float *X, int64_t n, int32_t d, const float *mean, const float *W, int32_t d_out,
                      float *Y, km_stream stream) {
  g_err[0] = 0;
  KMQ_CHECK(X != nullptr && mean != nullptr && W != nullptr && Y != nullptr, KM_EINVAL, "NULL argument");
  KMQ_CHECK(n >= 1 && n < (int64_t)INT32_MAX, KM_EINVAL, "n = %lld outside [1, 2^31)", (long long)n);
  KMQ_CHECK(d >= 1 && d % 4 == 0, KM_EINVAL, "pca_project needs d %% 4 == 0 (d = %d)", d);
  KMQ_CHECK(d_out >= 1, KM_EINVAL, "d_out = %d must be >= 1", d_out);
  KMQ_CHECK(aligned16(X) && aligned16(mean), KM_EINVAL, "X and mean must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Scratch ws(s);
  km_status st = ws.alloc(pca_project_bytes(d, d_out));
  if (st != KM_OK) return st;
  return launch_pca_project(X, n, d, (int64_t)d, mean, W, d_out, Y, ws.get(), s);
}

km_status rabitq_encode(const float *X, int64_t n, int32_t d, int64_t ldx, const float *P, float *m, uint32_t *bits,
                        float *alpha, float *Y, int32_t flags, km_stream stream) {
  g_err[0] = 0;
  KMQ_CHECK(X != nullptr && P != nullptr && m != nullptr && bits != nullptr && alpha != nullptr, KM_EINVAL,
            "NULL argument");
  KMQ_CHECK(n >= 1 && n < (int64_t)INT32_MAX, KM_EINVAL, "n = %lld outside [1, 2^31)", (long long)n);
  KMQ_CHECK(d >= 32 && d % 32 == 0, KM_EINVAL, "rabitq_encode needs d %% 32 == 0 (d = %d)", d);
  KMQ_CHECK(ldx >= d && ldx % 4 == 0, KM_EINVAL, "need ldx >= d and ldx %% 4 == 0");
  KMQ_CHECK(aligned16(X) && aligned16(m) && (Y == nullptr || aligned16(Y)), KM_EINVAL,
            "X, m and Y must be 16-byte aligned");
  KMQ_CHECK((flags & ~KM_Q_FIT_PARAMS) == 0, KM_EINVAL, "unknown flags 0x%x", flags);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Scratch ws(s);
  km_status st = ws.alloc(rabitq_encode_bytes(n, d, Y != nullptr));
  if (st != KM_OK) return st;
  return launch_rabitq_encode(X, n, d, ldx, P, m, bits, alpha, Y, flags, ws.get(), s);
}

}  // extern "C"

namespace kmq {
// scratch layout of one assignment call: centroid preparation | scores when the
// caller gives none but wants the objective | point-only terms | objective partials
struct AssignScratch {
  size_t b_prep, b_score, b_xc, b_part;
  size_t total() const { return b_prep + b_score + b_xc + b_part; }
};

static AssignScratch assign_scratch(const Points &p, int k, const float *score, const double *objective) {
  AssignScratch a;
  a.b_prep = al(prep_bytes(p, k));
  a.b_score = objective != nullptr && score == nullptr ? al(sizeof(float) * (size_t)p.n) : 0;
  a.b_xc = objective ? al(sizeof(float) * (size_t)p.n) : 0;
  a.b_part = objective ? al(sizeof(double) * (size_t)objective_blocks(p.n)) : 0;
  return a;
}

static km_status check_assign_args(const km_points *P, const void *C, int32_t k, const int32_t *assign, Points *p) {
  km_status st = check_points(P, p);
  if (st != KM_OK) return st;
  st = check_centroids(*p, C, k);
  if (st != KM_OK) return st;
  KMQ_CHECK(assign != nullptr, KM_EINVAL, "assign is NULL");
  return KM_OK;
}

// the launches of one assignment call on the scratch at w (layout as above)
static km_status assign_on(const Points &p, const void *C, int32_t k, int32_t *assign, float *score,
                           double *objective, const AssignScratch &a, uint8_t *w, hipStream_t s) {
  const size_t b_prep = a.b_prep, b_score = a.b_score, b_xc = a.b_xc;
  const bool need_score = b_score != 0;
  float *sc = need_score ? reinterpret_cast<float *>(w + b_prep) : score;
  float *xc = reinterpret_cast<float *>(w + b_prep + b_score);
  double *part = reinterpret_cast<double *>(w + b_prep + b_score + b_xc);
  CentroidPrep cp;
  km_status st = launch_prep(p, C, k, w, &cp, s);
  if (st != KM_OK) return st;
  st = launch_assign(p, C, cp, k, assign, sc, s);
  if (st != KM_OK) return st;
  if (objective) {
    st = launch_xconst(p, xc, s);
    if (st != KM_OK) return st;
    st = launch_objective(p, xc, sc, p.n, objective, part, objective_blocks(p.n), s);
  }
  return st;
}
}  // namespace kmq

extern "C" {

km_status kmeans_assign(const km_points *P, const void *C, int32_t k, int32_t *assign, float *score,
                        double *objective, km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_assign_args(P, C, k, assign, &p);
  if (st != KM_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const AssignScratch a = assign_scratch(p, k, score, objective);
  Scratch ws(s);
  st = ws.alloc(a.total());
  if (st != KM_OK) return st;
  return assign_on(p, C, k, assign, score, objective, a, ws.get(), s);
}

km_status kmeans_assign_noalloc(const km_points *P, const void *C, int32_t k, int32_t *assign, float *score,
                                double *objective, km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_assign_args(P, C, k, assign, &p);
  if (st != KM_OK) return st;
  const AssignScratch a = assign_scratch(p, k, score, objective);
  KMQ_CHECK(a.total() <= kStaticScratchBytes, KM_EINVAL,
            "kmeans_assign_noalloc needs %zu bytes of scratch for n = %lld, k = %d; its static buffer holds %zu",
            a.total(), (long long)p.n, k, kStaticScratchBytes);
  uint8_t *w = nullptr;
  st = static_scratch(&w);
  if (st != KM_OK) return st;
  return assign_on(p, C, k, assign, score, objective, a, w, reinterpret_cast<hipStream_t>(stream));
}

km_status kmeans_update(const km_points *P, const int32_t *assign, int32_t k, void *C, int64_t *counts, int32_t policy,
                        km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_points(P, &p);
  if (st != KM_OK) return st;
  st = check_centroids(p, C, k);
  if (st != KM_OK) return st;
  KMQ_CHECK(assign != nullptr, KM_EINVAL, "assign is NULL");
  KMQ_CHECK(policy == KM_EMPTY_SPLIT || policy == KM_EMPTY_KEEP, KM_EINVAL, "unknown empty-cluster policy %d", policy);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Scratch ws(s);
  st = ws.alloc(update_bytes(p, k));
  if (st != KM_OK) return st;
  return launch_update(p, assign, k, C, counts, policy, ws.get(), s);
}

namespace {
// hipEvent pairs around the launches of one fit (only when stats are requested)
class StageClock {
 public:
  StageClock(bool on, hipStream_t s) : on_(on), s_(s) {}
  ~StageClock() {
    for (auto &e : ev_) {
      (void)hipEventDestroy(e.first);
      (void)hipEventDestroy(e.second);
    }
  }
  km_status begin(int stage) {
    if (!on_) return KM_OK;
    hipEvent_t a, b;
    KMQ_HIP(hipEventCreate(&a));
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return hip_fail(hipErrorOutOfMemory, "hipEventCreate");
    }
    ev_.push_back({a, b});
    stage_.push_back(stage);
    KMQ_HIP(hipEventRecord(a, s_));
    return KM_OK;
  }
  km_status end() {
    if (!on_) return KM_OK;
    KMQ_HIP(hipEventRecord(ev_.back().second, s_));
    return KM_OK;
  }
  km_status collect(km_fit_stats *st) {
    if (!on_) return KM_OK;
    KMQ_HIP(hipStreamSynchronize(s_));
    double ms[4] = {0, 0, 0, 0};
    for (size_t i = 0; i < ev_.size(); ++i) {
      float t = 0.f;
      KMQ_HIP(hipEventElapsedTime(&t, ev_[i].first, ev_[i].second));
      ms[stage_[i]] += t;
    }
    st->assign_ms = ms[0];
    st->prep_ms = ms[1];
    st->update_ms = ms[2];
    st->other_ms = ms[3];
    return KM_OK;
  }

 private:
  bool on_;
  hipStream_t s_;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev_;
  std::vector<int> stage_;
};
enum { kStAssign = 0, kStPrep = 1, kStUpdate = 2, kStOther = 3 };
}  // namespace

#define KMQ_STAGE(clk, stage, expr)   \
  do {                                \
    st = (clk).begin(stage);          \
    if (st != KM_OK) return st;       \
    st = (expr);                      \
    if (st != KM_OK) return st;       \
    st = (clk).end();                 \
    if (st != KM_OK) return st;       \
  } while (0)

static km_status check_init_idx(const int64_t *init_idx, int k, int64_t n) {
  try {
    std::vector<int64_t> v(init_idx, init_idx + k);
    std::sort(v.begin(), v.end());
    KMQ_CHECK(v.front() >= 0 && v.back() < n, KM_EINVAL, "init_idx outside [0, n)");
    KMQ_CHECK(std::adjacent_find(v.begin(), v.end()) == v.end(), KM_EINVAL, "init_idx holds duplicates");
  } catch (const std::bad_alloc &) {
    set_error("host allocation failed");
    return KM_ENOMEM;
  }
  return KM_OK;
}

// Lloyd on validated arguments: STEP 1 from init_idx (HOST; NULL = C holds the
// start), iters x (STEP 2, STEP 3), final STEP 2; objective: DEVICE double[iters + 1].
static km_status fit_impl(const Points &p, int k, int iters, const int64_t *init_idx, void *C, int32_t *assign,
                          double *objective, int policy, StageClock &clk, hipStream_t s) {
  km_status st;
  const size_t b_prep = al(prep_bytes(p, k));
  const size_t b_upd = al(std::max(update_bytes(p, k), p.raw ? update_bytes(raw_points(p), k) : (size_t)0));
  const size_t b_score = objective ? al(sizeof(float) * (size_t)p.n) : 0;
  const size_t b_xc = objective ? al(sizeof(float) * (size_t)p.n) : 0;
  const size_t b_part = objective ? al(sizeof(double) * (size_t)objective_blocks(p.n)) : 0;
  const size_t b_idx = init_idx ? al(sizeof(int64_t) * (size_t)k) : 0;
  Scratch ws(s);
  st = ws.alloc(b_prep + b_upd + b_score + b_xc + b_part + b_idx);
  if (st != KM_OK) return st;
  uint8_t *w = ws.get();
  uint8_t *wprep = w;
  uint8_t *wupd = w + b_prep;
  float *sc = objective ? reinterpret_cast<float *>(w + b_prep + b_upd) : nullptr;
  float *xc = reinterpret_cast<float *>(w + b_prep + b_upd + b_score);
  double *part = reinterpret_cast<double *>(w + b_prep + b_upd + b_score + b_xc);
  int64_t *didx = reinterpret_cast<int64_t *>(w + b_prep + b_upd + b_score + b_xc + b_part);
  if (init_idx) {
    KMQ_HIP(hipMemcpyAsync(didx, init_idx, sizeof(int64_t) * (size_t)k, hipMemcpyHostToDevice, s));
    KMQ_STAGE(clk, kStOther, launch_gather_init(p, didx, k, C, s));
  }
  if (objective) KMQ_STAGE(clk, kStOther, launch_xconst(p, xc, s));
  CentroidPrep cp;
  for (int it = 0; it <= iters; ++it) {
    KMQ_STAGE(clk, kStPrep, launch_prep(p, C, k, wprep, &cp, s));
    KMQ_STAGE(clk, kStAssign, launch_assign(p, C, cp, k, assign, sc, s));
    if (objective)
      KMQ_STAGE(clk, kStOther, launch_objective(p, xc, sc, p.n, objective + it, part, objective_blocks(p.n), s));
    if (it == iters) break;  // the last pass only assigns (the final STEP 2)
    if (p.raw && it == iters - 1) {  // last update from the raw rows (Sec. 4.1)
      KMQ_STAGE(clk, kStUpdate, launch_update(raw_points(p), assign, k, C, nullptr, policy, wupd, s));
    } else {
      KMQ_STAGE(clk, kStUpdate, launch_update(p, assign, k, C, nullptr, policy, wupd, s));
    }
  }
  return KM_OK;
}

// Nearest integer to sqrt(k) (k is never the square of a half-integer).
static int meso_count(int k) {
  int r = 0;
  while ((int64_t)(r + 1) * (r + 1) <= k) ++r;
  return std::max(1, (int64_t)k - (int64_t)r * r > r ? r + 1 : r);
}

// Fine clusters per meso-cluster: one per non-empty meso-cluster, the other k - m
// shared in proportion to n_i - 1 (floor shares, then one more for the largest
// remainders, ties to the smaller index).  Sums to k, k_i <= n_i, when m <= k <= N.
static std::vector<int> fine_counts(const std::vector<int64_t> &n_i, int k) {
  const int km = (int)n_i.size();
  int64_t N = 0, m = 0;
  for (int64_t v : n_i) {
    N += v;
    m += v > 0;
  }
  const int64_t rem = k - m, cap = N - m;
  std::vector<int> ks(km);
  std::vector<int64_t> r(km, 0);
  int64_t given = 0;
  for (int i = 0; i < km; ++i) {
    const int64_t w = n_i[i] > 0 ? n_i[i] - 1 : 0;
    const int64_t share = cap > 0 ? rem * w / cap : 0;
    r[i] = cap > 0 ? rem * w % cap : 0;
    ks[i] = (int)((n_i[i] > 0 ? 1 : 0) + share);
    given += ks[i];
  }
  std::vector<int> order(km);
  for (int i = 0; i < km; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return r[a] > r[b]; });
  for (int64_t left = k - given, t = 0; left > 0; --left, ++t) ks[order[t]] += 1;
  return ks;
}

// The paper's fine counts (Sec. 4.4): the integer nearest to sqrt(n_i) for every
// non-empty meso-cluster (never a tie for integer n_i; at least 1 and at most n_i).
static std::vector<int> fine_counts_sqrt(const std::vector<int64_t> &n_i) {
  std::vector<int> ks(n_i.size(), 0);
  for (size_t i = 0; i < n_i.size(); ++i) {
    const int64_t v = n_i[i];
    if (v <= 0) continue;
    int64_t r = (int64_t)std::sqrt((double)v);
    while (r * r > v) --r;
    while ((r + 1) * (r + 1) <= v) ++r;
    ks[i] = (int)(v - r * r > r ? r + 1 : r);
  }
  return ks;
}

// FINE-CLUSTERING (Sec. 4.4) on validated arguments.  sqrt_rule: the paper's fine
// counts, k being the capacity of C; *k_used (nullable) receives the number of fine
// centroids.
static km_status fine_impl(const Points &p, const int32_t *meso, int k_meso, int k, int iters, bool c_given,
                           bool sqrt_rule, int *k_used, void *C, int32_t *assign, int32_t *k_fine, double *objective,
                           int policy, StageClock &clk,
                           hipStream_t s) {
  km_status st;
  // meso-cluster order of the points (stable) and the meso-cluster sizes
  Scratch wsort(s);
  st = wsort.alloc(sort_bytes(p.n, k_meso));
  if (st != KM_OK) return st;
  SortOut so{};
  KMQ_STAGE(clk, kStOther, launch_cluster_sort(meso, p.n, k_meso, wsort.get(), &so, s));
  std::vector<int> cnt(k_meso);
  KMQ_HIP(hipMemcpyAsync(cnt.data(), so.cnt, sizeof(int) * (size_t)k_meso, hipMemcpyDeviceToHost, s));
  KMQ_HIP(hipStreamSynchronize(s));
  std::vector<int64_t> n_i(cnt.begin(), cnt.end());
  int64_t N = 0, m = 0;
  for (int64_t v : n_i) {
    N += v;
    m += v > 0;
  }
  KMQ_CHECK(N >= 1, KM_EINVAL, "no point has a meso-cluster id in [0, %d)", k_meso);
  std::vector<int> kf;
  if (sqrt_rule) {
    kf = fine_counts_sqrt(n_i);
    int64_t kt = 0;
    for (int v : kf) kt += v;
    KMQ_CHECK(kt <= k, KM_EINVAL, "the fine counts sum to %lld, more than the %d centroids C holds", (long long)kt,
              k);
    k = (int)kt;  // the rest of C is left as it is
  } else {
    KMQ_CHECK(m <= k && k <= N, KM_EINVAL,
              "k = %d must lie between the number of non-empty meso-clusters (%lld) and the number of points with a "
              "meso-cluster (%lld)", k, (long long)m, (long long)N);
    kf = fine_counts(n_i, k);
  }
  if (k_used) *k_used = k;
  std::vector<int64_t> start(k_meso), off(k_meso + 1, 0);
  for (int i = 0, acc = 0; i < k_meso; ++i) {
    start[i] = acc;
    acc += cnt[i];
    off[i + 1] = off[i] + kf[i];
  }
  // host tables: initial rows (in meso order) and each centroid's segment
  std::vector<int64_t> idx(k);
  std::vector<int> seg(2 * (size_t)k);
  for (int i = 0; i < k_meso; ++i)
    for (int j = 0; j < kf[i]; ++j) {
      idx[off[i] + j] = start[i] + (int64_t)j * n_i[i] / kf[i];
      seg[off[i] + j] = (int)off[i];
      seg[k + off[i] + j] = (int)off[i + 1];
    }
  // the points of each meso-cluster as one contiguous run of rows
  Points q{};
  const size_t b_perm = al(permuted_bytes(p, N));
  const size_t b_prep = al(prep_bytes(slice_points(p, 0, N), k));
  const size_t b_upd = al(update_bytes(slice_points(p, 0, N), k));
  const size_t b_a = al(sizeof(int32_t) * (size_t)N);
  const size_t b_score = objective ? al(sizeof(float) * (size_t)N) : 0;
  const size_t b_xc = objective ? al(sizeof(float) * (size_t)N) : 0;
  const size_t b_part = objective ? al(sizeof(double) * (size_t)objective_blocks(N)) : 0;
  const size_t b_idx = al(sizeof(int64_t) * (size_t)k);
  const size_t b_seg = al(sizeof(int) * 2 * (size_t)k);
  // fp32, SQ8 and bf16: one assignment launch per pass over all meso-clusters
  // (segment and tile tables); other formats launch per meso-cluster
  const int seg_rows = assign_segment_rows(p);
  // a per-meso-cluster launch may split its few point tiles' centroid tiles over
  // groups (merging through per-point keys) where the launch over all N points
  // would not, and then the preparation sized for N holds no keys: give them room
  const size_t b_keys = seg_rows == 0 ? al(sizeof(unsigned long long) * (size_t)N) : 0;
  // point tiles of the segments with 128-centroid tiles first (n128 of them), then
  // those with 256-centroid tiles: one launch each
  std::vector<int4> segs;
  std::vector<int2> tiles;
  int64_t n128 = 0;
  if (seg_rows > 0) {
    for (int i = 0; i < k_meso; ++i)
      if (n_i[i] > 0) segs.push_back(make_int4((int)start[i], (int)n_i[i], (int)off[i], kf[i]));
    for (int cls = 128; cls <= 256; cls += 128) {
      for (int si = 0; si < (int)segs.size(); ++si) {
        if (segment_tile_centroids(segs[si].w) != cls) continue;
        for (int64_t tt = 0; tt * seg_rows < segs[si].y; ++tt) tiles.push_back(make_int2(si, (int)tt));
      }
      if (cls == 128) n128 = (int64_t)tiles.size();
    }
  }
  const size_t b_segs = al(sizeof(int4) * segs.size());
  const size_t b_tiles = al(sizeof(int2) * tiles.size());
  Scratch ws(s);
  st = ws.alloc(b_perm + b_prep + b_upd + b_a + b_score + b_xc + b_part + b_idx + b_seg + b_segs + b_tiles + b_keys);
  if (st != KM_OK) return st;
  uint8_t *w = ws.get();
  uint8_t *wperm = w;
  uint8_t *wprep = wperm + b_perm;
  uint8_t *wupd = wprep + b_prep;
  int32_t *ap = reinterpret_cast<int32_t *>(wupd + b_upd);
  float *sc = objective ? reinterpret_cast<float *>(wupd + b_upd + b_a) : nullptr;
  float *xc = reinterpret_cast<float *>(wupd + b_upd + b_a + b_score);
  double *part = reinterpret_cast<double *>(wupd + b_upd + b_a + b_score + b_xc);
  int64_t *didx = reinterpret_cast<int64_t *>(wupd + b_upd + b_a + b_score + b_xc + b_part);
  int *dseg = reinterpret_cast<int *>(wupd + b_upd + b_a + b_score + b_xc + b_part + b_idx);
  int4 *dsegs = reinterpret_cast<int4 *>(reinterpret_cast<uint8_t *>(dseg) + b_seg);
  int2 *dtiles = reinterpret_cast<int2 *>(reinterpret_cast<uint8_t *>(dsegs) + b_segs);
  auto *keys = b_keys ? reinterpret_cast<unsigned long long *>(reinterpret_cast<uint8_t *>(dtiles) + b_tiles) : nullptr;
  KMQ_STAGE(clk, kStOther, launch_permute_points(p, so.perm, N, wperm, &q, s));
  if (!segs.empty()) {
    KMQ_HIP(hipMemcpyAsync(dsegs, segs.data(), sizeof(int4) * segs.size(), hipMemcpyHostToDevice, s));
    KMQ_HIP(hipMemcpyAsync(dtiles, tiles.data(), sizeof(int2) * tiles.size(), hipMemcpyHostToDevice, s));
  }
  KMQ_HIP(hipMemcpyAsync(dseg, seg.data(), sizeof(int) * seg.size(), hipMemcpyHostToDevice, s));
  if (!c_given) {
    KMQ_HIP(hipMemcpyAsync(didx, idx.data(), sizeof(int64_t) * (size_t)k, hipMemcpyHostToDevice, s));
    KMQ_STAGE(clk, kStOther, launch_gather_init(q, didx, k, C, s));
  }
  const size_t crow = p.fmt == KM_SQ8 ? (size_t)p.d : sizeof(float) * (size_t)p.d;
  CentroidPrep cp;
  for (int it = 0; it <= iters; ++it) {
    KMQ_STAGE(clk, kStPrep, launch_prep(q, C, k, wprep, &cp, s));
    if (cp.keys == nullptr) cp.keys = keys;
    st = clk.begin(kStAssign);
    if (st != KM_OK) return st;
    if (!segs.empty()) {  // every meso-cluster against its own fine centroids, one launch per tile size
      st = launch_assign_segments(q, C, cp, dsegs, dtiles, n128, 128, ap, sc, s);
      if (st != KM_OK) return st;
      st = launch_assign_segments(q, C, cp, dsegs, dtiles + n128, (int64_t)tiles.size() - n128, 256, ap, sc, s);
      if (st != KM_OK) return st;
    }
    for (int i = 0; seg_rows == 0 && i < k_meso; ++i) {  // the same, one launch per meso-cluster
      if (n_i[i] == 0) continue;
      st = launch_assign(slice_points(q, start[i], n_i[i]), static_cast<const uint8_t *>(C) + off[i] * crow,
                         prep_slice(q, cp, (int)off[i], start[i]), kf[i], ap + start[i],
                         sc ? sc + start[i] : nullptr, s, (int)off[i]);
      if (st != KM_OK) return st;
    }
    st = clk.end();
    if (st != KM_OK) return st;
    if (it == iters) break;
    KMQ_STAGE(clk, kStUpdate, launch_update(q, ap, k, C, nullptr, policy, wupd, s, dseg, dseg + k));
  }
  if (objective) {
    KMQ_STAGE(clk, kStOther, launch_xconst(q, xc, s));
    KMQ_STAGE(clk, kStOther, launch_objective(q, xc, sc, N, objective, part, objective_blocks(N), s));
  }
  KMQ_STAGE(clk, kStOther, launch_scatter_assign(so.perm, ap, N, p.n, assign, s));
  if (k_fine) std::copy(kf.begin(), kf.end(), k_fine);
  return KM_OK;
}


km_status kmeans_fit(const km_points *P, int32_t k, int32_t iters, const int64_t *init_idx, void *C, int32_t *assign,
                     double *objective, int32_t policy, km_fit_stats *stats, km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_points(P, &p);
  if (st != KM_OK) return st;
  st = check_centroids(p, C, k);
  if (st != KM_OK) return st;
  KMQ_CHECK(assign != nullptr, KM_EINVAL, "assign is NULL");
  KMQ_CHECK(k <= p.n, KM_EINVAL, "k = %d exceeds n = %lld", k, (long long)p.n);
  KMQ_CHECK(iters >= 0, KM_EINVAL, "iters = %d must be >= 0", iters);
  KMQ_CHECK(policy == KM_EMPTY_SPLIT || policy == KM_EMPTY_KEEP, KM_EINVAL, "unknown empty-cluster policy %d", policy);
  if (init_idx) {
    st = check_init_idx(init_idx, k, p.n);
    if (st != KM_OK) return st;
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  (void)centroid_bytes;
  try {
    StageClock clk(stats != nullptr, s);
    st = fit_impl(p, k, iters, init_idx, C, assign, objective, policy, clk, s);
    if (st != KM_OK) return st;
    if (stats) {
      st = clk.collect(stats);
      if (st != KM_OK) return st;
      stats->assign_passes = iters + 1;
      stats->updates = iters;
    }
  } catch (const std::bad_alloc &) {
    set_error("host allocation failed");
    return KM_ENOMEM;
  }
  return KM_OK;
}

static km_status check_prune(const Points &p, const km_prune *pr, int *D0) {
  KMQ_CHECK(pr != nullptr, KM_EINVAL, "pruning parameters are NULL");
  KMQ_CHECK(p.fmt == KM_F32 || p.fmt == KM_SQ8, KM_EUNSUPPORTED,
            "dimension pruning is implemented for fp32 and SQ8 points (fmt = %d)", p.fmt);
  KMQ_CHECK(pr->reserved == 0, KM_EINVAL, "reserved field must be 0");
  KMQ_CHECK(pr->eps0 > 0.0, KM_EINVAL, "eps0 must be > 0");
  const int d0 = pr->d_front ? pr->d_front : prune_front_default(p.d);
  const int g = p.fmt == KM_F32 ? 8 : 16;  // the refinement reads 8 dims per lane
  KMQ_CHECK(p.d % g == 0, KM_EUNSUPPORTED, "pruning needs d %% %d == 0 (d = %d)", g, p.d);
  KMQ_CHECK(d0 >= 1 && d0 <= p.d && d0 % g == 0, KM_EINVAL,
            "d_front = %d must lie in [1, d] and be a multiple of %d", d0, g);
  KMQ_CHECK(d0 <= 256 && p.d - d0 <= 2048, KM_EUNSUPPORTED,
            "pruning supports d_front <= 256 and d - d_front <= 2048 (d_front = %d, d = %d)", d0, p.d);
  *D0 = d0;
  return KM_OK;
}

km_status kmeans_assign_pruned(const km_points *P, const void *C, int32_t k, const int32_t *prev, int32_t *assign,
                               double *dist, double *objective, const km_prune *pr, uint64_t *counters,
                               km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_points(P, &p);
  if (st != KM_OK) return st;
  st = check_centroids(p, C, k);
  if (st != KM_OK) return st;
  KMQ_CHECK(prev != nullptr && assign != nullptr, KM_EINVAL, "prev or assign is NULL");
  int D0 = 0;
  st = check_prune(p, pr, &D0);
  if (st != KM_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const size_t b_pr = al(pruned_bytes(p, k));
  Scratch ws(s);
  st = ws.alloc(b_pr + al(3 * sizeof(unsigned long long)));
  if (st != KM_OK) return st;
  unsigned long long *cnt = counters ? reinterpret_cast<unsigned long long *>(ws.get() + b_pr) : nullptr;
  if (cnt) {
    st = launch_zero_counters(cnt, s);
    if (st != KM_OK) return st;
  }
  st = launch_assign_pruned(p, C, k, prev, assign, dist, objective, pr->eps0, D0, cnt, ws.get(), s);
  if (st != KM_OK) return st;
  if (cnt) {
    KMQ_HIP(hipMemcpyAsync(counters, cnt, 3 * sizeof(unsigned long long), hipMemcpyDeviceToHost, s));
    KMQ_HIP(hipStreamSynchronize(s));
  }
  return KM_OK;
}

km_status kmeans_fit_pruned(const km_points *P, int32_t k, int32_t iters, const int64_t *init_idx, void *C,
                            int32_t *assign, double *objective, int32_t policy, const km_prune *pr,
                            km_fit_stats *stats, uint64_t *counters, km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_points(P, &p);
  if (st != KM_OK) return st;
  st = check_centroids(p, C, k);
  if (st != KM_OK) return st;
  KMQ_CHECK(assign != nullptr, KM_EINVAL, "assign is NULL");
  KMQ_CHECK(k <= p.n, KM_EINVAL, "k = %d exceeds n = %lld", k, (long long)p.n);
  KMQ_CHECK(iters >= 0, KM_EINVAL, "iters = %d must be >= 0", iters);
  KMQ_CHECK(policy == KM_EMPTY_SPLIT || policy == KM_EMPTY_KEEP, KM_EINVAL, "unknown empty-cluster policy %d", policy);
  int D0 = 0;
  st = check_prune(p, pr, &D0);
  if (st != KM_OK) return st;
  if (init_idx) {
    st = check_init_idx(init_idx, k, p.n);
    if (st != KM_OK) return st;
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const size_t b_prep = al(prep_bytes(p, k));
  const size_t b_upd = al(std::max(update_bytes(p, k), p.raw ? update_bytes(raw_points(p), k) : (size_t)0));
  const size_t b_score = objective ? al(sizeof(float) * (size_t)p.n) : 0;
  const size_t b_xc = objective ? al(sizeof(float) * (size_t)p.n) : 0;
  const size_t b_part = objective ? al(sizeof(double) * (size_t)objective_blocks(p.n)) : 0;
  const size_t b_idx = init_idx ? al(sizeof(int64_t) * (size_t)k) : 0;
  const size_t b_pr = al(pruned_bytes(p, k));
  const size_t b_cnt = al(3 * sizeof(unsigned long long));
  Scratch ws(s);
  st = ws.alloc(b_prep + b_upd + b_score + b_xc + b_part + b_idx + b_pr + b_cnt);
  if (st != KM_OK) return st;
  uint8_t *w = ws.get();
  uint8_t *wprep = w;
  uint8_t *wupd = w + b_prep;
  float *sc = objective ? reinterpret_cast<float *>(wupd + b_upd) : nullptr;
  float *xc = reinterpret_cast<float *>(wupd + b_upd + b_score);
  double *part = reinterpret_cast<double *>(wupd + b_upd + b_score + b_xc);
  int64_t *didx = reinterpret_cast<int64_t *>(wupd + b_upd + b_score + b_xc + b_part);
  uint8_t *wpr = wupd + b_upd + b_score + b_xc + b_part + b_idx;
  unsigned long long *cnt = counters ? reinterpret_cast<unsigned long long *>(wpr + b_pr) : nullptr;
  try {
    StageClock clk(stats != nullptr, s);
    if (cnt) KMQ_STAGE(clk, kStOther, launch_zero_counters(cnt, s));
    if (init_idx) {
      KMQ_HIP(hipMemcpyAsync(didx, init_idx, sizeof(int64_t) * (size_t)k, hipMemcpyHostToDevice, s));
      KMQ_STAGE(clk, kStOther, launch_gather_init(p, didx, k, C, s));
    }
    // the first pass is a full assignment
    CentroidPrep cp;
    KMQ_STAGE(clk, kStPrep, launch_prep(p, C, k, wprep, &cp, s));
    KMQ_STAGE(clk, kStAssign, launch_assign(p, C, cp, k, assign, sc, s));
    if (objective) {
      KMQ_STAGE(clk, kStOther, launch_xconst(p, xc, s));
      KMQ_STAGE(clk, kStOther, launch_objective(p, xc, sc, p.n, objective, part, objective_blocks(p.n), s));
    }
    for (int it = 1; it <= iters; ++it) {
      if (p.raw && it == iters) {  // last update from the raw rows (Sec. 4.1)
        KMQ_STAGE(clk, kStUpdate, launch_update(raw_points(p), assign, k, C, nullptr, policy, wupd, s));
      } else {
        KMQ_STAGE(clk, kStUpdate, launch_update(p, assign, k, C, nullptr, policy, wupd, s));
      }
      KMQ_STAGE(clk, kStAssign,
                launch_assign_pruned(p, C, k, assign, assign, nullptr, objective ? objective + it : nullptr,
                                     pr->eps0, D0, cnt, wpr, s));
    }
    if (stats) {
      st = clk.collect(stats);
      if (st != KM_OK) return st;
      stats->assign_passes = iters + 1;
      stats->updates = iters;
    }
    if (cnt) {
      KMQ_HIP(hipMemcpyAsync(counters, cnt, 3 * sizeof(unsigned long long), hipMemcpyDeviceToHost, s));
      KMQ_HIP(hipStreamSynchronize(s));
    }
  } catch (const std::bad_alloc &) {
    set_error("host allocation failed");
    return KM_ENOMEM;
  }
  return KM_OK;
}

km_status kmeans_fine(const km_points *P, const int32_t *meso_assign, int32_t k_meso, int32_t k, int32_t iters,
                      int32_t flags, void *C, int32_t *assign, int32_t *k_fine, double *objective, int32_t policy,
                      km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_points(P, &p);
  if (st != KM_OK) return st;
  st = check_centroids(p, C, k);
  if (st != KM_OK) return st;
  KMQ_CHECK(meso_assign != nullptr && assign != nullptr, KM_EINVAL, "meso_assign or assign is NULL");
  KMQ_CHECK(k_meso >= 1, KM_EINVAL, "k_meso = %d must be >= 1", k_meso);
  KMQ_CHECK(iters >= 0, KM_EINVAL, "iters = %d must be >= 0", iters);
  KMQ_CHECK((flags & ~(KM_FINE_C_GIVEN | KM_FINE_SQRT)) == 0, KM_EINVAL, "unknown flags 0x%x", flags);
  KMQ_CHECK(policy == KM_EMPTY_SPLIT || policy == KM_EMPTY_KEEP, KM_EINVAL, "unknown empty-cluster policy %d", policy);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  try {
    StageClock clk(false, s);
    return fine_impl(p, meso_assign, k_meso, k, iters, (flags & KM_FINE_C_GIVEN) != 0, (flags & KM_FINE_SQRT) != 0,
                     nullptr, C, assign, k_fine, objective, policy, clk, s);
  } catch (const std::bad_alloc &) {
    set_error("host allocation failed");
    return KM_ENOMEM;
  }
}

km_status kmeans_fit_hier(const km_points *P, int32_t k, const km_hier_params *hp, const int64_t *init_meso, void *C,
                          int32_t *assign, int32_t *meso_assign, int32_t *k_fine, double *objective, int32_t policy,
                          km_fit_stats *stats, double *phase_ms, km_stream stream) {
  g_err[0] = 0;
  Points p;
  km_status st = check_points(P, &p);
  if (st != KM_OK) return st;
  st = check_centroids(p, C, k);
  if (st != KM_OK) return st;
  KMQ_CHECK(hp != nullptr && init_meso != nullptr && assign != nullptr, KM_EINVAL,
            "hp, init_meso or assign is NULL");
  KMQ_CHECK(k <= p.n, KM_EINVAL, "k = %d exceeds n = %lld", k, (long long)p.n);
  const int km = hp->k_meso ? hp->k_meso : meso_count(k);
  KMQ_CHECK(km >= 1 && km <= k, KM_EINVAL, "k_meso = %d must lie in [1, k]", km);
  KMQ_CHECK(hp->iters_meso >= 0 && hp->iters_fine >= 0 && hp->iters_refine >= 0, KM_EINVAL,
            "iteration counts must be >= 0");
  KMQ_CHECK((hp->flags & ~KM_FINE_SQRT) == 0, KM_EINVAL, "unknown hierarchical flags 0x%x", hp->flags);
  KMQ_CHECK(policy == KM_EMPTY_SPLIT || policy == KM_EMPTY_KEEP, KM_EINVAL, "unknown empty-cluster policy %d", policy);
  st = check_init_idx(init_meso, km, p.n);
  if (st != KM_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Points pc = p;  // meso and fine phases cluster the compressed points only
  pc.raw = nullptr;
  pc.raw_ld = 0;
  const int R = hp->iters_refine;
  const size_t b_cm = al(centroid_bytes(p, km));
  const size_t b_am = meso_assign ? 0 : al(sizeof(int32_t) * (size_t)p.n);
  const size_t b_obj = (objective && R > 0) ? al(sizeof(double) * (size_t)(R + 1)) : 0;
  Scratch ws(s);
  st = ws.alloc(b_cm + b_am + b_obj);
  if (st != KM_OK) return st;
  void *Cm = ws.get();
  int32_t *am = meso_assign ? meso_assign : reinterpret_cast<int32_t *>(ws.get() + b_cm);
  double *objr = reinterpret_cast<double *>(ws.get() + b_cm + b_am);
  try {
    StageClock clk(stats != nullptr, s);
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    struct EvGuard {
      hipEvent_t *e;
      ~EvGuard() {
        for (int i = 0; i < 4; ++i)
          if (e[i]) (void)hipEventDestroy(e[i]);
      }
    } guard{ev};
    if (phase_ms)
      for (int i = 0; i < 4; ++i) KMQ_HIP(hipEventCreate(&ev[i]));
    if (phase_ms) KMQ_HIP(hipEventRecord(ev[0], s));
    st = fit_impl(pc, km, hp->iters_meso, init_meso, Cm, am, nullptr, policy, clk, s);
    if (st != KM_OK) return st;
    if (phase_ms) KMQ_HIP(hipEventRecord(ev[1], s));
    int kt = k;  // fine centroids made (fewer than k under the paper's counts)
    st = fine_impl(pc, am, km, k, hp->iters_fine, false, (hp->flags & KM_FINE_SQRT) != 0, &kt, C, assign, k_fine,
                   R > 0 ? nullptr : objective, policy, clk, s);
    if (st != KM_OK) return st;
    if (phase_ms) KMQ_HIP(hipEventRecord(ev[2], s));
    if (R > 0) {
      st = fit_impl(p, kt, R, nullptr, C, assign, objective ? objr : nullptr, policy, clk, s);
      if (st != KM_OK) return st;
      if (objective) KMQ_HIP(hipMemcpyAsync(objective, objr + R, sizeof(double), hipMemcpyDeviceToDevice, s));
    }
    if (phase_ms) {
      KMQ_HIP(hipEventRecord(ev[3], s));
      KMQ_HIP(hipEventSynchronize(ev[3]));
      for (int i = 0; i < 3; ++i) {
        float t = 0.f;
        KMQ_HIP(hipEventElapsedTime(&t, ev[i], ev[i + 1]));
        phase_ms[i] = t;
      }
    }
    if (stats) {
      st = clk.collect(stats);
      if (st != KM_OK) return st;
      stats->assign_passes = hp->iters_meso + 1 + hp->iters_fine + 1 + (R > 0 ? R + 1 : 0);
      stats->updates = hp->iters_meso + hp->iters_fine + R;
    }
  } catch (const std::bad_alloc &) {
    set_error("host allocation failed");
    return KM_ENOMEM;
  }
  return KM_OK;
}

km_status kmeans_cost(const float *X, int64_t n, int32_t d, int64_t ldx, const float *C, int32_t k,
                      const int32_t *assign, double *out, km_stream stream) {
  g_err[0] = 0;
  KMQ_CHECK(X != nullptr && C != nullptr && assign != nullptr && out != nullptr, KM_EINVAL, "NULL argument");
  KMQ_CHECK(n >= 1 && n < (int64_t)INT32_MAX, KM_EINVAL, "n = %lld outside [1, 2^31)", (long long)n);
  KMQ_CHECK(d >= 1 && ldx >= d, KM_EINVAL, "need d >= 1 and ldx >= d");
  KMQ_CHECK(k >= 1, KM_EINVAL, "k = %d must be >= 1", k);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Scratch ws(s);
  km_status st = ws.alloc(sizeof(double) * 1024);
  if (st != KM_OK) return st;
  return launch_cost(X, n, d, ldx, C, k, assign, out, reinterpret_cast<double *>(ws.get()), s);
}

}  // extern "C"
