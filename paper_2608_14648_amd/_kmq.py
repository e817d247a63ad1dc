"""ctypes binding of libkmq (include/kmq.h): argument marshalling only.

Every call takes torch tensors on the current HIP device, checks dtype, device
and contiguity, and passes raw device pointers plus the current stream to the
C ABI.  All arithmetic runs in the library's HIP kernels; there is no fallback:
a missing library or a non-OK status raises.
"""
from __future__ import annotations

import ctypes as ct
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkmq.so")

KM_F32, KM_BF16, KM_SQ8, KM_SIGN1, KM_HYBRID, KM_RABITQ, KM_LVQ4 = 0, 1, 2, 3, 4, 5, 6
KM_EMPTY_SPLIT, KM_EMPTY_KEEP = 0, 1
KM_Q_FIT_PARAMS = 1
KM_FINE_C_GIVEN = 1
KM_FINE_SQRT = 2
STATUS = {0: "KM_OK", -1: "KM_EINVAL", -2: "KM_EUNSUPPORTED", -3: "KM_ENOMEM", -4: "KM_EDEVICE"}
EXPORTS = ("quantize", "rabitq_encode", "pca_fit_cov", "pca_project", "kmeans_assign", "kmeans_assign_noalloc",
           "kmeans_update",
           "kmeans_fit", "kmeans_fine", "kmeans_fit_hier", "kmeans_assign_pruned", "kmeans_fit_pruned", "kmeans_cost",
           "km_last_error", "km_release")


class KmqError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class KmPoints(ct.Structure):
    _fields_ = [("fmt", ct.c_int32), ("d", ct.c_int32), ("n", ct.c_int64), ("data", ct.c_void_p),
                ("ld", ct.c_int64), ("alpha", ct.c_void_p), ("center", ct.c_void_p), ("front", ct.c_void_p),
                ("d_front", ct.c_int32), ("reserved", ct.c_int32), ("raw", ct.c_void_p), ("raw_ld", ct.c_int64),
                ("vparams", ct.c_void_p)]


class KmFitStats(ct.Structure):
    _fields_ = [("assign_ms", ct.c_double), ("prep_ms", ct.c_double), ("update_ms", ct.c_double),
                ("other_ms", ct.c_double), ("assign_passes", ct.c_int32), ("updates", ct.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class KmPrune(ct.Structure):
    _fields_ = [("eps0", ct.c_double), ("d_front", ct.c_int32), ("reserved", ct.c_int32)]


class KmHierParams(ct.Structure):
    _fields_ = [("k_meso", ct.c_int32), ("iters_meso", ct.c_int32), ("iters_fine", ct.c_int32),
                ("iters_refine", ct.c_int32), ("flags", ct.c_int32)]


_lib = None


def lib():
    """The loaded libkmq.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libkmq.so not found at {LIB_PATH}: build it with "
                               "`python -m paper_2608_14648_amd.build` (hipcc, gfx950)")
        L = ct.CDLL(LIB_PATH)
        vp, i32, i64 = ct.c_void_p, ct.c_int32, ct.c_int64
        sig = {
            "quantize": [vp, i64, i32, i64, i32, vp, vp, vp, i32, vp, i32, vp],
            "rabitq_encode": [vp, i64, i32, i64, vp, vp, vp, vp, vp, i32, vp],
            "pca_fit_cov": [vp, i64, i32, vp, vp, vp],
            "pca_project": [vp, i64, i32, vp, vp, i32, vp, vp],
            "kmeans_assign": [ct.POINTER(KmPoints), vp, i32, vp, vp, vp, vp],
            "kmeans_assign_noalloc": [ct.POINTER(KmPoints), vp, i32, vp, vp, vp, vp],
            "kmeans_update": [ct.POINTER(KmPoints), vp, i32, vp, vp, i32, vp],
            "kmeans_fit": [ct.POINTER(KmPoints), i32, i32, vp, vp, vp, vp, i32, ct.POINTER(KmFitStats), vp],
            "kmeans_fine": [ct.POINTER(KmPoints), vp, i32, i32, i32, i32, vp, vp, vp, vp, i32, vp],
            "kmeans_fit_hier": [ct.POINTER(KmPoints), i32, ct.POINTER(KmHierParams), vp, vp, vp, vp, vp, vp, i32,
                                ct.POINTER(KmFitStats), vp, vp],
            "kmeans_assign_pruned": [ct.POINTER(KmPoints), vp, i32, vp, vp, vp, vp, ct.POINTER(KmPrune), vp, vp],
            "kmeans_fit_pruned": [ct.POINTER(KmPoints), i32, i32, vp, vp, vp, vp, i32, ct.POINTER(KmPrune),
                                  ct.POINTER(KmFitStats), vp, vp],
            "kmeans_cost": [vp, i64, i32, i64, vp, i32, vp, vp, vp],
            "km_release": [],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = ct.c_int
        L.km_last_error.argtypes = []
        L.km_last_error.restype = ct.c_char_p
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise KmqError(status, lib().km_last_error().decode(errors="replace"))


def _stream():
    return ct.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return None if t is None else ct.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, dtype, name: str, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


class Points:
    """Compressed points handed to the clustering calls (mirrors ``km_points``)."""

    def __init__(self, fmt: int, data: torch.Tensor, d: int, alpha=None, center=None, front=None, d_front: int = 0,
                 raw=None, vparams=None):
        self.fmt, self.data, self.d = fmt, data, d
        self.alpha, self.center, self.front, self.d_front, self.raw = alpha, center, front, d_front, raw
        self.vparams = vparams
        self.n = data.shape[0]
        ld = data.stride(0) if fmt in (KM_F32, KM_BF16, KM_SQ8, KM_LVQ4) else d // 32
        if raw is not None:
            _rows(raw, torch.float32, "raw")
            if raw.shape[0] != self.n or raw.shape[1] != d:
                raise ValueError("raw must hold the same n points with d dims")
        self._c = KmPoints(fmt, d, self.n, data.data_ptr(), ld, _ptr(alpha) or None, _ptr(center) or None,
                           _ptr(front) or None, d_front, 0, _ptr(raw) or None, raw.stride(0) if raw is not None else 0,
                           _ptr(vparams) or None)

    @property
    def ref(self):
        return ct.byref(self._c)

    @property
    def device(self):
        return self.data.device

    def centroid_dtype(self):
        return torch.uint8 if self.fmt == KM_SQ8 else torch.float32


def _rows(t: torch.Tensor, dtype, name: str):
    """A 2-D tensor whose rows are contiguous (row stride may exceed the row length)."""
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.dtype != dtype or t.dim() != 2:
        raise ValueError(f"{name} must be a 2-D {dtype} tensor on the GPU")
    if t.stride(1) != 1 or t.stride(0) < t.shape[1]:
        raise ValueError(f"{name} rows must be contiguous")
    return t


def points_f32(X: torch.Tensor) -> Points:
    """fp32 points; rows must be contiguous, the row stride may be larger than d."""
    _rows(X, torch.float32, "X")
    return Points(KM_F32, X, X.shape[1])


def points_bf16(X: torch.Tensor, raw: torch.Tensor | None = None) -> Points:
    """bfloat16 points (torch.bfloat16); rows must be contiguous, the row stride may be larger than d.
    raw: optional fp32 rows for the last update of kmeans_fit."""
    _rows(X, torch.bfloat16, "X")
    return Points(KM_BF16, X, X.shape[1], raw=raw)


def points_sq8(codes: torch.Tensor) -> Points:
    _dev(codes, torch.uint8, "codes", 2)
    return Points(KM_SQ8, codes, codes.shape[1])


def points_sign1(bits: torch.Tensor, alpha: torch.Tensor, center: torch.Tensor, d: int,
                 raw: torch.Tensor | None = None) -> Points:
    _dev(bits, torch.int32, "bits", 2)
    _dev(alpha, torch.float32, "alpha", 1)
    _dev(center, torch.float32, "center", 1)
    if bits.shape[1] != d // 32:
        raise ValueError("bits must have d/32 words per row")
    return Points(KM_SIGN1, bits, d, alpha=alpha, center=center, raw=raw)


def points_rabitq(bits: torch.Tensor, alpha: torch.Tensor, d: int, raw: torch.Tensor | None = None) -> Points:
    """RabitQ points (codes of the rotated residual, from rabitq_encode); raw: optional
    fp32 rotated residual rows (X - m) P for the last update of kmeans_fit."""
    _dev(bits, torch.int32, "bits", 2)
    _dev(alpha, torch.float32, "alpha", 1)
    if bits.shape[1] != d // 32:
        raise ValueError("bits must have d/32 words per row")
    return Points(KM_RABITQ, bits, d, alpha=alpha, raw=raw)


def points_lvq4(codes: torch.Tensor, vparams: torch.Tensor, d: int, raw: torch.Tensor | None = None) -> Points:
    """LVQ4 points: packed 4-bit codes (uint8 n x ld, ld >= d/2, two dims per byte) and
    per-vector (s, b, A, N) float32 n x 4 as quantize_lvq4 returns them; raw: optional
    fp32 rows for the last update of kmeans_fit."""
    _rows(codes, torch.uint8, "codes")
    _dev(vparams, torch.float32, "vparams", 2)
    if codes.shape[1] < d // 2 or vparams.shape != (codes.shape[0], 4):
        raise ValueError("codes must hold d/2 bytes per row and vparams n x 4 floats")
    return Points(KM_LVQ4, codes, d, raw=raw, vparams=vparams)


def points_hybrid(front: torch.Tensor, bits: torch.Tensor, alpha: torch.Tensor, center: torch.Tensor,
                  d: int, raw: torch.Tensor | None = None) -> Points:
    _dev(front, torch.float32, "front", 2)
    _dev(bits, torch.int32, "bits", 2)
    _dev(alpha, torch.float32, "alpha", 1)
    _dev(center, torch.float32, "center", 1)
    if bits.shape[1] != d // 32:
        raise ValueError("bits must have d/32 words per row")
    return Points(KM_HYBRID, bits, d, alpha=alpha, center=center, front=front, d_front=front.shape[1], raw=raw)


# --------------------------------------------------------------------------

def quantize_sq8(X: torch.Tensor, params: torch.Tensor | None = None):
    """SQ8 codes (uint8 n x d) and params (lo[d] then hi[d]); fits params unless given."""
    _dev(X, torch.float32, "X", 2)
    n, d = X.shape
    codes = torch.empty((n, d), dtype=torch.uint8, device=X.device)
    flags = 0
    if params is None:
        params = torch.empty(2 * d, dtype=torch.float32, device=X.device)
        flags = KM_Q_FIT_PARAMS
    else:
        _dev(params, torch.float32, "params", 1)
    _check(lib().quantize(_ptr(X), n, d, X.stride(0), KM_SQ8, _ptr(codes), _ptr(params), None, 0, None, flags,
                          _stream()))
    return codes, params


def rabitq_encode(X: torch.Tensor, rotation: torch.Tensor, center: torch.Tensor | None = None,
                  want_rotated: bool = False):
    """RabitQ codes of X: (bits int32 n x d/32, centre m, alpha, rotated rows or None).
    rotation: float32 d x d orthogonal P (row-major); the codes are of (X - m) P.  Fits
    m (column mean) unless given; want_rotated also returns y = (X - m) P (n x d)."""
    _dev(X, torch.float32, "X", 2)
    _dev(rotation, torch.float32, "rotation", 2)
    n, d = X.shape
    if rotation.shape != (d, d):
        raise ValueError("rotation must be d x d")
    bits = torch.empty((n, d // 32), dtype=torch.int32, device=X.device)
    alpha = torch.empty(n, dtype=torch.float32, device=X.device)
    flags = 0
    if center is None:
        center = torch.empty(d, dtype=torch.float32, device=X.device)
        flags = KM_Q_FIT_PARAMS
    else:
        _dev(center, torch.float32, "center", 1)
    Y = torch.empty((n, d), dtype=torch.float32, device=X.device) if want_rotated else None
    _check(lib().rabitq_encode(_ptr(X), n, d, X.stride(0), _ptr(rotation), _ptr(center), _ptr(bits), _ptr(alpha),
                               _ptr(Y), flags, _stream()))
    return bits, center, alpha, Y


def quantize_bf16(X: torch.Tensor) -> torch.Tensor:
    """bfloat16 copy of fp32 points (nearest, ties to even), n x d torch.bfloat16."""
    _dev(X, torch.float32, "X", 2)
    n, d = X.shape
    out = torch.empty((n, d), dtype=torch.bfloat16, device=X.device)
    _check(lib().quantize(_ptr(X), n, d, X.stride(0), KM_BF16, _ptr(out), None, None, 0, None, 0, _stream()))
    return out


def quantize_lvq4(X: torch.Tensor):
    """LVQ4 codes (uint8 n x d/2, two 4-bit codes per byte, low nibble first) and the
    per-vector (s, b, A, N) as float32 n x 4."""
    _dev(X, torch.float32, "X", 2)
    n, d = X.shape
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device=X.device)
    par = torch.empty((n, 4), dtype=torch.float32, device=X.device)
    _check(lib().quantize(_ptr(X), n, d, X.stride(0), KM_LVQ4, _ptr(codes), _ptr(par), None, 0, None, 0, _stream()))
    return codes, par


def quantize_sign1(X: torch.Tensor, center: torch.Tensor | None = None, d_front: int = 0, want_front: bool = False):
    """1-bit codes (int32 n x d/32), mean m, alpha over dims [d_front, d) and optional fp32 front copy."""
    _dev(X, torch.float32, "X", 2)
    n, d = X.shape
    bits = torch.empty((n, d // 32), dtype=torch.int32, device=X.device)
    alpha = torch.empty(n, dtype=torch.float32, device=X.device)
    flags = 0
    if center is None:
        center = torch.empty(d, dtype=torch.float32, device=X.device)
        flags = KM_Q_FIT_PARAMS
    else:
        _dev(center, torch.float32, "center", 1)
    front = torch.empty((n, d_front), dtype=torch.float32, device=X.device) if (want_front and d_front) else None
    _check(lib().quantize(_ptr(X), n, d, X.stride(0), KM_SIGN1, _ptr(bits), _ptr(center), _ptr(alpha), d_front,
                          _ptr(front), flags, _stream()))
    return bits, center, alpha, front


def pca_fit_cov(X: torch.Tensor):
    _dev(X, torch.float32, "X", 2)
    n, d = X.shape
    mean = torch.empty(d, dtype=torch.float32, device=X.device)
    cov = torch.empty((d, d), dtype=torch.float32, device=X.device)
    _check(lib().pca_fit_cov(_ptr(X), n, d, _ptr(mean), _ptr(cov), _stream()))
    return mean, cov


def pca_project(X: torch.Tensor, mean: torch.Tensor, W: torch.Tensor, out: torch.Tensor | None = None):
    _dev(X, torch.float32, "X", 2)
    _dev(mean, torch.float32, "mean", 1)
    _dev(W, torch.float32, "W", 2)
    n, d = X.shape
    d_out = W.shape[1]
    if W.shape[0] != d:
        raise ValueError("W must be d x d_out")
    Y = torch.empty((n, d_out), dtype=torch.float32, device=X.device) if out is None else out
    _check(lib().pca_project(_ptr(X), n, d, _ptr(mean), _ptr(W), d_out, _ptr(Y), _stream()))
    return Y


def _check_C(P: Points, C: torch.Tensor):
    _dev(C, P.centroid_dtype(), "C", 2)
    if C.shape[1] != P.d:
        raise ValueError("C must be k x d")
    return C.shape[0]


def kmeans_assign(P: Points, C: torch.Tensor, score: bool = True, objective: bool = False):
    """(assign int32[n], score float[n] or None, objective double[1] on device or None)."""
    k = _check_C(P, C)
    a = torch.empty(P.n, dtype=torch.int32, device=P.device)
    sc = torch.empty(P.n, dtype=torch.float32, device=P.device) if score else None
    obj = torch.empty(1, dtype=torch.float64, device=P.device) if objective else None
    _check(lib().kmeans_assign(P.ref, _ptr(C), k, _ptr(a), _ptr(sc), _ptr(obj), _stream()))
    return a, sc, obj


def kmeans_assign_noalloc(P: Points, C: torch.Tensor, assign: torch.Tensor, score: torch.Tensor | None = None,
                          objective: torch.Tensor | None = None):
    """kmeans_assign into caller-given outputs, with the library's static scratch:
    assign int32[n], score float[n] or None, objective double[1] or None (device
    tensors).  The library allocates nothing for this call."""
    k = _check_C(P, C)
    _dev(assign, torch.int32, "assign", 1)
    if score is not None:
        _dev(score, torch.float32, "score", 1)
    if objective is not None:
        _dev(objective, torch.float64, "objective", 1)
    if assign.shape[0] != P.n or (score is not None and score.shape[0] != P.n) or \
            (objective is not None and objective.shape[0] != 1):
        raise ValueError("assign and score must hold n values, objective one")
    _check(lib().kmeans_assign_noalloc(P.ref, _ptr(C), k, _ptr(assign), _ptr(score), _ptr(objective), _stream()))
    return assign, score, objective


def kmeans_update(P: Points, assign: torch.Tensor, C: torch.Tensor, policy: int = KM_EMPTY_SPLIT,
                  counts: bool = True):
    """Updates C in place; returns (C, counts int64[k] or None)."""
    k = _check_C(P, C)
    _dev(assign, torch.int32, "assign", 1)
    cnt = torch.empty(k, dtype=torch.int64, device=P.device) if counts else None
    _check(lib().kmeans_update(P.ref, _ptr(assign), k, _ptr(C), _ptr(cnt), policy, _stream()))
    return C, cnt


def kmeans_fit(P: Points, k: int, iters: int, init_idx=None, C: torch.Tensor | None = None,
               policy: int = KM_EMPTY_SPLIT, objective: bool = True, assign: torch.Tensor | None = None,
               stats: KmFitStats | None = None):
    """Lloyd's algorithm on the device.  init_idx: host int64[k] (or None with C holding the start).
    stats: optional KmFitStats filled with per-stage device times (the call then waits for the stream).
    Returns (C, assign, objective double[iters+1] on device or None)."""
    if C is None:
        C = torch.empty((k, P.d), dtype=P.centroid_dtype(), device=P.device)
    else:
        _check_C(P, C)
    a = torch.empty(P.n, dtype=torch.int32, device=P.device) if assign is None else assign
    obj = torch.empty(iters + 1, dtype=torch.float64, device=P.device) if objective else None
    idx_p = None
    if init_idx is not None:
        idx = np.ascontiguousarray(np.asarray(init_idx, dtype=np.int64))
        if idx.shape != (k,):
            raise ValueError("init_idx must hold k indices")
        idx_p = idx.ctypes.data_as(ct.c_void_p)
    _check(lib().kmeans_fit(P.ref, k, iters, idx_p, _ptr(C), _ptr(a), _ptr(obj), policy,
                            ct.byref(stats) if stats is not None else None, _stream()))
    return C, a, obj


def kmeans_assign_pruned(P: Points, C: torch.Tensor, prev: torch.Tensor, eps0: float = 2.1, d_front: int = 0,
                         dist: bool = True, objective: bool = False, counters: bool = False):
    """One pruned STEP 2 from the previous assignment `prev` (fp32 or SQ8 points).
    Returns (assign, dist double[n] or None, objective double[1] or None,
    counters numpy uint64[3] or None)."""
    k = _check_C(P, C)
    _dev(prev, torch.int32, "prev", 1)
    a = torch.empty(P.n, dtype=torch.int32, device=P.device)
    dd = torch.empty(P.n, dtype=torch.float64, device=P.device) if dist else None
    obj = torch.empty(1, dtype=torch.float64, device=P.device) if objective else None
    cnt = np.zeros(3, dtype=np.uint64) if counters else None
    pr = KmPrune(eps0, d_front, 0)
    _check(lib().kmeans_assign_pruned(P.ref, _ptr(C), k, _ptr(prev), _ptr(a), _ptr(dd), _ptr(obj), ct.byref(pr),
                                      cnt.ctypes.data_as(ct.c_void_p) if counters else None, _stream()))
    return a, dd, obj, cnt


def kmeans_fit_pruned(P: Points, k: int, iters: int, init_idx=None, C: torch.Tensor | None = None,
                      policy: int = KM_EMPTY_SPLIT, eps0: float = 2.1, d_front: int = 0, objective: bool = True,
                      stats: KmFitStats | None = None, counters: bool = False):
    """Lloyd with dimension pruning in every assignment pass after the first.
    Returns (C, assign, objective double[iters+1] or None, counters numpy uint64[3] or None)."""
    if C is None:
        C = torch.empty((k, P.d), dtype=P.centroid_dtype(), device=P.device)
    else:
        _check_C(P, C)
    a = torch.empty(P.n, dtype=torch.int32, device=P.device)
    obj = torch.empty(iters + 1, dtype=torch.float64, device=P.device) if objective else None
    idx_p = None
    if init_idx is not None:
        idx = np.ascontiguousarray(np.asarray(init_idx, dtype=np.int64))
        if idx.shape != (k,):
            raise ValueError("init_idx must hold k indices")
        idx_p = idx.ctypes.data_as(ct.c_void_p)
    cnt = np.zeros(3, dtype=np.uint64) if counters else None
    pr = KmPrune(eps0, d_front, 0)
    _check(lib().kmeans_fit_pruned(P.ref, k, iters, idx_p, _ptr(C), _ptr(a), _ptr(obj), policy, ct.byref(pr),
                                   ct.byref(stats) if stats is not None else None,
                                   cnt.ctypes.data_as(ct.c_void_p) if counters else None, _stream()))
    return C, a, obj, cnt


def kmeans_fine(P: Points, meso_assign: torch.Tensor, k_meso: int, k: int, iters: int,
                C: torch.Tensor | None = None, policy: int = KM_EMPTY_SPLIT, objective: bool = False,
                sqrt_rule: bool = False):
    """FINE-CLUSTERING inside each meso-cluster (hierarchical k-means).  C given: the
    initial fine centroids (k rows); otherwise they are taken from the points.
    sqrt_rule: k_i = round(sqrt(n_i)) (the paper's counts), k being the capacity of C;
    the returned C then holds the k_fine.sum() fine centroids made.
    Returns (C, assign int32[n], k_fine numpy int32[k_meso], objective double[1] or None)."""
    _dev(meso_assign, torch.int32, "meso_assign", 1)
    if meso_assign.shape[0] != P.n:
        raise ValueError("meso_assign must hold n ids")
    flags = 0
    if C is None:
        C = torch.empty((k, P.d), dtype=P.centroid_dtype(), device=P.device)
    else:
        if _check_C(P, C) != k:
            raise ValueError("C must hold k rows")
        flags = KM_FINE_C_GIVEN
    a = torch.empty(P.n, dtype=torch.int32, device=P.device)
    kf = np.zeros(k_meso, dtype=np.int32)
    obj = torch.empty(1, dtype=torch.float64, device=P.device) if objective else None
    if sqrt_rule:
        flags |= KM_FINE_SQRT
    _check(lib().kmeans_fine(P.ref, _ptr(meso_assign), k_meso, k, iters, flags, _ptr(C), _ptr(a),
                             kf.ctypes.data_as(ct.c_void_p), _ptr(obj), policy, _stream()))
    return (C[:int(kf.sum())] if sqrt_rule else C), a, kf, obj


def kmeans_fit_hier(P: Points, k: int, init_meso, iters_meso: int, iters_fine: int, iters_refine: int = 0,
                    k_meso: int = 0, policy: int = KM_EMPTY_SPLIT, objective: bool = True,
                    stats: KmFitStats | None = None, phases: bool = False, meso: bool = False,
                    sqrt_rule: bool = False):
    """Hierarchical k-means: meso Lloyd with k_meso (0 = round(sqrt(k))) centroids from
    the rows init_meso, Lloyd inside every meso-cluster, optional vanilla refinement.
    sqrt_rule: the paper's fine counts round(sqrt(n_i)); k is then the capacity of C
    and the returned C holds the k_fine.sum() centroids made.
    Returns (C, assign, k_fine numpy int32[k_meso], objective double[1] or None,
    phase times [meso, fine, refine] in ms or None); with meso=True the meso
    assignment (int32[n]) is appended."""
    idx = np.ascontiguousarray(np.asarray(init_meso, dtype=np.int64))
    km = k_meso if k_meso else len(idx)
    if idx.ndim != 1 or len(idx) != km:
        raise ValueError("init_meso must hold k_meso indices")
    hp = KmHierParams(k_meso, iters_meso, iters_fine, iters_refine, KM_FINE_SQRT if sqrt_rule else 0)
    C = torch.empty((k, P.d), dtype=P.centroid_dtype(), device=P.device)
    a = torch.empty(P.n, dtype=torch.int32, device=P.device)
    kf = np.zeros(len(idx), dtype=np.int32)
    obj = torch.empty(1, dtype=torch.float64, device=P.device) if objective else None
    ph = np.zeros(3, dtype=np.float64) if phases else None
    am = torch.empty(P.n, dtype=torch.int32, device=P.device) if meso else None
    _check(lib().kmeans_fit_hier(P.ref, k, ct.byref(hp), idx.ctypes.data_as(ct.c_void_p), _ptr(C), _ptr(a), _ptr(am),
                                 kf.ctypes.data_as(ct.c_void_p), _ptr(obj), policy,
                                 ct.byref(stats) if stats is not None else None,
                                 ph.ctypes.data_as(ct.c_void_p) if phases else None, _stream()))
    if sqrt_rule:
        C = C[:int(kf.sum())]
    return (C, a, kf, obj, ph, am) if meso else (C, a, kf, obj, ph)


def kmeans_cost(X: torch.Tensor, C: torch.Tensor, assign: torch.Tensor):
    """sum ||x - c_a||^2 (fp64, device tensor of 1)."""
    _dev(X, torch.float32, "X", 2)
    _dev(C, torch.float32, "C", 2)
    _dev(assign, torch.int32, "assign", 1)
    out = torch.empty(1, dtype=torch.float64, device=X.device)
    _check(lib().kmeans_cost(_ptr(X), X.shape[0], X.shape[1], X.stride(0), _ptr(C), C.shape[0], _ptr(assign),
                             _ptr(out), _stream()))
    return out


def release():
    _check(lib().km_release())
