"""CPU oracle for Lloyd k-means on compressed vectors -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never calls it.

Thin numpy/ctypes layer over ``libkmq_oracle.so`` (plain C, fp64 sums, exact
integer paths; see ``kmq_oracle.h`` for the definition each routine follows) plus
the Lloyd driver (Sec. 2.3: STEP 1 random init, T x (STEP 2 assign, STEP 3
update), then one more STEP 2) and the PCA eigensolve (numpy ``eigh``).
"""
from __future__ import annotations

import ctypes as ct
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# KMQ_ORACLE_LIB names another build of kmq_oracle.c (a sanitizer build in the tests)
_LIB_PATH = os.environ.get("KMQ_ORACLE_LIB") or os.path.join(HERE, "libkmq_oracle.so")
_lib = None

EMPTY_SPLIT = 0
EMPTY_KEEP = 1

_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(np.uint8, flags="C_CONTIGUOUS")
_u16p = np.ctypeslib.ndpointer(np.uint16, flags="C_CONTIGUOUS")
_i8p = np.ctypeslib.ndpointer(np.int8, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(np.uint32, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")
_i64 = ct.c_int64
_i32 = ct.c_int32


def _null(dtype):
    return np.ctypeslib.ndpointer(dtype, flags="C_CONTIGUOUS")


def _centroid_rows(C, k: int, d: int):
    """The update writes k rows of d values into C: refuse a C of another shape
    before the C code can run past it."""
    if C.shape != (k, d):
        raise ValueError(f"centroids of shape {C.shape} for k = {k}, d = {d}")
    return C


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = ct.CDLL(_LIB_PATH)
        sig = {
            "orc_sq8_fit": [_f32p, _i64, _i32, _f32p, _f32p],
            "orc_sq8_encode": [_f32p, _i64, _i32, _f32p, _f32p, _u8p],
            "orc_col_mean": [_f32p, _i64, _i32, _f32p],
            "orc_bf16_round": [_f32p, _i64, _u16p],
            "orc_sign1_encode": [_f32p, _i64, _i32, _f32p, _i32, _u32p, _f32p],
            "orc_sign1_decode": [_u32p, _f32p, _i64, _i32, _i32, _f32p, _f32p, _i64],
            "orc_pca_cov": [_f32p, _i64, _i32, _f64p, _f64p],
            "orc_pca_cov_entry": [_f32p, _i64, _i32, _f64p, _i32, _i32],
            "orc_project": [_f32p, _i64, _i32, _f32p, _f32p, _i32, _f32p],
            "orc_assign_f32": [_f32p, _i64, _i32, _i64, _f32p, _i32, _i32p, _f64p],
            "orc_assign_sq8": [_u8p, _i64, _i32, _u8p, _i32, _i32p, _i64p],
            "orc_sign1_prep": [_f32p, _i32, _i32, _f32p, _i32, _i8p, _f32p, _i32p, _i32p, _f32p],
            "orc_assign_sign1": [_u32p, _f32p, _i64, _i32, _i32, _i8p, _f32p, _i32p, _f32p, _i32, _i32p,
                                 _f32p, _f64p],
            "orc_rabitq_prep": [_f32p, _i32, _i32, _i8p, _f32p, _f32p, _i32p, _f32p],
            "orc_assign_rabitq": [_u32p, _f32p, _i64, _i32, _i8p, _f32p, _f32p, _i32p, _f32p, _i32, _i32p, _f32p,
                                  _f64p],
            "orc_lvq4_encode": [_f32p, _i64, _i32, _u8p, _f32p],
            "orc_lvq4_decode": [_u8p, _f32p, _i64, _i32, _f32p],
            "orc_assign_lvq4": [_u8p, _f32p, _i64, _i32, _u8p, _f32p, _i32p, _i32, _i32p, _f32p, _f64p],
            "orc_update_lvq4": [_u8p, _f32p, _i64, _i32, _i32p, _i32, _f32p, _i64p, _i32],
            "orc_assign_hybrid": [_f32p, _u32p, _f32p, _i64, _i32, _i32, _f32p, _i8p, _f32p, _i32p, _f32p,
                                  _i32, _i32p, _f64p],
            "orc_update_f32": [_f32p, _i64, _i32, _i64, _i32p, _i32, _f32p, _i64p, _i32],
            "orc_update_sq8": [_u8p, _i64, _i32, _i32p, _i32, _u8p, _i64p, _i32],
            "orc_update_sign1": [ct.c_void_p, _u32p, _f32p, _i64, _i32, _i32, _f32p, _i32p, _i32, _f32p, _i64p,
                                 _i32],
            "orc_cost_f32": [_f32p, _i64, _i32, _i64, _f32p, _i32p],
            "orc_partition_cost": [_f32p, _i64, _i32, _i32p, _i32],
            "orc_prune_factor": [_i32, _i32, ct.c_double],
            "orc_assign_pruned_f32": [_f32p, _i64, _i32, _f32p, _i32, _i32p, ct.c_double, _i32, _i32, _i32p, _f64p,
                                      _i64p],
            "orc_assign_pruned_sq8": [_u8p, _i64, _i32, _u8p, _i32, _i32p, ct.c_double, _i32, _i32, _i32p, _i64p,
                                      _i64p],
            "orc_num_threads": [],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = None
        L.orc_pca_cov_entry.restype = ct.c_double
        L.orc_cost_f32.restype = ct.c_double
        L.orc_partition_cost.restype = ct.c_double
        L.orc_num_threads.restype = ct.c_int
        L.orc_prune_factor.restype = ct.c_double
        _lib = L
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return lib().orc_num_threads()


# --------------------------------------------------------------------------
# Preprocessing (Sec. 3.1)

def sq8_fit(X):
    X = _c(X, np.float32)
    n, d = X.shape
    lo = np.empty(d, np.float32)
    hi = np.empty(d, np.float32)
    lib().orc_sq8_fit(X, n, d, lo, hi)
    return lo, hi


def sq8_encode(X, lo, hi):
    X = _c(X, np.float32)
    n, d = X.shape
    codes = np.empty((n, d), np.uint8)
    lib().orc_sq8_encode(X, n, d, _c(lo, np.float32), _c(hi, np.float32), codes)
    return codes


def col_mean(X):
    X = _c(X, np.float32)
    n, d = X.shape
    m = np.empty(d, np.float32)
    lib().orc_col_mean(X, n, d, m)
    return m


def sign1_encode(X, m, d0: int = 0):
    """Bits of x - m for all d dims (n x d/32 uint32, LSB first) and alpha over dims [d0, d)."""
    X = _c(X, np.float32)
    n, d = X.shape
    assert d % 32 == 0 and d0 % 32 == 0
    bits = np.empty((n, d // 32), np.uint32)
    alpha = np.empty(n, np.float32)
    lib().orc_sign1_encode(X, n, d, _c(m, np.float32), d0, bits, alpha)
    return bits, alpha


def sign1_decode(bits, alpha, d: int, m, d0: int = 0):
    """Decoded vectors m + alpha (2b - 1) on dims [d0, d) (fp32, n x d; front dims left 0)."""
    bits = _c(bits, np.uint32)
    n = bits.shape[0]
    out = np.zeros((n, d), np.float32)
    lib().orc_sign1_decode(bits, _c(alpha, np.float32), n, d, d0, _c(m, np.float32), out, d)
    return out


def bf16_round(X):
    """Nearest bfloat16 of every value (ties to even), as uint16 bit patterns of X's shape."""
    X = _c(X, np.float32)
    out = np.empty(X.shape, np.uint16)
    lib().orc_bf16_round(X.reshape(-1), X.size, out.reshape(-1))
    return out


def bf16_decode(codes):
    """fp32 values of bfloat16 bit patterns (the pattern is the top half of the fp32 one)."""
    codes = np.asarray(codes, dtype=np.uint16)
    return (codes.astype(np.uint32) << np.uint32(16)).view(np.float32)


def pca_cov(X):
    X = _c(X, np.float32)
    n, d = X.shape
    mean = np.empty(d, np.float64)
    cov = np.empty((d, d), np.float64)
    lib().orc_pca_cov(X, n, d, mean, cov)
    return mean, cov


def col_mean64(X):
    """fp64 column mean (for sampled covariance entries)."""
    return np.asarray(X, dtype=np.float64).mean(axis=0)


def pca_cov_entry(X, mean64, i: int, j: int) -> float:
    X = _c(X, np.float32)
    n, d = X.shape
    return lib().orc_pca_cov_entry(X, n, d, _c(mean64, np.float64), i, j)


def pca_basis(cov, d_out: int):
    """Top-d_out eigenvectors of the covariance as columns (d x d_out, fp32), eigenvalues
    sorted descending; each eigenvector's largest-|.| entry is made positive."""
    w, V = np.linalg.eigh(np.asarray(cov, dtype=np.float64))
    order = np.argsort(w)[::-1]
    w = w[order]
    V = V[:, order]
    piv = np.argmax(np.abs(V), axis=0)
    sgn = np.sign(V[piv, np.arange(V.shape[1])])
    sgn[sgn == 0] = 1.0
    V = V * sgn
    return np.ascontiguousarray(V[:, :d_out], dtype=np.float32), w


def project(X, mean, W):
    X = _c(X, np.float32)
    W = _c(W, np.float32)
    n, d = X.shape
    dout = W.shape[1]
    Y = np.empty((n, dout), np.float32)
    lib().orc_project(X, n, d, _c(mean, np.float32), W, dout, Y)
    return Y


# --------------------------------------------------------------------------
# STEP 2

def assign_f32(X, C):
    X = _c(X, np.float32)
    C = _c(C, np.float32)
    n, d = X.shape
    a = np.empty(n, np.int32)
    dist = np.empty(n, np.float64)
    lib().orc_assign_f32(X, n, d, d, C, C.shape[0], a, dist)
    return a, dist


def assign_bf16(codes, C):
    """bfloat16 points: the fp32 step on the stored values and on the centroids rounded
    to bfloat16 (products of bfloat16 values are exact in fp64)."""
    return assign_f32(bf16_decode(codes), bf16_decode(bf16_round(C)))


def assign_sq8(codes, Cc):
    codes = _c(codes, np.uint8)
    Cc = _c(Cc, np.uint8)
    n, d = codes.shape
    a = np.empty(n, np.int32)
    dist = np.empty(n, np.int64)
    lib().orc_assign_sq8(codes, n, d, Cc, Cc.shape[0], a, dist)
    return a, dist


def sign1_prep(C, m, d0: int = 0):
    """Per-centroid symmetric int8 quantisation of the residual C - m on dims [d0, d)."""
    C = _c(C, np.float32)
    k, d = C.shape
    q = np.empty((k, d - d0), np.int8)
    sigma = np.empty(k, np.float32)
    T = np.empty(k, np.int32)
    Q = np.empty(k, np.int32)
    u = np.empty(k, np.float32)
    lib().orc_sign1_prep(C, k, d, _c(m, np.float32), d0, q, sigma, T, Q, u)
    return q, sigma, T, Q, u


def assign_sign1(bits, alpha, C, m, d0: int = 0):
    bits = _c(bits, np.uint32)
    C = _c(C, np.float32)
    n = bits.shape[0]
    k, d = C.shape
    q, sigma, T, Q, u = sign1_prep(C, m, d0)
    a = np.empty(n, np.int32)
    score = np.empty(n, np.float32)
    dist = np.empty(n, np.float64)
    lib().orc_assign_sign1(bits, _c(alpha, np.float32), n, d, d0, q, sigma, T, u, k, a, score, dist)
    return a, score, dist


def rabitq_prep(C):
    """Per-centroid SQ4 code of the centroid residuals (rotated space, centre 0)."""
    C = _c(C, np.float32)
    k, d = C.shape
    q = np.empty((k, d), np.int8)
    s = np.empty(k, np.float32)
    b = np.empty(k, np.float32)
    T = np.empty(k, np.int32)
    N = np.empty(k, np.float32)
    lib().orc_rabitq_prep(C, k, d, q, s, b, T, N)
    return q, s, b, T, N


def assign_rabitq(bits, alpha, C):
    """(assignments, winning fp32 scores, alpha^2 d + score in fp64)."""
    bits = _c(bits, np.uint32)
    C = _c(C, np.float32)
    n = bits.shape[0]
    k, d = C.shape
    q, s, b, T, N = rabitq_prep(C)
    a = np.empty(n, np.int32)
    score = np.empty(n, np.float32)
    dist = np.empty(n, np.float64)
    lib().orc_assign_rabitq(bits, _c(alpha, np.float32), n, d, q, s, b, T, N, k, a, score, dist)
    return a, score, dist


def lvq4_encode(X):
    """LVQ4 codes (uint8 n x d, one code per byte) and per-vector (s, b, A, N), float n x 4."""
    X = _c(X, np.float32)
    n, d = X.shape
    codes = np.empty((n, d), np.uint8)
    par = np.empty((n, 4), np.float32)
    lib().orc_lvq4_encode(X, n, d, codes, par)
    return codes, par


def lvq4_decode(codes, par):
    codes = _c(codes, np.uint8)
    n, d = codes.shape
    out = np.empty((n, d), np.float32)
    lib().orc_lvq4_decode(codes, _c(par, np.float32), n, d, out)
    return out


def lvq4_pack(codes):
    """Two 4-bit codes per byte: dim 2i in the low nibble, dim 2i+1 in the high one."""
    codes = np.asarray(codes, dtype=np.uint8)
    return np.ascontiguousarray(codes[:, 0::2] | (codes[:, 1::2] << 4))


def assign_lvq4(codes, par, C):
    """Points as LVQ4 codes; centroids C (fp32) coded with LVQ4 for the pass."""
    codes = _c(codes, np.uint8)
    n, d = codes.shape
    yc, ypar = lvq4_encode(C)
    yS = yc.astype(np.int32).sum(1).astype(np.int32)
    a = np.empty(n, np.int32)
    score = np.empty(n, np.float32)
    dist = np.empty(n, np.float64)
    lib().orc_assign_lvq4(codes, _c(par, np.float32), n, d, yc, ypar, yS, len(C), a, score, dist)
    return a, score, dist


def assign_hybrid(front, bits, alpha, C, m, d0: int):
    front = _c(front, np.float32)
    bits = _c(bits, np.uint32)
    C = _c(C, np.float32)
    n = bits.shape[0]
    k, d = C.shape
    assert front.shape == (n, d0)
    q, sigma, T, Q, u = sign1_prep(C, m, d0)
    a = np.empty(n, np.int32)
    dist = np.empty(n, np.float64)
    lib().orc_assign_hybrid(front, bits, _c(alpha, np.float32), n, d, d0, C, q, sigma, T, u, k, a, dist)
    return a, dist


# --------------------------------------------------------------------------
# STEP 3

def update_f32(X, a, k: int, C_old, policy: int = EMPTY_SPLIT):
    X = _c(X, np.float32)
    n, d = X.shape
    C = _centroid_rows(np.array(C_old, dtype=np.float32, copy=True, order="C"), k, d)
    counts = np.empty(k, np.int64)
    lib().orc_update_f32(X, n, d, d, _c(a, np.int32), k, C, counts, policy)
    return C, counts


def update_bf16(codes, a, k: int, C_old, policy: int = EMPTY_SPLIT):
    """bfloat16 points: fp32 centroids = mean of the stored (decoded) member values."""
    return update_f32(bf16_decode(codes), a, k, C_old, policy)


def update_lvq4(codes, par, a, k: int, C_old, policy: int = EMPTY_SPLIT):
    codes = _c(codes, np.uint8)
    n, d = codes.shape
    C = _centroid_rows(np.array(C_old, dtype=np.float32, copy=True, order="C"), k, d)
    counts = np.empty(k, np.int64)
    lib().orc_update_lvq4(codes, _c(par, np.float32), n, d, _c(a, np.int32), k, C, counts, policy)
    return C, counts


def update_sq8(codes, a, k: int, C_old, policy: int = EMPTY_SPLIT):
    codes = _c(codes, np.uint8)
    n, d = codes.shape
    C = _centroid_rows(np.array(C_old, dtype=np.uint8, copy=True, order="C"), k, d)
    counts = np.empty(k, np.int64)
    lib().orc_update_sq8(codes, n, d, _c(a, np.int32), k, C, counts, policy)
    return C, counts


def update_sign1(bits, alpha, d: int, m, a, k: int, C_old, policy: int = EMPTY_SPLIT, front=None, d0: int = 0):
    bits = _c(bits, np.uint32)
    n = bits.shape[0]
    C = _centroid_rows(np.array(C_old, dtype=np.float32, copy=True, order="C"), k, d)
    counts = np.empty(k, np.int64)
    fp = None
    if d0 > 0:
        front = _c(front, np.float32)
        assert front.shape == (n, d0)
        fp = front.ctypes.data_as(ct.c_void_p)
    lib().orc_update_sign1(fp, bits, _c(alpha, np.float32), n, d, d0, _c(m, np.float32), _c(a, np.int32), k, C,
                           counts, policy)
    return C, counts


# --------------------------------------------------------------------------
# Objective

def cost_f32(X, C, a) -> float:
    X = _c(X, np.float32)
    n, d = X.shape
    return lib().orc_cost_f32(X, n, d, d, _c(C, np.float32), _c(a, np.int32))


def partition_cost(X, a, k: int) -> float:
    """Full-precision cost of a partition: sum ||x - mean of x's cluster||^2 (fp64)."""
    X = _c(X, np.float32)
    n, d = X.shape
    return lib().orc_partition_cost(X, n, d, _c(a, np.int32), k)


# --------------------------------------------------------------------------
# Lloyd driver (Sec. 2.3)

def init_centroids(P: dict, idx):
    """STEP 1: clustering-space representation of the sampled rows."""
    idx = np.asarray(idx, dtype=np.int64)
    fmt = P["fmt"]
    if fmt == "f32":
        return np.ascontiguousarray(P["X"][idx], dtype=np.float32)
    if fmt == "sq8":
        return np.ascontiguousarray(P["codes"][idx], dtype=np.uint8)
    if fmt == "bf16":
        return np.ascontiguousarray(bf16_decode(P["codes"][idx]))
    if fmt == "sign1":
        return sign1_decode(P["bits"][idx], P["alpha"][idx], P["d"], P["m"], 0)
    if fmt == "rabitq":
        return sign1_decode(P["bits"][idx], P["alpha"][idx], P["d"], np.zeros(P["d"], np.float32), 0)
    if fmt == "lvq4":
        return lvq4_decode(P["codes"][idx], P["par"][idx])
    if fmt == "hybrid":
        d0 = P["d0"]
        C = sign1_decode(P["bits"][idx], P["alpha"][idx], P["d"], P["m"], d0)
        C[:, :d0] = P["front"][idx]
        return C
    raise ValueError(fmt)


def assign(P: dict, C):
    """(assignments, per-point in-space distance) for one STEP 2."""
    fmt = P["fmt"]
    if fmt == "f32":
        return assign_f32(P["X"], C)
    if fmt == "sq8":
        return assign_sq8(P["codes"], C)
    if fmt == "bf16":
        return assign_bf16(P["codes"], C)
    if fmt == "sign1":
        a, _, dist = assign_sign1(P["bits"], P["alpha"], C, P["m"], 0)
        return a, dist
    if fmt == "rabitq":
        a, _, dist = assign_rabitq(P["bits"], P["alpha"], C)
        return a, dist
    if fmt == "lvq4":
        a, _, dist = assign_lvq4(P["codes"], P["par"], C)
        return a, dist
    if fmt == "hybrid":
        return assign_hybrid(P["front"], P["bits"], P["alpha"], C, P["m"], P["d0"])
    raise ValueError(fmt)


def update(P: dict, a, k: int, C, policy: int = EMPTY_SPLIT):
    fmt = P["fmt"]
    if fmt == "f32":
        return update_f32(P["X"], a, k, C, policy)
    if fmt == "sq8":
        return update_sq8(P["codes"], a, k, C, policy)
    if fmt == "bf16":
        return update_bf16(P["codes"], a, k, C, policy)
    if fmt == "sign1":
        return update_sign1(P["bits"], P["alpha"], P["d"], P["m"], a, k, C, policy)
    if fmt == "rabitq":
        return update_sign1(P["bits"], P["alpha"], P["d"], np.zeros(P["d"], np.float32), a, k, C, policy)
    if fmt == "lvq4":
        return update_lvq4(P["codes"], P["par"], a, k, C, policy)
    if fmt == "hybrid":
        return update_sign1(P["bits"], P["alpha"], P["d"], P["m"], a, k, C, policy, front=P["front"], d0=P["d0"])
    raise ValueError(fmt)


def fit(P: dict, k: int, iters: int, init_idx, policy: int = EMPTY_SPLIT, C0=None):
    """Lloyd: T x (assign, update), then a final assign.  Returns (C, a, J[0..T]).

    If P holds "raw" (fp32 rows in the clustering space), the last update averages
    those instead of the compressed points (the raw-vector last iteration of
    Sec. 4.1 that removes the outward bias of decoded 1-bit codes)."""
    C = init_centroids(P, init_idx) if C0 is None else np.array(C0, copy=True)
    if len(C) != k:
        raise ValueError(f"{len(C)} initial centroids for k = {k}")
    J = []
    for t in range(iters):
        a, dist = assign(P, C)
        J.append(float(np.sum(dist, dtype=np.float64)))
        if t == iters - 1 and P.get("raw") is not None:
            C, _ = update_f32(P["raw"], a, k, C, policy)
        else:
            C, _ = update(P, a, k, C, policy)
    a, dist = assign(P, C)
    J.append(float(np.sum(dist, dtype=np.float64)))
    return C, a, J


# --------------------------------------------------------------------------
# Hierarchical k-means (Sec. 4.4 "Other Accelerators", Table 7): MESO-CLUSTERING
# of all points into about sqrt(k) clusters, FINE-CLUSTERING by Lloyd inside each
# meso-cluster, then optional iterations of vanilla Lloyd over all points with all
# k centroids.  Every Lloyd run is the driver above.

_ROW_KEYS = ("X", "codes", "bits", "alpha", "front", "par", "raw")


def n_rows(P: dict) -> int:
    for key in _ROW_KEYS:
        if P.get(key) is not None:
            return len(P[key])
    raise ValueError("no point rows")


def subset(P: dict, rows, keep_raw: bool = False):
    """The same points' format dict restricted to `rows` (in the given order)."""
    Q = dict(P)
    for key in _ROW_KEYS:
        if P.get(key) is not None:
            Q[key] = np.ascontiguousarray(P[key][rows])
    if not keep_raw:
        Q.pop("raw", None)
    return Q


def meso_count(k: int) -> int:
    """Number of meso-clusters: the integer nearest to sqrt(k) (never a tie for integer k)."""
    r = 0
    while (r + 1) * (r + 1) <= k:
        r += 1
    return max(1, r + 1 if k - r * r > r else r)


def fine_counts(n_meso, k: int):
    """Fine clusters per meso-cluster.  One for every non-empty meso-cluster, the
    remaining k - m split in proportion to n_i - 1 (floor shares, then one more for
    the largest remainders, ties to the smaller index).  Sums to k; k_i <= n_i."""
    n_meso = [int(v) for v in n_meso]
    N = sum(n_meso)
    m = sum(1 for v in n_meso if v > 0)
    if not m <= k <= N:
        raise ValueError("need (non-empty meso-clusters) <= k <= n")
    rem, cap = k - m, N - m
    ks, rems = [], []
    for v in n_meso:
        w = v - 1 if v > 0 else 0
        share, r = (divmod(rem * w, cap) if cap > 0 else (0, 0))
        ks.append((1 if v > 0 else 0) + share)
        rems.append(r)
    left = k - sum(ks)
    for i in sorted(range(len(n_meso)), key=lambda i: (-rems[i], i))[:left]:
        ks[i] += 1
    return np.asarray(ks, dtype=np.int32)


def fine_counts_sqrt(n_meso):
    """Fine clusters per meso-cluster as Sec. 4.4 states them: the integer nearest to
    sqrt(n_i) for every non-empty meso-cluster (0 for an empty one).  Exact integer
    arithmetic: r = floor(sqrt(v)), and r + 1 when v - r^2 > r (sqrt(v) > r + 1/2
    exactly then, since (r + 1/2)^2 = r^2 + r + 1/4); never a tie.  1 <= k_i <= n_i."""
    out = []
    for v in (int(x) for x in n_meso):
        if v <= 0:
            out.append(0)
            continue
        r = 0
        while (r + 1) * (r + 1) <= v:
            r += 1
        out.append(r + 1 if v - r * r > r else r)
    return np.asarray(out, dtype=np.int32)


def fine_init_positions(n_i: int, k_i: int):
    """Initial fine centroids of a meso-cluster: its members (ascending point index)
    at positions floor(j n_i / k_i), j = 0 .. k_i - 1 (distinct since k_i <= n_i)."""
    return (np.arange(k_i, dtype=np.int64) * n_i) // k_i


def fit_fine(P: dict, a_meso, k_meso: int, k: int, iters: int, policy: int = EMPTY_SPLIT, C0=None,
             sqrt_rule: bool = False):
    """FINE-CLUSTERING: Lloyd (T = iters) inside every meso-cluster i on its members,
    with k_i fine centroids (fine_counts; with sqrt_rule fine_counts_sqrt, k then
    being an upper bound on their sum); fine centroid j of meso-cluster i is global
    centroid off_i + j, off_i = k_0 + ... + k_{i-1}.  C0 (optional, sum k_i rows)
    replaces the initial centroids.  Returns (C, a, k_i, J) with C holding sum k_i
    rows and J[t] the in-space objective of pass t summed over the meso-clusters;
    points with a meso id outside [0, k_meso) get -1."""
    a_meso = np.asarray(a_meso, dtype=np.int64)
    valid = (a_meso >= 0) & (a_meso < k_meso)
    n_i = np.bincount(a_meso[valid], minlength=k_meso)
    if sqrt_rule:
        k_i = fine_counts_sqrt(n_i)
        if int(k_i.sum()) > k:
            raise ValueError("the fine counts exceed k")
        k = int(k_i.sum())
    else:
        k_i = fine_counts(n_i, k)
    off = np.concatenate([[0], np.cumsum(k_i)])
    a = np.full(len(a_meso), -1, dtype=np.int32)
    C = None
    J = np.zeros(iters + 1, dtype=np.float64)
    for i in range(k_meso):
        if n_i[i] == 0:
            continue
        rows = np.nonzero(a_meso == i)[0]
        sub = subset(P, rows)
        Ci0 = None if C0 is None else np.asarray(C0)[off[i]:off[i + 1]]
        Ci, ai, Ji = fit(sub, int(k_i[i]), iters, fine_init_positions(len(rows), int(k_i[i])), policy, C0=Ci0)
        if C is None:
            C = np.empty((k, Ci.shape[1]), dtype=Ci.dtype)
        C[off[i]:off[i + 1]] = Ci
        a[rows] = off[i] + ai
        J += np.asarray(Ji)
    return C, a, k_i, J


def fit_hier(P: dict, k: int, iters_meso: int, iters_fine: int, iters_refine: int, init_meso,
             k_meso: int = 0, policy: int = EMPTY_SPLIT, sqrt_rule: bool = False):
    """Hierarchical k-means.  MESO: Lloyd with k_meso (default meso_count(k))
    centroids on all points from the rows init_meso; FINE: fit_fine (sqrt_rule as
    there); REFINE: iters_refine vanilla Lloyd iterations over all points with all
    the fine centroids (then a final assignment), the last update from P["raw"] if
    given.  Meso and fine use the compressed points only.  Returns (C, a, J, info)
    with J the in-space objective of the returned partition."""
    km = k_meso if k_meso else meso_count(k)
    Pc = subset(P, slice(None))
    Cm, am, Jm = fit(Pc, km, iters_meso, init_meso, policy)
    C, a, k_i, Jf = fit_fine(Pc, am, km, k, iters_fine, policy, sqrt_rule=sqrt_rule)
    J = float(Jf[-1])
    if iters_refine > 0:
        C, a, Jr = fit(P, len(C), iters_refine, None, policy, C0=C)
        J = float(Jr[-1])
    return C, a, J, {"k_meso": km, "C_meso": Cm, "a_meso": am, "J_meso": Jm, "k_fine": k_i, "J_fine": Jf}


# --------------------------------------------------------------------------
# Dimension pruning inside STEP 2 (Sec. 3.1 "SuperKMeans", Table 4): the first
# pass is a full assignment; every later pass starts each point from its previous
# centroid and drops other centroids with the ADSampling test on partial distances
# over the front d' dims and then every `step` dims, comparing the survivors on the
# full distance.  Meant for randomly rotated points (the test assumes the
# variance is spread evenly over the dims).

def prune_front_dims(d: int) -> int:
    """Default d': 12.5 % of d rounded up to a multiple of 32 (at most d)."""
    return min(d, 32 * ((d + 255) // 256))


def prune_factor(D: int, d: int, eps0: float) -> float:
    return float(lib().orc_prune_factor(D, d, eps0))


def assign_pruned(P: dict, C, prev, eps0: float = 2.1, d_front: int = 0, step: int = 64):
    """One pruned STEP 2 from the previous assignment.  Returns (a, dist, counters) with
    counters = [candidates tested at d', passed d', compared on the full distance]."""
    fmt = P["fmt"]
    prev = _c(prev, np.int32)
    cnt = np.zeros(3, np.int64)
    if fmt == "f32":
        X = _c(P["X"], np.float32)
        n, d = X.shape
        D0 = d_front or prune_front_dims(d)
        a = np.empty(n, np.int32)
        dist = np.empty(n, np.float64)
        lib().orc_assign_pruned_f32(X, n, d, _c(C, np.float32), len(C), prev, eps0, D0, step, a, dist, cnt)
        return a, dist, cnt
    if fmt == "sq8":
        X = _c(P["codes"], np.uint8)
        n, d = X.shape
        D0 = d_front or prune_front_dims(d)
        a = np.empty(n, np.int32)
        dist = np.empty(n, np.int64)
        lib().orc_assign_pruned_sq8(X, n, d, _c(C, np.uint8), len(C), prev, eps0, D0, step, a, dist, cnt)
        return a, dist.astype(np.float64), cnt
    raise ValueError(f"dimension pruning is defined for f32 and sq8 points, not {fmt}")


def fit_pruned(P: dict, k: int, iters: int, init_idx, policy: int = EMPTY_SPLIT, eps0: float = 2.1,
               d_front: int = 0, step: int = 64, C0=None):
    """Lloyd with pruned assignment passes: STEP 1, a full STEP 2, then iters x
    (STEP 3, pruned STEP 2 from the previous assignment).  Returns (C, a, J[0..T],
    counters summed over the pruned passes)."""
    C = init_centroids(P, init_idx) if C0 is None else np.array(C0, copy=True)
    a, dist = assign(P, C)
    J = [float(np.sum(dist, dtype=np.float64))]
    total = np.zeros(3, np.int64)
    for _ in range(iters):
        C, _ = update(P, a, k, C, policy)
        a, dist, cnt = assign_pruned(P, C, a, eps0, d_front, step)
        J.append(float(np.sum(dist, dtype=np.float64)))
        total += cnt
    return C, a, J, total
