"""Chunk-deterministic Gaussian-mixture generator (numpy PCG64).

Recipe (stated once so both sides of every parity test draw identical inputs):

* ``default_rng(seed)`` draws the K component means (``N(0, 1)`` per dim, scaled
  by ``sqrt(lam_i)``) and then one uniform label in ``[0, K)`` per point.
* Points are produced in chunks of ``CHUNK`` (131072) rows; chunk ``c`` draws its noise
  from ``default_rng(SeedSequence(seed).spawn(n_chunks)[c])`` so any chunk can be
  regenerated on its own.  ``x = mu[label] + sigma * sqrt(lam) * z``.
* Optional row normalisation to unit L2 norm, applied after scaling.
* Arithmetic in float64, cast to float32 at the end.
* Initial centroids: ``default_rng(seed + 1).choice(N, k, replace=False)`` in
  draw order (random sampling of k points, the paper's STEP 1, Sec. 2.3).

The per-dim variance profile ``lam_i = i**-power`` (i = 1..d) gives the decaying
spectrum used for the PCA workload; ``power = 0`` is isotropic.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, replace

import numpy as np

CHUNK = 1 << 17  # 131072 rows


@dataclass(frozen=True)
class MixtureSpec:
    n: int
    d: int
    components: int
    sigma: float
    normalize: bool
    power: float = 0.0  # per-dim variance lam_i = i**-power
    seed: int = 0

    def with_n(self, n: int) -> "MixtureSpec":
        return replace(self, n=n)


def _lam(spec: MixtureSpec) -> np.ndarray:
    i = np.arange(1, spec.d + 1, dtype=np.float64)
    return i ** (-spec.power) if spec.power else np.ones(spec.d)


def _means_labels(spec: MixtureSpec):
    rng = np.random.default_rng(spec.seed)
    scale = np.sqrt(_lam(spec))
    means = rng.standard_normal((spec.components, spec.d)) * scale
    labels = rng.integers(0, spec.components, size=spec.n)
    return means, labels, scale


def n_chunks(spec: MixtureSpec) -> int:
    return max(1, -(-spec.n // CHUNK))


SUB = 16384  # rows drawn per call; consecutive draws continue the same stream


def make_chunk(spec: MixtureSpec, c: int, _ml=None, out: np.ndarray | None = None) -> np.ndarray:
    """Rows [c*CHUNK, min(n, (c+1)*CHUNK)) as float32, regenerated independently."""
    means, labels, scale = _ml if _ml is not None else _means_labels(spec)
    lo = c * CHUNK
    hi = min(spec.n, lo + CHUNK)
    ss = np.random.SeedSequence(spec.seed).spawn(n_chunks(spec))[c]
    rng = np.random.default_rng(ss)
    if out is None:
        out = np.empty((hi - lo, spec.d), dtype=np.float32)
    buf = np.empty((min(SUB, hi - lo), spec.d))
    for s0 in range(0, hi - lo, SUB):
        s1 = min(hi - lo, s0 + SUB)
        z = rng.standard_normal((s1 - s0, spec.d))
        z *= spec.sigma * scale
        g = buf[:s1 - s0]
        np.take(means, labels[lo + s0:lo + s1], axis=0, out=g)
        z += g
        if spec.normalize:
            nrm = np.sqrt(np.einsum("ij,ij->i", z, z))
            nrm[nrm == 0] = 1.0
            z /= nrm[:, None]
        out[s0:s1] = z
    return out


def make_points(spec: MixtureSpec, out: np.ndarray | None = None, threads: int | None = None) -> np.ndarray:
    """All N rows as a C-contiguous float32 array (chunks generated in parallel)."""
    if out is None:
        out = np.empty((spec.n, spec.d), dtype=np.float32)
    ml = _means_labels(spec)
    nc = n_chunks(spec)

    def work(c):
        lo = c * CHUNK
        make_chunk(spec, c, ml, out=out[lo:min(spec.n, lo + CHUNK)])

    threads = threads or min(16, os.cpu_count() or 1, nc)
    if threads <= 1 or nc == 1:
        for c in range(nc):
            work(c)
    else:
        with _cf.ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nc)))
    return out


def for_each_chunk(spec: MixtureSpec, fn, threads: int | None = None):
    """Call fn(row0, rows_f32) for every chunk (in parallel threads), without holding all rows."""
    ml = _means_labels(spec)
    nc = n_chunks(spec)

    def work(c):
        fn(c * CHUNK, make_chunk(spec, c, ml))

    threads = threads or min(16, os.cpu_count() or 1, nc)
    if threads <= 1 or nc == 1:
        for c in range(nc):
            work(c)
    else:
        with _cf.ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nc)))


def random_rotation(d: int, seed: int = 7) -> np.ndarray:
    """A seeded random orthogonal d x d matrix (Haar measure: QR of a Gaussian matrix
    with the signs of R's diagonal folded into Q), fp32.  The random rotation the
    1-bit codes are taken after is an input drawn here, shared by both sides."""
    g = np.random.default_rng(seed).standard_normal((d, d))
    q, r = np.linalg.qr(g)
    q *= np.sign(np.diag(r))[None, :]
    return np.ascontiguousarray(q, dtype=np.float32)


def init_indices(n: int, k: int, seed: int = 0) -> np.ndarray:
    """k distinct row indices drawn at random (Forgy initialisation)."""
    return np.random.default_rng(seed + 1).choice(n, k, replace=False).astype(np.int64)


# The five workloads: (generator spec, k, Lloyd iterations, formats/preprocessing).
CONFIGS = {
    1: dict(name="gmm20k_d128_k64_f32", spec=MixtureSpec(20_000, 128, 64, 0.3, False), k=64, iters=10,
            formats=("f32",)),
    2: dict(name="gmm1m_d768_k1000_f32_sq8", spec=MixtureSpec(1_000_000, 768, 1000, 0.15, True), k=1000, iters=20,
            formats=("f32", "sq8")),
    3: dict(name="gmm1m_d1024_k1024_sign1", spec=MixtureSpec(1_000_000, 1024, 1024, 0.15, True), k=1024, iters=20,
            formats=("sign1",)),
    4: dict(name="gmm10m_d1024_pca256_k4096", spec=MixtureSpec(10_000_000, 1024, 4096, 0.15, True, power=0.5),
            k=4096, iters=10, formats=("pca",), d_out=256),
    5: dict(name="gmm10m_d1024_front384_sign1_k4096", spec=MixtureSpec(10_000_000, 1024, 4096, 0.15, True, power=0.5),
            k=4096, iters=10, formats=("hybrid",), d_front=384),
}


def config(i: int) -> dict:
    return CONFIGS[i]
