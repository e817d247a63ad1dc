"""Helpers for the GPU parity tests (tolerances and comparisons against the oracle).

Tolerances (stated once, used by every parity test):
* integer / 1-bit paths: assignments, integer codes and counts bit-exact; 1-bit
  scores bit-exact (both sides evaluate the same fp32 expression);
* fp paths: >= 99.9 % of assignments equal (checked when n >= 1000), and every
  disagreement is a near tie: the oracle's fp64 distances to the two candidates
  differ by at most 1e-5 of the terms that cancel in ||c||^2 - 2<x,c> (that is
  ||x||^2 + ||c||^2), the resolution of an fp32 GEMM-form distance;
* centroids: per centroid ||dC_j|| / ||C_j|| <= 1e-4 given identical assignments;
* objectives: |dJ| / J <= 1e-4.
"""
import numpy as np
import pytest

FP_AGREE = 0.999
NEAR_TIE_REL = 1e-5
CENT_REL = 1e-4
OBJ_REL = 1e-4


def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def to_dev(a, torch):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    return t.detach().cpu().numpy()


def say(msg):
    print(msg, flush=True)


def assert_fp_assign(a_gpu, a_orc, d_of, label=""):
    """a_gpu/a_orc: int arrays; d_of(rows, cands) -> (fp64 distance, magnitude of the cancelling
    terms) of each row to its candidate."""
    a_gpu = np.asarray(a_gpu)
    a_orc = np.asarray(a_orc)
    mis = np.nonzero(a_gpu != a_orc)[0]
    agree = 1.0 - len(mis) / max(1, len(a_orc))
    if len(mis):
        dg, sg = d_of(mis, a_gpu[mis])
        do, so = d_of(mis, a_orc[mis])
        rel = np.abs(dg - do) / np.maximum(np.maximum(sg, so), 1e-30)
        assert (rel <= NEAR_TIE_REL).all(), f"{label}: mismatch that is not a near tie, rel gap {rel.max():.3e}"
    if len(a_orc) >= 1000:
        assert agree >= FP_AGREE, f"{label}: agreement {agree:.6f} < {FP_AGREE}"
    return agree


def assert_centroids(C_gpu, C_orc, label="", rel=CENT_REL):
    C_gpu = np.asarray(C_gpu, dtype=np.float64)
    C_orc = np.asarray(C_orc, dtype=np.float64)
    num = np.linalg.norm(C_gpu - C_orc, axis=1)
    den = np.maximum(np.linalg.norm(C_orc, axis=1), 1e-30)
    worst = (num / den).max()
    assert worst <= rel, f"{label}: centroid rel error {worst:.3e} > {rel}"
    return worst


def f32_dist(X, C):
    X = np.asarray(X, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)

    def d_of(rows, cands):
        return ((X[rows] - C[cands]) ** 2).sum(1), (X[rows] ** 2).sum(1) + (C[cands] ** 2).sum(1)
    return d_of


def unpack_bits(bits, d):
    b = np.asarray(bits).view(np.uint32)
    return ((b[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(b.shape[0], d).astype(np.int8)
