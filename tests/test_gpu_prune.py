"""GPU parity of dimension pruning inside STEP 2 (Sec. 3.1 SuperKMeans with the
ADSampling test) against the CPU oracle.

SQ8: distances are exact integers and the test is the same fp32 expression on
both sides, so assignments, distances, survivor counters and whole pruned Lloyd
runs are bit-exact.  fp32: the GPU sums in fp32 (the front on the matrix cores),
the oracle in fp64, so a decision can differ where it is within rounding of the
threshold; every assignment that differs must be explained by such a decision or
by a near tie (tolerances stated below), and at least 99.9 % must agree.
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import CENT_REL, assert_centroids, host, say, to_dev, torch_cuda

pytestmark = pytest.mark.gpu

# fp32 decision tolerance: relative to the magnitudes that cancel in the compared
# quantities (||x||^2 + ||c||^2 and the threshold), the resolution of fp32 sums
PRUNE_REL = 2e-5


@pytest.fixture(scope="module")
def torch():
    t = torch_cuda()
    import paper_2608_14648_amd  # noqa: F401  (fails loudly if the library is missing)
    return t


@pytest.fixture(scope="module")
def km(torch):
    import paper_2608_14648_amd as km
    km.lib()
    return km


def rotated_blobs(n, d, comps, seed, sigma=0.35):
    import synth
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((comps, d))
    X = mu[rng.integers(0, comps, n)] + sigma * rng.standard_normal((n, d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    return (X @ synth.random_rotation(d, seed % 17 + 1)).astype(np.float32)


def sq8_pair(km, torch, X):
    lo, hi = orc.sq8_fit(X)
    codes = orc.sq8_encode(X, lo, hi)
    return codes, lo, hi, km.points_sq8(to_dev(codes, torch))


SQ8_SHAPES = [(1, 16, 1, 2.1, 0), (5, 32, 3, 2.1, 0), (300, 64, 17, 0.5, 0), (1000, 128, 64, 2.1, 0),
              (2049, 256, 130, 2.1, 0), (517, 768, 257, 2.1, 0), (517, 768, 257, 1.0, 48), (700, 1024, 300, 2.1, 0),
              (300, 2048, 40, 2.1, 0), (400, 96, 20, 1e12, 0)]


@pytest.mark.parametrize("n,d,k,eps0,d_front", SQ8_SHAPES)
def test_assign_pruned_sq8_bit_exact(km, torch, n, d, k, eps0, d_front):
    say(f"pruned sq8 n={n} d={d} k={k} eps0={eps0} d_front={d_front}")
    X = rotated_blobs(n, d, max(2, k // 2), seed=n + d + k)
    codes, lo, hi, Pg = sq8_pair(km, torch, X)
    rng = np.random.default_rng(n + k)
    C = orc.sq8_encode(X[rng.integers(0, n, k)] + 0.05 * rng.standard_normal((k, d)).astype(np.float32), lo, hi)
    if k >= 4:
        C[3] = C[1]  # equal centroids: ties to the smaller index
    prev = rng.integers(0, k, n).astype(np.int32)
    a_o, dist_o, cnt_o = orc.assign_pruned({"fmt": "sq8", "codes": codes}, C, prev, eps0, d_front)
    a, dist, obj, cnt = km.kmeans_assign_pruned(Pg, to_dev(C, torch), to_dev(prev, torch), eps0, d_front,
                                                objective=True, counters=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(dist), dist_o)
    assert cnt.astype(np.int64).tolist() == cnt_o.tolist()
    assert host(obj)[0] == dist_o.sum()
    if eps0 > 1e6:  # nothing is dropped: the exact nearest centroid
        a_ex, _ = orc.assign_sq8(codes, C)
        np.testing.assert_array_equal(host(a), a_ex)


def test_fit_pruned_sq8_bit_exact(km, torch):
    """Pruned Lloyd on SQ8 codes of rotated 768-dim embeddings (fewer rows): centroids,
    assignments, objectives and counters bit-exact against the oracle."""
    import synth
    spec = synth.config(2)["spec"].with_n(30000)
    X = synth.make_points(spec) @ synth.random_rotation(spec.d, 9)
    X = X.astype(np.float32)
    codes, _, _, Pg = sq8_pair(km, torch, X)
    k, T = 300, 5
    idx = synth.init_indices(len(X), k)
    C_o, a_o, J_o, cnt_o = orc.fit_pruned({"fmt": "sq8", "codes": codes}, k, T, idx)
    C, a, J, cnt = km.kmeans_fit_pruned(Pg, k, T, idx, counters=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(C), C_o)
    np.testing.assert_array_equal(host(a), a_o)
    assert host(J).tolist() == J_o
    assert cnt.astype(np.int64).tolist() == cnt_o.tolist()
    assert cnt_o[1] < 0.3 * cnt_o[0]  # the test does drop most candidates here


def explain_f32(X, C, prev, g, o, eps0, D0):
    """True when the fp32 and fp64 choices g and o of one point differ only by a
    decision within rounding: a near tie of their full distances, or a checkpoint of
    either candidate within rounding of the threshold."""
    x = X.astype(np.float64)
    d = len(x)
    tau = ((x - C[prev].astype(np.float64)) ** 2).sum()
    full = {}
    for j in (g, o):
        diff = (x - C[j].astype(np.float64)) ** 2
        full[j] = diff.sum()
    mag = (x ** 2).sum() + max((C[g].astype(np.float64) ** 2).sum(), (C[o].astype(np.float64) ** 2).sum())
    if abs(full[g] - full[o]) <= PRUNE_REL * mag:
        return True
    for j in (g, o):
        if j == prev:
            continue
        pre = np.cumsum((x - C[j].astype(np.float64)) ** 2)
        for D in range(D0, d, 64):
            lim = tau * orc.prune_factor(D, d, eps0)
            scale = lim + (x[:D] ** 2).sum() + (C[j, :D].astype(np.float64) ** 2).sum()
            if abs(pre[D - 1] - lim) <= PRUNE_REL * scale:
                return True
    return False


def check_f32_against_oracle(X, C, prev, a, a_o, eps0, D0, label):
    mis = np.nonzero(a != a_o)[0]
    for i in mis:
        assert explain_f32(X[i], C, prev[i], a[i], a_o[i], eps0, D0), \
            f"{label}: point {i} GPU {a[i]} oracle {a_o[i]} not explained by rounding"
    if len(a) >= 1000:
        assert 1 - len(mis) / len(a) >= 0.999, f"{label}: agreement {1 - len(mis) / len(a)}"
    return len(mis)


F32_SHAPES = [(1, 32, 1, 0), (5, 64, 3, 0), (300, 96, 17, 0), (1000, 128, 64, 0), (2049, 256, 130, 0),
              (517, 768, 257, 0), (517, 768, 257, 40), (700, 1024, 300, 0), (300, 2048, 40, 0), (400, 136, 50, 8)]


@pytest.mark.parametrize("n,d,k,d_front", F32_SHAPES)
def test_assign_pruned_f32(km, torch, n, d, k, d_front):
    say(f"pruned f32 n={n} d={d} k={k} d_front={d_front}")
    X = rotated_blobs(n, d, max(2, k // 2), seed=n + d + k + 1)
    rng = np.random.default_rng(n + k + 1)
    C = (X[rng.integers(0, n, k)] + 0.05 * rng.standard_normal((k, d))).astype(np.float32)
    prev = rng.integers(0, k, n).astype(np.int32)
    D0 = d_front or orc.prune_front_dims(d)
    a_o, dist_o, cnt_o = orc.assign_pruned({"fmt": "f32", "X": X}, C, prev, 2.1, d_front)
    a, dist, obj, cnt = km.kmeans_assign_pruned(km.points_f32(to_dev(X, torch)), to_dev(C, torch),
                                                to_dev(prev, torch), 2.1, d_front, objective=True, counters=True)
    torch.cuda.synchronize()
    a, dist = host(a), host(dist)
    nmis = check_f32_against_oracle(X, C, prev, a, a_o, 2.1, D0, f"n={n} d={d} k={k}")
    same = a == a_o
    np.testing.assert_allclose(dist[same], dist_o[same], rtol=1e-5, atol=1e-6)
    # survivor counts differ only by decisions within rounding
    assert np.all(np.abs(cnt.astype(np.int64) - cnt_o) <= 2 + 1e-3 * cnt_o)
    assert abs(host(obj)[0] - dist_o.sum()) <= 1e-5 * dist_o.sum() + 1e-6 + nmis * 4.0


def test_assign_pruned_f32_without_pruning_is_exact(km, torch):
    n, d, k = 2000, 256, 100
    X = rotated_blobs(n, d, 40, seed=5)
    rng = np.random.default_rng(6)
    C = (X[rng.integers(0, n, k)] + 0.05 * rng.standard_normal((k, d))).astype(np.float32)
    prev = rng.integers(0, k, n).astype(np.int32)
    a, _, _, cnt = km.kmeans_assign_pruned(km.points_f32(to_dev(X, torch)), to_dev(C, torch), to_dev(prev, torch),
                                           1e12, counters=True)
    a_o, _ = orc.assign_f32(X, C)
    torch.cuda.synchronize()
    assert cnt[0] == cnt[1] == cnt[2] == n * (k - 1)
    mis = np.nonzero(host(a) != a_o)[0]
    for i in mis:
        assert explain_f32(X[i], C, prev[i], host(a)[i], a_o[i], 1e12, orc.prune_front_dims(d))


def test_fit_pruned_f32_lockstep(km, torch):
    """Pruned Lloyd on rotated fp32 embeddings: each pruned pass from the oracle's
    centroids and previous assignment (explained mismatches only), each update from
    the oracle's assignment; the fit's first pass and objective agree."""
    import synth
    spec = synth.config(2)["spec"].with_n(20000)
    X = (synth.make_points(spec) @ synth.random_rotation(spec.d, 9)).astype(np.float32)
    Po = {"fmt": "f32", "X": X}
    Pg = km.points_f32(to_dev(X, torch))
    k, T = 200, 4
    D0 = orc.prune_front_dims(spec.d)
    idx = synth.init_indices(len(X), k)
    C_o = orc.init_centroids(Po, idx)
    a_o, _ = orc.assign(Po, C_o)
    for t in range(T):
        say(f"pruned f32 lockstep step {t}")
        C_n, _ = orc.update(Po, a_o, k, C_o)
        C = to_dev(C_o, torch)
        km.kmeans_update(Pg, to_dev(a_o, torch), C)
        torch.cuda.synchronize()
        assert_centroids(host(C), C_n, f"update {t}", rel=CENT_REL)
        a_n, _, _ = orc.assign_pruned(Po, C_n, a_o, 2.1)
        a, _, _, _ = km.kmeans_assign_pruned(Pg, to_dev(C_n, torch), to_dev(a_o, torch), 2.1)
        torch.cuda.synchronize()
        check_f32_against_oracle(X, C_n, a_o, host(a), a_n, 2.1, D0, f"pass {t + 1}")
        C_o, a_o = C_n, a_n
    C, a, J, cnt = km.kmeans_fit_pruned(Pg, k, T, idx, counters=True)
    C_f, a_f, J_f, cnt_f = orc.fit_pruned(Po, k, T, idx)
    torch.cuda.synchronize()
    assert abs(host(J)[0] - J_f[0]) <= 1e-5 * J_f[0]
    assert abs(host(J)[-1] - J_f[-1]) <= 1e-3 * J_f[-1]
    # survivor counts of the two runs agree up to the rounding-level divergence above
    assert np.all(np.abs(cnt.astype(np.float64) - cnt_f) <= 0.01 * cnt_f + 10)
