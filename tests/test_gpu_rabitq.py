"""GPU parity of RabitQ as the paper runs it (Sec. 3.1, Eq. 3-5): codes of the
randomly rotated, centred residual, per-centroid SQ4 centroid codes with bias,
and the raw-vector last update (Sec. 4.1).  Assignments and scores are bit-exact
(the same fp32 expression on exact integer sums); centroids and objectives use
the tolerances stated in gpu_util.py.
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import OBJ_REL, assert_centroids, host, say, to_dev, torch_cuda, unpack_bits

pytestmark = pytest.mark.gpu


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


def blobs(n, d, comps, seed, sigma=0.4):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((comps, d))
    X = mu[rng.integers(0, comps, n)] + sigma * rng.standard_normal((n, d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    return X.astype(np.float32)


def rotated(X, seed):
    """Oracle side of the encoding: m, P, y = (x - m) P, bits and alpha of y."""
    import synth
    d = X.shape[1]
    m = orc.col_mean(X)
    P = synth.random_rotation(d, seed)
    Y = orc.project(X, m, P)
    bits, alpha = orc.sign1_encode(Y, np.zeros(d, np.float32), 0)
    return m, P, Y, bits, alpha


@pytest.mark.parametrize("n,d", [(1, 32), (1000, 128), (3001, 1024), (500, 1536)])
def test_rabitq_encode(km, torch, n, d):
    say(f"rabitq encode n={n} d={d}")
    X = blobs(n, d, 5, seed=n + d)
    m, P, Y, bits_o, alpha_o = rotated(X, seed=d)
    bits, mg, alpha, Yg = km.rabitq_encode(to_dev(X, torch), to_dev(P, torch), center=to_dev(m, torch),
                                           want_rotated=True)
    torch.cuda.synchronize()
    # fp32 dot products of length d: error bounded relative to the row norm ||x - m||
    rn = np.linalg.norm(X.astype(np.float64) - m.astype(np.float64), axis=1, keepdims=True)
    assert (np.abs(host(Yg).astype(np.float64) - Y) <= 2e-6 * rn + 1e-12).all()
    # the GPU rotation (fp32 MFMA) and the oracle's (fp64 sums) differ by rounding:
    # signs may differ only where a rotated coordinate is within rounding of 0
    diff = unpack_bits(host(bits).view(np.uint32), d) != unpack_bits(bits_o, d)
    scale = np.abs(Y).max(1, keepdims=True) + 1e-30
    assert (np.abs(Y)[diff] <= 1e-5 * np.broadcast_to(scale, Y.shape)[diff]).all()
    np.testing.assert_allclose(host(alpha), alpha_o, rtol=2e-5, atol=1e-7)
    # fitted centre: the column mean
    _, m2, _, _ = km.rabitq_encode(to_dev(X, torch), to_dev(P, torch))
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(m2), m, rtol=2e-7, atol=1e-9)


def pick(n, k, seed):
    rng = np.random.default_rng(seed + 99)
    return rng.choice(n, k, replace=False) if n >= k else rng.integers(0, n, k)


# d <= 1280 runs the resident-bits kernel, d > 1280 the 256 x 256 int8 kernel
@pytest.mark.parametrize("n,d,k", [(1, 32, 1), (5, 64, 3), (300, 96, 3), (1000, 128, 64), (2049, 256, 130),
                                   (517, 1024, 257), (130, 64, 300), (700, 64, 600), (300, 1536, 70),
                                   (700, 2048, 300), (600, 1152, 140), (300, 1280, 70)])
def test_assign_rabitq_bit_exact(km, torch, n, d, k):
    say(f"assign rabitq n={n} d={d} k={k}")
    X = blobs(n, d, max(2, k), seed=n + d + k)
    m, P, Y, bits, alpha = rotated(X, seed=k)
    rng = np.random.default_rng(n + k)
    C = (Y[pick(n, k, n)] + rng.standard_normal((k, d)).astype(np.float32) * 0.02).astype(np.float32)
    if k >= 4:
        C[3] = C[1]  # exact ties resolve to the smaller index
    if k >= 3:
        C[2] = 0.1   # a constant centroid (SQ4 range 0)
    a_o, sc_o, dist_o = orc.assign_rabitq(bits, alpha, C)
    Pg = km.points_rabitq(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), d)
    a, sc, obj = km.kmeans_assign(Pg, to_dev(C, torch), score=True, objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(sc), sc_o)
    assert abs(host(obj)[0] - dist_o.sum()) <= 1e-5 * abs(dist_o.sum()) + 1e-6


@pytest.mark.parametrize("n,d,k,empties", [(1, 32, 1, ()), (300, 64, 5, (1, 3)), (5000, 128, 64, (0, 7, 63)),
                                           (3001, 1024, 130, (5,)), (700, 1536, 40, (2,))])
@pytest.mark.parametrize("policy", [0, 1])
def test_update_rabitq(km, torch, n, d, k, empties, policy):
    say(f"update rabitq n={n} d={d} k={k} policy={policy}")
    X = blobs(n, d, 8, seed=n + d)
    _, _, _, bits, alpha = rotated(X, seed=3)
    rng = np.random.default_rng(n)
    live = np.setdiff1d(np.arange(k), np.asarray(empties, dtype=np.int64))
    a = rng.choice(live, n).astype(np.int32)
    C0 = (rng.standard_normal((k, d)) * 0.05).astype(np.float32)
    Po = {"fmt": "rabitq", "bits": bits, "alpha": alpha, "d": d}
    C_o, cnt_o = orc.update(Po, a, k, C0, policy)
    C = to_dev(C0, torch)
    Pg = km.points_rabitq(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), d)
    _, cnt = km.kmeans_update(Pg, to_dev(a, torch), C, policy)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_o)
    assert_centroids(host(C), C_o, "rabitq update")


def test_fit_rabitq_lockstep_and_raw_last_update(km, torch):
    """Unit-normalised mixture shaped like the 1-bit workload (fewer rows): every
    assignment pass bit-exact and every update within tolerance when both sides start
    from the same centroids; then kmeans_fit with raw rows, one update: its centroids
    are the raw-row means of the first pass, as in the oracle."""
    import synth
    spec = synth.config(3)["spec"].with_n(20000)
    X = synth.make_points(spec)
    d = spec.d
    m, P, Y, bits, alpha = rotated(X, seed=11)
    k, T = 64, 4
    idx = synth.init_indices(len(X), k)
    Po = {"fmt": "rabitq", "bits": bits, "alpha": alpha, "d": d}
    Pg = km.points_rabitq(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), d)
    C_o = orc.init_centroids(Po, idx)
    for t in range(T + 1):
        say(f"lockstep rabitq iteration {t}")
        a_o, dist_o = orc.assign(Po, C_o)
        a, _, obj = km.kmeans_assign(Pg, to_dev(C_o, torch), score=False, objective=True)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(a), a_o)
        assert abs(host(obj)[0] - dist_o.sum()) <= OBJ_REL * abs(dist_o.sum())
        if t == T:
            break
        C_n, cnt_o = orc.update(Po, a_o, k, C_o)
        C = to_dev(C_o, torch)
        _, cnt = km.kmeans_update(Pg, to_dev(a_o, torch), C)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(cnt), cnt_o)
        assert_centroids(host(C), C_n, f"iter {t}")
        C_o = C_n
    # kmeans_fit, one update from the raw rotated rows
    Pr = km.points_rabitq(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), d, raw=to_dev(Y, torch))
    C1, a1, J1 = km.kmeans_fit(Pr, k, 1, idx)
    torch.cuda.synchronize()
    Po_raw = dict(Po, raw=Y)
    C1_o, a1_o, J1_o = orc.fit(Po_raw, k, 1, idx)
    assert_centroids(host(C1), C1_o, "raw last update")
    np.testing.assert_allclose(host(J1)[0], J1_o[0], rtol=1e-6)
