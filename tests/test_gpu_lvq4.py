"""GPU parity of LVQ4 (Sec. 3.1 LVQ with B = 4, Eq. 1-2) against the CPU oracle:
encoding (codes and per-vector parameters bit-exact), assignment (assignments and
scores bit-exact: both sides form the same fp32 expression from exact integer dot
products of the codes), update (decoded means within the centroid tolerance),
Lloyd in lock-step and the raw-row last update.  Tolerances are the ones stated in
gpu_util.py.
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import OBJ_REL, assert_centroids, host, say, to_dev, torch_cuda

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


def blobs(n, d, comps, seed, sigma=0.3, normalize=True):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((comps, d))
    X = mu[rng.integers(0, comps, n)] + sigma * rng.standard_normal((n, d))
    if normalize:
        X /= np.linalg.norm(X, axis=1, keepdims=True)
    return X.astype(np.float32)


def pick(n, k, seed):
    rng = np.random.default_rng(seed + 99)
    return rng.choice(n, k, replace=False) if n >= k else rng.integers(0, n, k)


def encode(X):
    codes, par = orc.lvq4_encode(X)
    return codes, orc.lvq4_pack(codes), par


# rows of up to 1024 and 2048 dims stay in registers between the two passes (the
# limits: 1024, 2048); 2080 reads the row twice
@pytest.mark.parametrize("n,d", [(1, 32), (3, 64), (1000, 128), (3001, 768), (200, 1024), (257, 1536), (100, 2048),
                                 (60, 2080)])
def test_quantize_lvq4_bit_exact(km, torch, n, d):
    say(f"quantize lvq4 n={n} d={d}")
    X = blobs(n, d, 5, seed=n + d, normalize=False)
    if n >= 3:
        X[1] = 0.25      # constant row: range 0, scale 1, every code 0
        X[2, ::2] = -1.0  # two-valued row: codes 0 and 15 only
        X[2, 1::2] = 2.0
    codes_o, packed_o, par_o = encode(X)
    codes, par = km.quantize_lvq4(to_dev(X, torch))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(codes), packed_o)
    np.testing.assert_array_equal(host(par), par_o)


# every shape runs the 256 x 256 int8 kernel: ragged n and k tails, k below and above a tile,
# d from one 32-dim step to several 1024-byte stages
ASSIGN_SHAPES = [(1, 32, 1), (5, 64, 3), (300, 96, 3), (1000, 128, 64), (2049, 256, 130), (517, 768, 257),
                 (130, 64, 300), (700, 64, 600), (300, 1536, 70), (700, 2048, 300)]


@pytest.mark.parametrize("n,d,k", ASSIGN_SHAPES)
def test_assign_lvq4_bit_exact(km, torch, n, d, k):
    say(f"assign lvq4 n={n} d={d} k={k}")
    X = blobs(n, d, max(2, k), seed=n + d + k)
    _, packed, par = encode(X)
    rng = np.random.default_rng(n + k)
    C = (X[pick(n, k, n)] + rng.standard_normal((k, d)).astype(np.float32) * 0.02).astype(np.float32)
    if k >= 4:
        C[3] = C[1]  # identical codes: the smaller index wins
    if k >= 3:
        C[2] = 0.1   # constant centroid (range 0)
    codes_o, _, _ = encode(X)
    a_o, sc_o, dist_o = orc.assign_lvq4(codes_o, par, C)
    P = km.points_lvq4(to_dev(packed, torch), to_dev(par, torch), d)
    a, sc, obj = km.kmeans_assign(P, to_dev(C, torch), score=True, objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(sc), sc_o)
    if k >= 4:
        assert not (host(a) == 3).any()
    assert abs(host(obj)[0] - dist_o.sum()) <= 1e-5 * abs(dist_o.sum()) + 1e-6


def test_assign_lvq4_strided_rows(km, torch):
    n, d, k = 777, 128, 70
    X = blobs(n, d, 20, seed=4)
    codes_o, packed, par = encode(X)
    wide = np.zeros((n, 96), np.uint8)  # row stride 96 bytes > d/2 = 64
    wide[:, :64] = packed
    wide[:, 64:] = 0xAB                 # bytes past d/2 must not be read as codes
    C = X[pick(n, k, 3)].copy()
    P = km.points_lvq4(to_dev(wide, torch)[:, :64], to_dev(par, torch), d)
    assert P._c.ld == 96
    a, sc, _ = km.kmeans_assign(P, to_dev(C, torch), score=True)
    torch.cuda.synchronize()
    a_o, sc_o, _ = orc.assign_lvq4(codes_o, par, C)
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(sc), sc_o)


def rand_assign(n, k, seed, empties=(), invalid=0):
    rng = np.random.default_rng(seed)
    live = np.setdiff1d(np.arange(k), np.asarray(empties, dtype=np.int64))
    a = rng.choice(live, n).astype(np.int32)
    if invalid:
        idx = rng.choice(n, invalid, replace=False)
        a[idx[: invalid // 2]] = -1
        a[idx[invalid // 2:]] = k + 3
    return a


@pytest.mark.parametrize("n,d,k,empties", [(1, 32, 1, ()), (300, 64, 5, (1, 3)), (5000, 128, 64, (0, 7, 63)),
                                           (3001, 768, 130, (5,)), (2000, 96, 300, ()), (40, 64, 50, ()),
                                           (700, 2048, 40, (2,))])
@pytest.mark.parametrize("policy", [0, 1])
def test_update_lvq4(km, torch, n, d, k, empties, policy):
    say(f"update lvq4 n={n} d={d} k={k} policy={policy}")
    codes, packed, par = encode(blobs(n, d, 8, seed=n + k, normalize=False))
    a = rand_assign(n, k, seed=n + d, empties=empties, invalid=min(10, n // 10))
    C0 = np.random.default_rng(2).standard_normal((k, d)).astype(np.float32)
    C_o, cnt_o = orc.update_lvq4(codes, par, a, k, C0, policy)
    C = to_dev(C0, torch)
    P = km.points_lvq4(to_dev(packed, torch), to_dev(par, torch), d)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), C, policy)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_o)
    assert_centroids(host(C), C_o, "lvq4 update")


def test_fit_lvq4_init_gather_is_exact(km, torch):
    """STEP 1 with no Lloyd iteration: the centroids are the decoded sampled points."""
    X = blobs(3000, 256, 20, seed=8)
    codes, packed, par = encode(X)
    idx = np.random.default_rng(9).choice(3000, 40, replace=False)
    C, _, _ = km.kmeans_fit(km.points_lvq4(to_dev(packed, torch), to_dev(par, torch), 256), 40, 0, idx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(C), orc.lvq4_decode(codes[idx], par[idx]))


def test_fit_lvq4_lockstep_and_raw_last_update(km, torch):
    """Unit-normalised mixture shaped like the 768-dim embedding workload (fewer rows):
    every assignment pass bit-exact and every update within tolerance when both sides
    start from the same centroids; then kmeans_fit with raw rows and one update, whose
    centroids are the raw-row means of the first pass."""
    import synth
    spec = synth.config(2)["spec"].with_n(20000)
    X = synth.make_points(spec)
    d = spec.d
    codes, packed, par = encode(X)
    k, T = 64, 4
    idx = synth.init_indices(len(X), k)
    Po = {"fmt": "lvq4", "codes": codes, "par": par}
    Pg = km.points_lvq4(to_dev(packed, torch), to_dev(par, torch), d)
    C_o = orc.init_centroids(Po, idx)
    for t in range(T + 1):
        say(f"lockstep lvq4 iteration {t}")
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
    Pr = km.points_lvq4(to_dev(packed, torch), to_dev(par, torch), d, raw=to_dev(X, torch))
    C1, a1, J1 = km.kmeans_fit(Pr, k, 1, idx)
    torch.cuda.synchronize()
    C1_o, a1_o, J1_o = orc.fit(dict(Po, raw=X), k, 1, idx)
    assert_centroids(host(C1), C1_o, "raw last update")
    np.testing.assert_allclose(host(J1)[0], J1_o[0], rtol=1e-6)
