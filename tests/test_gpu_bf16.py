"""GPU parity of the bfloat16 point format against the CPU oracle: encoding
(bit-exact), assignment (fp tolerance on the bfloat16 values, exact ties to the
smallest index), update (centroid tolerance), and Lloyd in lock-step.
Tolerances are the ones stated in gpu_util.py.
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import OBJ_REL, assert_centroids, assert_fp_assign, f32_dist, host, say, to_dev, torch_cuda

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


def blobs(n, d, comps, seed, sigma=0.3, normalize=False):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((comps, d))
    lab = rng.integers(0, comps, n)
    X = mu[lab] + sigma * rng.standard_normal((n, d))
    if normalize:
        X /= np.linalg.norm(X, axis=1, keepdims=True)
    return X.astype(np.float32)


def pick(n, k, seed):
    rng = np.random.default_rng(seed + 99)
    return rng.choice(n, k, replace=False) if n >= k else rng.integers(0, n, k)


def bf16_dev(codes, torch):
    """uint16 patterns -> torch.bfloat16 device tensor holding the same bits."""
    return to_dev(codes.view(np.int16), torch).view(torch.bfloat16)


def bf16_host(t):
    return t.view(__import__("torch").int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("n,d", [(1, 8), (257, 8), (1000, 128), (3001, 776)])
def test_quantize_bf16_bit_exact(km, torch, n, d):
    say(f"quantize bf16 n={n} d={d}")
    X = blobs(n, d, 5, seed=n + d)
    rng = np.random.default_rng(n)
    # exact ties, subnormals, overflow, infinities and NaN among ordinary values
    u = X.view(np.uint32).copy()
    u[:, 0] = (u[:, 0] & 0xFFFF0000) | 0x8000
    X = u.view(np.float32)
    special = np.array([2.0 ** -134, 3 * 2.0 ** -134, 2.0 ** -149, -0.0, np.float32(3.4e38), np.inf, -np.inf,
                        np.nan], np.float32)
    X.reshape(-1)[rng.choice(X.size, min(X.size, len(special)), replace=False)] = special[: min(X.size, 8)]
    out = km.quantize_bf16(to_dev(X, torch))
    torch.cuda.synchronize()
    got = bf16_host(out)
    exp = orc.bf16_round(X)
    nan = np.isnan(X)
    np.testing.assert_array_equal(got[~nan], exp[~nan])
    assert ((got[nan] & 0x7F80) == 0x7F80).all() and ((got[nan] & 0x7F) != 0).all()


ASSIGN_SHAPES = [(1, 8, 1), (5, 16, 3), (300, 32, 3), (1000, 128, 64), (2049, 96, 130), (517, 768, 257),
                 (700, 136, 129), (130, 64, 300), (600, 1000, 70), (64, 8, 5), (600, 64, 900)]


@pytest.mark.parametrize("n,d,k", ASSIGN_SHAPES)
def test_assign_bf16(km, torch, n, d, k):
    say(f"assign bf16 n={n} d={d} k={k}")
    X = blobs(n, d, max(2, k // 2), seed=n + d + k)
    codes = orc.bf16_round(X)
    C = X[pick(n, k, n)].copy()
    C += np.random.default_rng(1).standard_normal(C.shape).astype(np.float32) * 0.01
    if k >= 4:
        C[3] = C[1]  # identical centroids: the smaller index must win every time
    a_o, dist_o = orc.assign_bf16(codes, C)
    P = km.points_bf16(bf16_dev(codes, torch))
    a, sc, obj = km.kmeans_assign(P, to_dev(C, torch), score=True, objective=True)
    torch.cuda.synchronize()
    a = host(a)
    assert a.min() >= 0 and a.max() < k
    if k >= 4:
        assert not (a == 3).any()
    Xb = orc.bf16_decode(codes).astype(np.float64)
    Cb = orc.bf16_decode(orc.bf16_round(C)).astype(np.float64)
    assert_fp_assign(a, a_o, f32_dist(Xb, Cb), "bf16")
    exp_sc = (Cb[a] ** 2).sum(1) - 2 * (Xb * Cb[a]).sum(1)
    np.testing.assert_allclose(host(sc), exp_sc, rtol=1e-4, atol=1e-4 * (1 + np.abs(Xb).max() ** 2 * d))
    J = host(obj)[0]
    assert abs(J - dist_o.sum()) <= OBJ_REL * dist_o.sum() + 1e-3


def test_assign_bf16_strided_rows(km, torch):
    n, d, k = 777, 64, 70
    W = blobs(n, 96, 20, seed=4)
    codes_w = orc.bf16_round(W)
    codes = np.ascontiguousarray(codes_w[:, :d])
    C = orc.bf16_decode(codes[pick(n, k, 3)]).copy()
    Xt = bf16_dev(codes_w, torch)[:, :d]
    P = km.points_bf16(Xt)
    assert P._c.ld == 96
    a, _, _ = km.kmeans_assign(P, to_dev(C, torch), score=False)
    a_o, _ = orc.assign_bf16(codes, C)
    assert_fp_assign(host(a), a_o, f32_dist(orc.bf16_decode(codes), C), "bf16 strided")


def rand_assign(n, k, seed, empties=(), invalid=0):
    rng = np.random.default_rng(seed)
    live = np.setdiff1d(np.arange(k), np.asarray(empties, dtype=np.int64))
    a = rng.choice(live, n).astype(np.int32)
    if invalid:
        idx = rng.choice(n, invalid, replace=False)
        a[idx[: invalid // 2]] = -1
        a[idx[invalid // 2:]] = k + 3
    return a


@pytest.mark.parametrize("n,d,k,empties", [(1, 32, 1, ()), (300, 32, 5, (1, 3)), (5000, 128, 64, (0, 7, 63)),
                                           (3001, 776, 130, (5,)), (2000, 96, 300, ()), (40, 64, 50, ()),
                                           (1200, 8, 9, (8,))])
@pytest.mark.parametrize("policy", [0, 1])
def test_update_bf16(km, torch, n, d, k, empties, policy):
    say(f"update bf16 n={n} d={d} k={k} policy={policy}")
    codes = orc.bf16_round(blobs(n, d, 8, seed=n + k))
    a = rand_assign(n, k, seed=n + d, empties=empties, invalid=min(10, n // 10))
    C0 = np.random.default_rng(2).standard_normal((k, d)).astype(np.float32)
    C_o, cnt_o = orc.update_bf16(codes, a, k, C0, policy)
    C = to_dev(C0, torch)
    _, cnt = km.kmeans_update(km.points_bf16(bf16_dev(codes, torch)), to_dev(a, torch), C, policy)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_o)
    assert_centroids(host(C), C_o, "bf16 update")


def test_fit_bf16_init_gather_is_exact(km, torch):
    """STEP 1 with no Lloyd iteration: the centroids are the sampled stored values."""
    X = blobs(3000, 136, 20, seed=8)
    codes = orc.bf16_round(X)
    idx = np.random.default_rng(9).choice(3000, 40, replace=False)
    C, a, J = km.kmeans_fit(km.points_bf16(bf16_dev(codes, torch)), 40, 0, idx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(C), orc.bf16_decode(codes[idx]))


def test_fit_bf16_lockstep_and_free_running(km, torch):
    """Unit-normalised mixture shaped like the 768-dim embedding workload (fewer rows):
    every step compared with the oracle fed the same centroids, then a free-running fit."""
    import synth
    spec = synth.config(2)["spec"].with_n(20000)
    X = synth.make_points(spec)
    codes = orc.bf16_round(X)
    k, T = 64, 5
    idx = synth.init_indices(len(X), k)
    Po = {"fmt": "bf16", "codes": codes}
    P = km.points_bf16(bf16_dev(codes, torch))
    Xb = orc.bf16_decode(codes)
    C_o = orc.init_centroids(Po, idx)
    for t in range(T + 1):
        say(f"lockstep bf16 iteration {t}")
        a_o, dist_o = orc.assign_bf16(codes, C_o)
        a, _, obj = km.kmeans_assign(P, to_dev(C_o, torch), score=False, objective=True)
        torch.cuda.synchronize()
        Cb = orc.bf16_decode(orc.bf16_round(C_o))
        assert_fp_assign(host(a), a_o, f32_dist(Xb, Cb), f"iter {t}")
        assert abs(host(obj)[0] - dist_o.sum()) <= OBJ_REL * dist_o.sum()
        if t == T:
            break
        C_n, cnt_o = orc.update_bf16(codes, a_o, k, C_o)
        C = to_dev(C_o, torch)
        _, cnt = km.kmeans_update(P, to_dev(a_o, torch), C)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(cnt), cnt_o)
        assert_centroids(host(C), C_n, f"iter {t}")
        C_o = C_n
    C_f, a_f, J_f = orc.fit(Po, k, T, idx)
    C, a, J = km.kmeans_fit(P, k, T, idx)
    torch.cuda.synchronize()
    assert_fp_assign(host(a), a_f, f32_dist(Xb, orc.bf16_decode(orc.bf16_round(C_f))), "free-running")
    np.testing.assert_allclose(host(J), J_f, rtol=OBJ_REL)
