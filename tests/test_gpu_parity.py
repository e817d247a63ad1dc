"""GPU parity: every step of the HIP path against the CPU oracle on the same
seeded inputs, at sizes the oracle finishes in seconds that still span several
tiles and ragged tails.  Tolerances are stated in gpu_util.py.
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import (CENT_REL, OBJ_REL, assert_centroids, assert_fp_assign, f32_dist, host, say, to_dev,
                      torch_cuda, unpack_bits)

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
    return rng.choice(n, k, replace=n < k) if n >= k else rng.integers(0, n, k)


ASSIGN_SHAPES = [(1, 32, 1), (5, 32, 3), (300, 32, 3), (1000, 128, 64), (2049, 96, 130), (517, 768, 257),
                 (700, 160, 129), (130, 64, 300)]


# --------------------------------------------------------------------------- assign

# (600, 32, 2500) and (500, 4, 2100): one stage per centroid tile, three tiles per workgroup
@pytest.mark.parametrize("n,d,k", ASSIGN_SHAPES + [(700, 36, 129), (64, 4, 5), (3000, 64, 1024), (1500, 32, 1100),
                                                   (200, 96, 2000), (600, 32, 2500), (500, 4, 2100)])
def test_assign_f32(km, torch, n, d, k):
    say(f"assign f32 n={n} d={d} k={k}")
    X = blobs(n, d, max(2, k // 2), seed=n + d + k)
    C = X[pick(n, k, n)].copy()
    C += np.random.default_rng(1).standard_normal(C.shape).astype(np.float32) * 0.01
    a_o, dist_o = orc.assign_f32(X, C)
    P = km.points_f32(to_dev(X, torch))
    a, sc, obj = km.kmeans_assign(P, to_dev(C, torch), score=True, objective=True)
    torch.cuda.synchronize()
    a = host(a)
    assert a.min() >= 0 and a.max() < k
    assert_fp_assign(a, a_o, f32_dist(X, C), "f32")
    # score = ||c||^2 - 2<x,c> of the chosen centroid
    Xd, Cd = X.astype(np.float64), C.astype(np.float64)
    exp_sc = (Cd[a] ** 2).sum(1) - 2 * (Xd * Cd[a]).sum(1)
    np.testing.assert_allclose(host(sc), exp_sc, rtol=1e-4, atol=1e-4 * (1 + np.abs(Xd).max() ** 2 * d))
    J = host(obj)[0]
    assert abs(J - dist_o.sum()) <= OBJ_REL * dist_o.sum() + 1e-3


@pytest.mark.parametrize("fmt", ["f32", "hybrid", "sq8", "bf16"])
def test_assign_ties_across_centroid_groups(km, torch, fmt):
    """k = 1100 spreads the five 256-centroid tiles over five workgroups per point
    tile at this n, merged through (score, index) keys; copies of centroids 5 and
    130 placed in other groups' tiles must never win."""
    n, d, k = 3000, 96, 1100
    X = blobs(n, d, 40, seed=17)
    C = X[pick(n, k, 17)].copy()
    C[900] = C[5]    # tile 3 vs tile 0
    C[1050] = C[130]  # tile 4 vs tile 0
    C[640] = C[5]
    if fmt == "sq8":  # exact integer scores: bit-exact against the oracle
        lo, hi = orc.sq8_fit(X)
        codes, Cq = orc.sq8_encode(X, lo, hi), orc.sq8_encode(C, lo, hi)
        a_o, dist_o = orc.assign_sq8(codes, Cq)
        a, sc, _ = km.kmeans_assign(km.points_sq8(to_dev(codes, torch)), to_dev(Cq, torch), score=True)
        torch.cuda.synchronize()
        a = host(a)
        np.testing.assert_array_equal(a, a_o)
        sq = (Cq.astype(np.int64) - 128)
        exp_sc = (sq[a] ** 2).sum(1) - 2 * (sq[a] * (codes.astype(np.int64) - 128)).sum(1)
        np.testing.assert_array_equal(host(sc).astype(np.int64), exp_sc)
    elif fmt == "bf16":
        codes = orc.bf16_round(X)
        a_o, _ = orc.assign_bf16(codes, C)
        Pb = km.points_bf16(to_dev(codes.view(np.int16), torch).view(torch.bfloat16))
        a, _, _ = km.kmeans_assign(Pb, to_dev(C, torch), score=False)
        a = host(a)
        Xb = orc.bf16_decode(codes).astype(np.float64)
        Cb = orc.bf16_decode(orc.bf16_round(C)).astype(np.float64)
        assert_fp_assign(a, a_o, f32_dist(Xb, Cb), "bf16 groups")
    if fmt == "f32":
        a_o, _ = orc.assign_f32(X, C)
        a, _, _ = km.kmeans_assign(km.points_f32(to_dev(X, torch)), to_dev(C, torch), score=False)
        a = host(a)
        assert_fp_assign(a, a_o, f32_dist(X, C), "f32 groups")
    elif fmt == "hybrid":
        d0 = 32
        m = orc.col_mean(X)
        bits, alpha = orc.sign1_encode(X, m, d0)
        front = np.ascontiguousarray(X[:, :d0])
        a_o, _ = orc.assign_hybrid(front, bits, alpha, C, m, d0)
        P = km.points_hybrid(to_dev(front, torch), to_dev(bits.view(np.int32), torch), to_dev(alpha, torch),
                             to_dev(m, torch), d)
        a, _, _ = km.kmeans_assign(P, to_dev(C, torch), score=False)
        a = host(a)
    if fmt in ("f32", "sq8", "bf16"):  # each centroid is a data point, which picks it (or an equal copy)
        assert (a == 5).any() and (a == 130).any()
    assert not np.isin(a, [640, 900, 1050]).any()


def test_assign_f32_strided_rows(km, torch):
    n, d, k = 777, 64, 70
    W = blobs(n, 96, 20, seed=4)
    X = W[:, :d]
    C = np.ascontiguousarray(X[pick(n, k, 3)])
    Xt = to_dev(W, torch)[:, :d]
    P = km.points_f32(Xt)
    assert P._c.ld == 96
    a, _, _ = km.kmeans_assign(P, to_dev(C, torch), score=False)
    a_o, _ = orc.assign_f32(np.ascontiguousarray(X), C)
    assert_fp_assign(host(a), a_o, f32_dist(X, C), "f32 strided")


# (700, 16, 900): 4 centroid-tile groups merged through exact integer keys; (500, 32, 2100):
# 9 tiles over 5 groups (uneven); (300, 8208, 20): rows beyond 8192 dims take the
# register-staged int8 kernel
@pytest.mark.parametrize("n,d,k", [(1, 16, 1), (5, 16, 3), (300, 32, 3), (1000, 128, 64), (2049, 96, 130),
                                   (517, 768, 257), (130, 48, 300), (700, 16, 900), (500, 32, 2100),
                                   (300, 8208, 20)])
def test_assign_sq8_bit_exact(km, torch, n, d, k):
    say(f"assign sq8 n={n} d={d} k={k}")
    rng = np.random.default_rng(n * 7 + d + k)
    X = blobs(n, d, max(2, k // 2), seed=n + k)
    lo, hi = orc.sq8_fit(X)
    codes = orc.sq8_encode(X, lo, hi)
    C = codes[pick(n, k, n)].copy()
    if k >= 3:
        C[k - 1] = C[0]          # exact ties resolve to the smallest index
        C[k // 2] = C[1]
    C[0, : min(d, 8)] = rng.integers(0, 256, min(d, 8))
    a_o, dist_o = orc.assign_sq8(codes, C)
    a, sc, obj = km.kmeans_assign(km.points_sq8(to_dev(codes, torch)), to_dev(C, torch), score=True, objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(a), a_o)
    xt = codes.astype(np.int64) - 128
    exp = dist_o - (xt * xt).sum(1)
    np.testing.assert_array_equal(host(sc), exp.astype(np.float32))
    if dist_o.max() < 2 ** 24:  # every per-point term is exact in the fp32 score
        assert host(obj)[0] == float(dist_o.sum())
    else:  # long rows: terms above 2^24 carry fp32 rounding (2^-24 relative each)
        assert abs(host(obj)[0] - dist_o.sum()) <= 2 ** -23 * dist_o.sum()


# Codes at the ends of the range reach the extremes of the SQ8 key 2<x~,c~> - ||c~||^2
# (-48896 d with x~ = 127, c~ = -128; 16384 d with x~ = c~ = -128).  d <= 1024 selects
# with packed 32-bit keys whose range holds exactly at 1024 dimensions (1008: a partial
# last stage); 1040 and 1104 take the unpacked selection; 128-centroid tiles for
# k = 100, 256-centroid tiles merged across groups for k = 700.
@pytest.mark.parametrize("n,d,k", [(600, 1024, 100), (1500, 1024, 700), (777, 1008, 300), (400, 1040, 260),
                                   (300, 1104, 90)])
def test_assign_sq8_extreme_codes(km, torch, n, d, k):
    say(f"assign sq8 extreme codes n={n} d={d} k={k}")
    rng = np.random.default_rng(n + d + k)
    codes = rng.choice(np.array([0, 255], np.uint8), size=(n, d))
    codes[0::7] = 255
    codes[1::7] = 0
    codes[2::7, : d // 2] = 0
    C = rng.choice(np.array([0, 255], np.uint8), size=(k, d))
    C[0::5] = 0
    C[1::5] = 255
    C[2::5] = codes[3]           # exact matches and ties
    C[3::5, d // 3:] = 0
    C[k - 1] = C[2]
    a_o, dist_o = orc.assign_sq8(codes, C)
    a, sc, _ = km.kmeans_assign(km.points_sq8(to_dev(codes, torch)), to_dev(C, torch), score=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(a), a_o)
    xt = codes.astype(np.int64) - 128
    exp = dist_o - (xt * xt).sum(1)
    np.testing.assert_array_equal(host(sc), exp.astype(np.float32))


def sign1_inputs(n, d, k, seed, d0=0):
    X = blobs(n, d, max(2, k), seed=seed, sigma=0.4, normalize=True)
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m, d0)
    rng = np.random.default_rng(seed + 5)
    C = (X[pick(n, k, seed)] + rng.standard_normal((k, d)).astype(np.float32) * 0.02).astype(np.float32)
    return X, m, bits, alpha, C


# d > 1280 takes the 256 x 256 int8 kernel instead of the resident-bits one
@pytest.mark.parametrize("n,d,k", [(1, 32, 1), (5, 64, 3), (300, 96, 3), (1000, 128, 64), (2049, 256, 130),
                                   (517, 1024, 257), (700, 160, 129), (130, 64, 300), (700, 64, 600),
                                   (300, 1536, 70), (700, 2048, 300), (1, 1312, 3), (600, 1152, 140),
                                   (300, 1280, 70)])
def test_assign_sign1_bit_exact(km, torch, n, d, k):
    say(f"assign sign1 n={n} d={d} k={k}")
    X, m, bits, alpha, C = sign1_inputs(n, d, k, seed=n + d + k)
    if k >= 4:
        C[3] = C[1]
    a_o, sc_o, dist_o = orc.assign_sign1(bits, alpha, C, m)
    P = km.points_sign1(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), to_dev(m, torch), d)
    a, sc, obj = km.kmeans_assign(P, to_dev(C, torch), score=True, objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(sc), sc_o)
    assert abs(host(obj)[0] - dist_o.sum()) <= 1e-5 * dist_o.sum() + 1e-6


# (700, 256, 128, 300): one tail stage; (300, 1280, 512, 1100): a 768-dim tail and
# centroid-tile groups
@pytest.mark.parametrize("n,d,d0,k", [(300, 64, 32, 3), (1000, 128, 32, 64), (2049, 256, 96, 130),
                                      (517, 1024, 384, 257), (700, 256, 128, 300), (1000, 384, 128, 64),
                                      (300, 1280, 512, 1100), (50, 96, 64, 7), (600, 128, 32, 1100)])
def test_assign_hybrid(km, torch, n, d, d0, k):
    say(f"assign hybrid n={n} d={d} d0={d0} k={k}")
    X, m, bits, alpha, C = sign1_inputs(n, d, k, seed=n + d + k + d0, d0=d0)
    front = np.ascontiguousarray(X[:, :d0])
    a_o, dist_o = orc.assign_hybrid(front, bits, alpha, C, m, d0)
    P = km.points_hybrid(to_dev(front, torch), to_dev(bits.view(np.int32), torch), to_dev(alpha, torch),
                         to_dev(m, torch), d)
    a, sc, obj = km.kmeans_assign(P, to_dev(C, torch), score=True, objective=True)
    torch.cuda.synchronize()
    q, sigma, T, Q, u = orc.sign1_prep(C, m, d0)
    sgn = np.where(unpack_bits(bits, d)[:, d0:] > 0, 1.0, -1.0)

    def d_of(rows, cands):
        fr = ((front[rows].astype(np.float64) - C[cands, :d0]) ** 2).sum(1)
        xt = alpha[rows, None].astype(np.float64) * sgn[rows]
        ct = sigma[cands, None].astype(np.float64) * q[cands]
        tl = ((xt - ct) ** 2).sum(1)
        mag = (front[rows].astype(np.float64) ** 2).sum(1) + (C[cands, :d0].astype(np.float64) ** 2).sum(1) + \
            (xt ** 2).sum(1) + (ct ** 2).sum(1)
        return fr + tl, mag
    assert_fp_assign(host(a), a_o, d_of, "hybrid")
    assert abs(host(obj)[0] - dist_o.sum()) <= OBJ_REL * dist_o.sum()


# --------------------------------------------------------------------------- update

def rand_assign(n, k, seed, empties=(), invalid=0):
    rng = np.random.default_rng(seed)
    live = np.setdiff1d(np.arange(k), np.asarray(empties, dtype=np.int64))
    a = rng.choice(live, n).astype(np.int32)
    if invalid:
        idx = rng.choice(n, invalid, replace=False)
        a[idx[: invalid // 2]] = -1
        a[idx[invalid // 2:]] = k + 3
    return a


# (60000, 32, 20000): k above the LDS cursor limit of the scatter (global cursors)
UPDATE_SHAPES = [(1, 32, 1, ()), (300, 32, 5, (1, 3)), (5000, 128, 64, (0, 7, 63)), (3001, 768, 130, (5,)),
                 (2000, 96, 300, ()), (40, 64, 50, ()), (60000, 32, 20000, (0, 19999))]


@pytest.mark.parametrize("n,d,k,empties", UPDATE_SHAPES)
@pytest.mark.parametrize("policy", [0, 1])
def test_update_f32(km, torch, n, d, k, empties, policy):
    say(f"update f32 n={n} d={d} k={k} policy={policy}")
    X = blobs(n, d, 8, seed=n + k)
    a = rand_assign(n, k, seed=n + d, empties=empties, invalid=min(10, n // 10))
    C0 = np.random.default_rng(2).standard_normal((k, d)).astype(np.float32)
    C_o, cnt_o = orc.update_f32(X, a, k, C0, policy)
    C = to_dev(C0, torch)
    _, cnt = km.kmeans_update(km.points_f32(to_dev(X, torch)), to_dev(a, torch), C, policy)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_o)
    assert_centroids(host(C), C_o, "f32 update")


@pytest.mark.parametrize("n,d,k,empties", [(1, 16, 1, ()), (300, 32, 5, (1, 3)), (5000, 128, 64, (0, 7, 63)),
                                           (3001, 768, 130, (5,)), (40, 64, 50, ())])
@pytest.mark.parametrize("policy", [0, 1])
def test_update_sq8_bit_exact(km, torch, n, d, k, empties, policy):
    say(f"update sq8 n={n} d={d} k={k} policy={policy}")
    rng = np.random.default_rng(n + d)
    codes = rng.integers(0, 256, (n, d)).astype(np.uint8)
    codes[: n // 3, ::3] = 255
    codes[: n // 4, 1::5] = 0
    a = rand_assign(n, k, seed=n + 3, empties=empties, invalid=min(6, n // 10))
    C0 = rng.integers(0, 256, (k, d)).astype(np.uint8)
    C_o, cnt_o = orc.update_sq8(codes, a, k, C0, policy)
    C = to_dev(C0, torch)
    _, cnt = km.kmeans_update(km.points_sq8(to_dev(codes, torch)), to_dev(a, torch), C, policy)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_o)
    np.testing.assert_array_equal(host(C), C_o)


@pytest.mark.parametrize("n,d,k,empties", [(1, 32, 1, ()), (300, 64, 5, (1, 3)), (5000, 128, 64, (0, 7, 63)),
                                           (3001, 1024, 130, (5,)), (700, 160, 40, (2,))])
@pytest.mark.parametrize("policy", [0, 1])
def test_update_sign1(km, torch, n, d, k, empties, policy):
    say(f"update sign1 n={n} d={d} k={k} policy={policy}")
    X, m, bits, alpha, _ = sign1_inputs(n, d, 2, seed=n + d)
    a = rand_assign(n, k, seed=n, empties=empties, invalid=min(6, n // 10))
    C0 = (m + np.random.default_rng(3).standard_normal((k, d)) * 0.05).astype(np.float32)
    C_o, cnt_o = orc.update_sign1(bits, alpha, d, m, a, k, C0, policy)
    P = km.points_sign1(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), to_dev(m, torch), d)
    C = to_dev(C0, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), C, policy)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_o)
    assert_centroids(host(C), C_o, "sign1 update")


@pytest.mark.parametrize("n,d,d0,k,empties", [(300, 64, 32, 5, (1,)), (3001, 1024, 384, 130, (5, 9)),
                                              (2000, 256, 96, 64, ())])
def test_update_hybrid(km, torch, n, d, d0, k, empties):
    say(f"update hybrid n={n} d={d} d0={d0} k={k}")
    X, m, bits, alpha, _ = sign1_inputs(n, d, 2, seed=n + d, d0=d0)
    front = np.ascontiguousarray(X[:, :d0])
    a = rand_assign(n, k, seed=n + 1, empties=empties)
    C0 = (m + np.random.default_rng(3).standard_normal((k, d)) * 0.05).astype(np.float32)
    C_o, cnt_o = orc.update_sign1(bits, alpha, d, m, a, k, C0, 0, front=front, d0=d0)
    P = km.points_hybrid(to_dev(front, torch), to_dev(bits.view(np.int32), torch), to_dev(alpha, torch),
                         to_dev(m, torch), d)
    C = to_dev(C0, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), C, 0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_o)
    assert_centroids(host(C), C_o, "hybrid update")


def test_update_is_deterministic(km, torch):
    n, d, k = 20000, 256, 100
    X = blobs(n, d, 10, seed=11)
    a = rand_assign(n, k, seed=5)
    P = km.points_f32(to_dev(X, torch))
    ad = to_dev(a, torch)
    C1 = torch.zeros((k, d), dtype=torch.float32, device="cuda")
    C2 = torch.zeros((k, d), dtype=torch.float32, device="cuda")
    km.kmeans_update(P, ad, C1)
    km.kmeans_update(P, ad, C2)
    assert torch.equal(C1, C2)


# --------------------------------------------------------------------------- quantize

@pytest.mark.parametrize("n,d", [(1, 16), (1000, 128), (3001, 768), (4097, 48)])
def test_quantize_sq8_bit_exact(km, torch, n, d):
    say(f"quantize sq8 n={n} d={d}")
    X = blobs(n, d, 5, seed=n + d)
    X[:, 3] = 0.25  # a constant column maps to code 0
    lo, hi = orc.sq8_fit(X)
    codes_o = orc.sq8_encode(X, lo, hi)
    codes, params = km.quantize_sq8(to_dev(X, torch))
    torch.cuda.synchronize()
    p = host(params)
    np.testing.assert_array_equal(p[:d], lo)
    np.testing.assert_array_equal(p[d:], hi)
    np.testing.assert_array_equal(host(codes), codes_o)
    codes2, _ = km.quantize_sq8(to_dev(X, torch), params=to_dev(np.concatenate([lo, hi]), torch))
    np.testing.assert_array_equal(host(codes2), codes_o)


@pytest.mark.parametrize("n,d,d0", [(1, 32, 0), (1000, 128, 0), (3001, 1024, 0), (777, 96, 32), (2000, 1024, 384)])
def test_quantize_sign1(km, torch, n, d, d0):
    say(f"quantize sign1 n={n} d={d} d0={d0}")
    X = blobs(n, d, 5, seed=n + d, normalize=True)
    m_o = orc.col_mean(X)
    bits_o, alpha_o = orc.sign1_encode(X, m_o, d0)
    # given the same m: bits bit-exact, alpha to fp64-sum rounding
    bits, m, alpha, front = km.quantize_sign1(to_dev(X, torch), center=to_dev(m_o, torch), d_front=d0,
                                              want_front=d0 > 0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(bits).view(np.uint32), bits_o)
    np.testing.assert_allclose(host(alpha), alpha_o, rtol=2e-7, atol=0)
    if d0:
        np.testing.assert_array_equal(host(front), X[:, :d0])
    # fitted mean: fp64 column sums in another order, within one fp32 rounding
    bits2, m2, alpha2, _ = km.quantize_sign1(to_dev(X, torch), d_front=d0)
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(m2), m_o, rtol=2e-7, atol=1e-9)
    diff = unpack_bits(host(bits2).view(np.uint32), d) != unpack_bits(bits_o, d)
    if diff.any():  # only where x sits within rounding of the mean
        r = np.abs(X - m_o)[diff]
        assert (r <= 1e-6).all()


# --------------------------------------------------------------------------- PCA

# (30001, 520): three column blocks (six tiles, a partial one), eight row splits
# with a partial last stage each; the fold of several fp32 runs per split is
# covered at full size (10M x 1024) by test_c4_pca_full_size
@pytest.mark.parametrize("n,d", [(1, 4), (5000, 64), (20001, 256), (3000, 132), (30001, 520)])
def test_pca_cov(km, torch, n, d):
    say(f"pca cov n={n} d={d}")
    lam = np.arange(1, d + 1) ** -0.5
    X = (np.random.default_rng(n).standard_normal((n, d)) * np.sqrt(lam) + 0.3).astype(np.float32)
    mean_o, cov_o = orc.pca_cov(X)
    mean, cov = km.pca_fit_cov(to_dev(X, torch))
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(mean), mean_o, rtol=1e-6, atol=1e-7)
    c = host(cov).astype(np.float64)
    np.testing.assert_array_equal(c, c.T)
    err = np.linalg.norm(c - cov_o) / max(np.linalg.norm(cov_o), 1e-30)
    assert err <= 1e-5, err
    # entry by entry, each against the scale of its own row and column: a wrong
    # small off-diagonal entry cannot hide under the diagonal
    sd = np.sqrt(np.clip(np.diag(cov_o), 0.0, None))
    bad = np.abs(c - cov_o) > 2e-5 * np.outer(sd, sd) + 1e-12
    assert not bad.any(), (int(bad.sum()), np.argwhere(bad)[:5].tolist())


@pytest.mark.parametrize("n,d,dout", [(1, 4, 4), (5000, 64, 16), (3001, 256, 128), (2000, 1024, 256), (700, 96, 36)])
def test_pca_project(km, torch, n, d, dout):
    say(f"pca project n={n} d={d} dout={dout}")
    X = blobs(n, d, 6, seed=n + d)
    mean64, cov = orc.pca_cov(X) if n > 1 else (X[0].astype(np.float64), np.eye(d))
    W, _ = orc.pca_basis(cov, dout)
    mean = mean64.astype(np.float32)
    Y_o = orc.project(X, mean, W)
    Y = km.pca_project(to_dev(X, torch), to_dev(mean, torch), to_dev(W, torch))
    torch.cuda.synchronize()
    Yh = host(Y)
    scale = np.abs(Y_o).max() + 1e-30
    np.testing.assert_allclose(Yh, Y_o, rtol=0, atol=2e-5 * scale)


# (1500, 1024, 300): two output tiles, the second partial; (257, 36, 40): one
# partial stage and a partial output tile; (300, 4100, 8): past the direct-copy
# kernel's 4096 dims, the register-staged kernel.  W is a seeded orthonormal basis
# (an input), so no eigensolve of a large covariance is needed.
@pytest.mark.parametrize("n,d,dout", [(1500, 1024, 300), (257, 36, 40), (300, 4100, 8)])
def test_pca_project_shapes(km, torch, n, d, dout):
    say(f"pca project shapes n={n} d={d} dout={dout}")
    X = blobs(n, d, 5, seed=n + d + dout) + np.float32(0.25)
    mean = X.astype(np.float64).mean(0).astype(np.float32)
    W = np.linalg.qr(np.random.default_rng(d + dout).standard_normal((d, dout)))[0].astype(np.float32)
    Y_o = orc.project(X, mean, W)
    Y = km.pca_project(to_dev(X, torch), to_dev(mean, torch), to_dev(W, torch))
    torch.cuda.synchronize()
    scale = np.abs(Y_o).max() + 1e-30
    np.testing.assert_allclose(host(Y), Y_o, rtol=0, atol=2e-5 * scale)


# --------------------------------------------------------------------------- Lloyd

def test_fit_f32_lockstep_config1(km, torch):
    """Configuration 1 in full: 20k x 128 Gaussian mixture, k=64, 10 iterations, compared
    step by step (the GPU step is always fed the oracle's centroids)."""
    import synth
    cfg = synth.config(1)
    X = synth.make_points(cfg["spec"])
    k, T = cfg["k"], cfg["iters"]
    idx = synth.init_indices(len(X), k)
    P = km.points_f32(to_dev(X, torch))
    C_o = X[idx].copy()
    for t in range(T + 1):
        say(f"lockstep f32 iteration {t}")
        a_o, dist_o = orc.assign_f32(X, C_o)
        a, _, obj = km.kmeans_assign(P, to_dev(C_o, torch), score=False, objective=True)
        torch.cuda.synchronize()
        assert_fp_assign(host(a), a_o, f32_dist(X, C_o), f"iter {t}")
        assert abs(host(obj)[0] - dist_o.sum()) <= OBJ_REL * dist_o.sum()
        if t == T:
            break
        C_n, cnt_o = orc.update_f32(X, a_o, k, C_o)
        C = to_dev(C_o, torch)
        _, cnt = km.kmeans_update(P, to_dev(a_o, torch), C)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(cnt), cnt_o)
        assert_centroids(host(C), C_n, f"iter {t}")
        C_o = C_n


def test_fit_f32_free_running_config1(km, torch):
    import synth
    cfg = synth.config(1)
    X = synth.make_points(cfg["spec"])
    k, T = cfg["k"], cfg["iters"]
    idx = synth.init_indices(len(X), k)
    C_o, a_o, J_o = orc.fit({"fmt": "f32", "X": X}, k, T, idx)
    C, a, J = km.kmeans_fit(km.points_f32(to_dev(X, torch)), k, T, idx)
    torch.cuda.synchronize()
    assert_fp_assign(host(a), a_o, f32_dist(X, C_o), "free-running")
    np.testing.assert_allclose(host(J), J_o, rtol=OBJ_REL)
    assert_centroids(host(C), C_o, "final")


def test_fit_sq8_bit_exact_trajectory(km, torch):
    """SQ8 Lloyd is all-integer: the whole trajectory must match the oracle exactly."""
    import synth
    spec = synth.config(2)["spec"].with_n(30000)
    X = synth.make_points(spec)
    lo, hi = orc.sq8_fit(X)
    codes = orc.sq8_encode(X, lo, hi)
    k, T = 100, 8
    idx = synth.init_indices(len(X), k)
    C_o, a_o, J_o = orc.fit({"fmt": "sq8", "codes": codes}, k, T, idx)
    C, a, J = km.kmeans_fit(km.points_sq8(to_dev(codes, torch)), k, T, idx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(C), C_o)
    np.testing.assert_array_equal(host(J), np.array(J_o))


def test_fit_sign1_lockstep(km, torch):
    import synth
    spec = synth.config(3)["spec"].with_n(20000)
    X = synth.make_points(spec)
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m)
    k, T, d = 64, 4, spec.d
    idx = synth.init_indices(len(X), k)
    Po = {"fmt": "sign1", "bits": bits, "alpha": alpha, "m": m, "d": d}
    P = km.points_sign1(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), to_dev(m, torch), d)
    C_o = orc.init_centroids(Po, idx)
    Cg, _, _ = km.kmeans_fit(P, k, 0, idx, objective=False)
    np.testing.assert_array_equal(host(Cg), C_o)  # STEP 1 decodes m + alpha (2b - 1) exactly
    for t in range(T):
        say(f"lockstep sign1 iteration {t}")
        a_o, _ = orc.assign(Po, C_o)
        a, _, _ = km.kmeans_assign(P, to_dev(C_o, torch), score=False)
        np.testing.assert_array_equal(host(a), a_o)
        C_n, _ = orc.update(Po, a_o, k, C_o)
        C = to_dev(C_o, torch)
        km.kmeans_update(P, to_dev(a_o, torch), C)
        torch.cuda.synchronize()
        assert_centroids(host(C), C_n, f"iter {t}")
        C_o = C_n


def test_fit_hybrid_lockstep(km, torch):
    import synth
    spec = synth.config(5)["spec"].with_n(20000)
    X = synth.make_points(spec)
    d, d0 = spec.d, 384
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m, d0)
    front = np.ascontiguousarray(X[:, :d0])
    k, T = 64, 3
    idx = synth.init_indices(len(X), k)
    Po = {"fmt": "hybrid", "front": front, "bits": bits, "alpha": alpha, "m": m, "d": d, "d0": d0}
    P = km.points_hybrid(to_dev(front, torch), to_dev(bits.view(np.int32), torch), to_dev(alpha, torch),
                         to_dev(m, torch), d)
    C_o = orc.init_centroids(Po, idx)
    Cg, _, _ = km.kmeans_fit(P, k, 0, idx, objective=False)
    np.testing.assert_array_equal(host(Cg), C_o)
    for t in range(T):
        say(f"lockstep hybrid iteration {t}")
        a_o, dist_o = orc.assign(Po, C_o)
        a, _, obj = km.kmeans_assign(P, to_dev(C_o, torch), score=False, objective=True)
        torch.cuda.synchronize()
        q, sigma, _, _, _ = orc.sign1_prep(C_o, m, d0)
        sgn = np.where(unpack_bits(bits, d)[:, d0:] > 0, 1.0, -1.0)

        def d_of(rows, cands):
            fr = ((front[rows].astype(np.float64) - C_o[cands, :d0]) ** 2).sum(1)
            xt = alpha[rows, None].astype(np.float64) * sgn[rows]
            ct = sigma[cands, None].astype(np.float64) * q[cands]
            mag = (front[rows].astype(np.float64) ** 2).sum(1) + (C_o[cands, :d0].astype(np.float64) ** 2).sum(1) + \
                (xt ** 2).sum(1) + (ct ** 2).sum(1)
            return fr + ((xt - ct) ** 2).sum(1), mag
        assert_fp_assign(host(a), a_o, d_of, f"iter {t}")
        assert abs(host(obj)[0] - dist_o.sum()) <= OBJ_REL * dist_o.sum()
        C_n, _ = orc.update(Po, a_o, k, C_o)
        C = to_dev(C_o, torch)
        km.kmeans_update(P, to_dev(a_o, torch), C)
        torch.cuda.synchronize()
        assert_centroids(host(C), C_n, f"iter {t}")
        C_o = C_n


def test_partition_cost(km, torch):
    X = blobs(5000, 128, 10, seed=3)
    a = rand_assign(5000, 40, seed=2)
    mu, _ = orc.update_f32(X, a, 40, np.zeros((40, 128), np.float32), 1)
    want = orc.partition_cost(X, a, 40)
    Xd = to_dev(X, torch)
    C = torch.zeros((40, 128), dtype=torch.float32, device="cuda")
    km.kmeans_update(km.points_f32(Xd), to_dev(a, torch), C, 1)
    got = host(km.kmeans_cost(Xd, C, to_dev(a, torch)))[0]
    assert abs(got - want) <= 1e-5 * want


def test_fit_k_equals_n_and_k1(km, torch):
    X = blobs(37, 32, 4, seed=8)
    C, a, J = km.kmeans_fit(km.points_f32(to_dev(X, torch)), 37, 2, np.arange(37))
    torch.cuda.synchronize()
    assert host(a).tolist() == list(range(37))
    assert abs(host(J)[-1]) <= 1e-5 * float((X.astype(np.float64) ** 2).sum())
    C, a, J = km.kmeans_fit(km.points_f32(to_dev(X, torch)), 1, 2, [5])
    np.testing.assert_allclose(host(C)[0], X.astype(np.float64).mean(0), rtol=1e-5, atol=1e-6)
