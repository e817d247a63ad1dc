"""GPU parity at the full workload sizes, in the launch configuration bench.py
times, checked on sampled outputs the oracle computes one by one (or through
properties that hold at any size).  Inputs come from the seeded generator or
from the oracle, never from the HIP path.

Workloads: 1M x 768 (fp32, SQ8, bfloat16, LVQ4 and a pruned SQ8 pass, k = 1000), 1M x 1024 1-bit and
RabitQ (k = 1024),
10M x 1024 -> PCA 256 (k = 4096), 10M x 1024 fp32-front-384 + 1-bit (k = 4096) and the
hierarchical FINE phase on 10M x 1024 SQ8 codes (k = 12649).
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import OBJ_REL, assert_centroids, assert_fp_assign, f32_dist, host, say, to_dev, torch_cuda, unpack_bits

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

SAMPLE = 2000


@pytest.fixture(scope="module")
def torch():
    t = torch_cuda()
    import paper_2608_14648_amd  # noqa: F401
    return t


@pytest.fixture(scope="module")
def km(torch):
    import paper_2608_14648_amd as km
    km.lib()
    return km


def generate(spec):
    import synth
    say(f"generating {spec.n} x {spec.d}")
    X = synth.make_points(spec)
    say("generated")
    return X


def sample_rows(n, seed=0):
    return np.sort(np.random.default_rng(seed + 123).choice(n, SAMPLE, replace=False))


@pytest.fixture(scope="module")
def c2(torch):
    import synth
    cfg = synth.config(2)
    X = generate(cfg["spec"])
    Xd = to_dev(X, torch)
    return cfg, X, Xd


@pytest.fixture(scope="module")
def c3(torch):
    import synth
    cfg = synth.config(3)
    X = generate(cfg["spec"])
    return cfg, X, to_dev(X, torch)


# --------------------------------------------------------------------------- 1M x 768

@pytest.mark.timeout(300)
def test_c2_f32_assign_and_update_sampled(km, torch, c2):
    cfg, X, Xd = c2
    import synth
    k = cfg["k"]
    idx = synth.init_indices(len(X), k)
    C = np.ascontiguousarray(X[idx])
    P = km.points_f32(Xd)
    say("c2 f32 assign")
    a, _, obj = km.kmeans_assign(P, to_dev(C, torch), score=False, objective=True)
    torch.cuda.synchronize()
    a = host(a)
    rows = sample_rows(len(X))
    a_o, dist_o = orc.assign_f32(X[rows], C)
    assert_fp_assign(a[rows], a_o, lambda r, c: f32_dist(X[rows], C)(r, c), "c2 f32 sampled")
    # the in-space objective is the sum of fp64 distances to the chosen centroids
    J = host(obj)[0]
    J_o = orc.cost_f32(X, C, a)
    assert abs(J - J_o) <= OBJ_REL * J_o
    say("c2 f32 update")
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    cnt = host(cnt)
    np.testing.assert_array_equal(cnt, np.bincount(a, minlength=k))
    Cn = host(Cd)
    for j in np.random.default_rng(1).choice(np.nonzero(cnt)[0], 25, replace=False):
        members = np.nonzero(a == j)[0].astype(np.int32)
        mj, _ = orc.update_f32(X[members], np.zeros(len(members), np.int32), 1, C[j:j + 1], orc.EMPTY_KEEP)
        assert_centroids(Cn[j:j + 1], mj, f"cluster {j}")


def test_c2_sq8_quantize_assign_sampled(km, torch, c2):
    cfg, X, Xd = c2
    import synth
    k = cfg["k"]
    say("c2 sq8 quantize")
    codes, params = km.quantize_sq8(Xd)
    torch.cuda.synchronize()
    lo, hi = orc.sq8_fit(X)
    p = host(params)
    np.testing.assert_array_equal(p[: X.shape[1]], lo)
    np.testing.assert_array_equal(p[X.shape[1]:], hi)
    rows = sample_rows(len(X), 2)
    codes_h = host(codes)
    np.testing.assert_array_equal(codes_h[rows], orc.sq8_encode(X[rows], lo, hi))
    # assignment on oracle-encoded codes, bit-exact
    codes_o = orc.sq8_encode(X, lo, hi)
    idx = synth.init_indices(len(X), k)
    C = np.ascontiguousarray(codes_o[idx])
    say("c2 sq8 assign")
    a, sc, obj = km.kmeans_assign(km.points_sq8(to_dev(codes_o, torch)), to_dev(C, torch), score=True,
                                  objective=True)
    torch.cuda.synchronize()
    a = host(a)
    a_o, dist_o = orc.assign_sq8(codes_o[rows], C)
    np.testing.assert_array_equal(a[rows], a_o)
    # update: exact integer centroids for sampled clusters
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(km.points_sq8(to_dev(codes_o, torch)), to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), np.bincount(a, minlength=k))
    Cn = host(Cd)
    for j in np.random.default_rng(3).choice(np.nonzero(host(cnt))[0], 25, replace=False):
        members = np.nonzero(a == j)[0]
        mj, _ = orc.update_sq8(codes_o[members], np.zeros(len(members), np.int32), 1, C[j:j + 1], orc.EMPTY_KEEP)
        np.testing.assert_array_equal(Cn[j], mj[0])


def _bf16_dev(codes, torch):
    return to_dev(codes.view(np.int16), torch).view(torch.bfloat16)


@pytest.mark.timeout(300)
def test_c2_bf16_sampled(km, torch, c2):
    """The bfloat16 workload (1M x 768, k = 1000, the 16-wave assignment kernel):
    encoding bit-exact on sampled rows; the assignment of sampled rows within the
    fp tolerance against the oracle and the in-space objective within OBJ_REL; the
    counts exact and sampled clusters' means within the centroid tolerance."""
    cfg, X, Xd = c2
    import synth
    k = cfg["k"]
    say("c2 bf16 encode")
    got = km.quantize_bf16(Xd)
    torch.cuda.synchronize()
    codes_o = orc.bf16_round(X)
    rows = sample_rows(len(X), 4)
    np.testing.assert_array_equal(host(got.view(torch.int16))[rows].view(np.uint16), codes_o[rows])
    del got
    idx = synth.init_indices(len(X), k)
    C = np.ascontiguousarray(X[idx])
    P = km.points_bf16(_bf16_dev(codes_o, torch))
    say("c2 bf16 assign")
    a, _, obj = km.kmeans_assign(P, to_dev(C, torch), score=False, objective=True)
    torch.cuda.synchronize()
    a = host(a)
    Cb = orc.bf16_decode(orc.bf16_round(C))
    a_o, _ = orc.assign_bf16(codes_o[rows], C)
    assert_fp_assign(a[rows], a_o, f32_dist(orc.bf16_decode(codes_o[rows]), Cb), "c2 bf16 sampled")
    J_o = orc.cost_f32(orc.bf16_decode(codes_o), Cb, a)
    assert abs(host(obj)[0] - J_o) <= OBJ_REL * J_o
    say("c2 bf16 update")
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    cnt = host(cnt)
    np.testing.assert_array_equal(cnt, np.bincount(a, minlength=k))
    Cn = host(Cd)
    for j in np.random.default_rng(5).choice(np.nonzero(cnt)[0], 25, replace=False):
        members = np.nonzero(a == j)[0]
        mj, _ = orc.update_bf16(codes_o[members], np.zeros(len(members), np.int32), 1, C[j:j + 1], orc.EMPTY_KEEP)
        assert_centroids(Cn[j:j + 1], mj, f"bf16 cluster {j}")


@pytest.mark.timeout(300)
def test_c2_lvq4_sampled(km, torch, c2):
    """The LVQ4 workload (1M x 768, k = 1000): codes and per-vector parameters
    bit-exact on sampled rows; assignments and scores of sampled rows bit-exact
    against the oracle; the counts exact and sampled clusters' decoded means within
    the centroid tolerance."""
    cfg, X, Xd = c2
    import synth
    k = cfg["k"]
    say("c2 lvq4 encode")
    packed, par = km.quantize_lvq4(Xd)
    torch.cuda.synchronize()
    rows = sample_rows(len(X), 6)
    codes_o, par_o = orc.lvq4_encode(X[rows])
    np.testing.assert_array_equal(host(packed)[rows], orc.lvq4_pack(codes_o))
    np.testing.assert_array_equal(host(par)[rows], par_o)
    idx = synth.init_indices(len(X), k)
    C = np.ascontiguousarray(X[idx])
    P = km.points_lvq4(packed, par, X.shape[1])
    say("c2 lvq4 assign")
    a, sc, _ = km.kmeans_assign(P, to_dev(C, torch), score=True)
    torch.cuda.synchronize()
    a, sc = host(a), host(sc)
    a_o, sc_o, _ = orc.assign_lvq4(codes_o, par_o, C)
    np.testing.assert_array_equal(a[rows], a_o)
    np.testing.assert_array_equal(sc[rows], sc_o)
    say("c2 lvq4 update")
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    cnt = host(cnt)
    np.testing.assert_array_equal(cnt, np.bincount(a, minlength=k))
    Cn = host(Cd)
    pk, pp = host(packed), host(par)
    for j in np.random.default_rng(7).choice(np.nonzero(cnt)[0], 25, replace=False):
        members = np.nonzero(a == j)[0]
        cj, pj = orc.lvq4_encode(X[members])
        mj, _ = orc.update_lvq4(cj, pj, np.zeros(len(members), np.int32), 1, C[j:j + 1], orc.EMPTY_KEEP)
        np.testing.assert_array_equal(pk[members], orc.lvq4_pack(cj))
        np.testing.assert_array_equal(pp[members], pj)
        assert_centroids(Cn[j:j + 1], mj, f"lvq4 cluster {j}")


@pytest.mark.timeout(300)
def test_c2_pruned_sq8_sampled(km, torch, c2):
    """One pruned SQ8 pass of the pruning workload's size (1M x 768, k = 1000, front
    96 dims = 12.5 %, eps0 = 2.1) from a seeded previous assignment: the assignment
    and distance of sampled rows bit-exact against the oracle's pruned pass (a row's
    result depends only on the row, its previous centroid and the centroids)."""
    cfg, X, Xd = c2
    import synth
    k, d = cfg["k"], X.shape[1]
    lo, hi = orc.sq8_fit(X)
    codes_o = orc.sq8_encode(X, lo, hi)
    C = np.ascontiguousarray(codes_o[synth.init_indices(len(X), k)])
    prev = np.random.default_rng(11).integers(0, k, len(X)).astype(np.int32)
    say("c2 pruned sq8 pass")
    a, dist, _, _ = km.kmeans_assign_pruned(km.points_sq8(to_dev(codes_o, torch)), to_dev(C, torch),
                                            to_dev(prev, torch), 2.1, d // 8)
    torch.cuda.synchronize()
    rows = sample_rows(len(X), 10)
    a_o, dist_o, _ = orc.assign_pruned({"fmt": "sq8", "codes": codes_o[rows]}, C, prev[rows], 2.1, d // 8)
    np.testing.assert_array_equal(host(a)[rows], a_o)
    np.testing.assert_array_equal(host(dist)[rows], dist_o)


def test_c2_fit_descends(km, torch, c2):
    cfg, X, Xd = c2
    import synth
    k, T = cfg["k"], cfg["iters"]
    idx = synth.init_indices(len(X), k)
    say("c2 f32 fit")
    C, a, J = km.kmeans_fit(km.points_f32(Xd), k, T, idx, policy=km.KM_EMPTY_KEEP)
    torch.cuda.synchronize()
    J = host(J)
    assert (np.diff(J) <= 1e-6 * J[:-1]).all(), J
    # the reported final objective is the fp64 cost of the final partition against the final centroids
    J_o = orc.cost_f32(X, host(C), host(a))
    assert abs(J[-1] - J_o) <= OBJ_REL * J_o


# --------------------------------------------------------------------------- 1M x 1024 1-bit

@pytest.mark.timeout(300)
def test_c3_sign1_sampled(km, torch, c3):
    cfg, X, Xd = c3
    import synth
    k, d = cfg["k"], cfg["spec"].d
    say("c3 quantize")
    m_o = orc.col_mean(X)
    bits_g, m_g, alpha_g, _ = km.quantize_sign1(Xd)
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(m_g), m_o, rtol=2e-7, atol=1e-9)
    bits_o, alpha_o = orc.sign1_encode(X, m_o)
    rows = sample_rows(len(X), 4)
    bits_g2, _, alpha_g2, _ = km.quantize_sign1(Xd, center=to_dev(m_o, torch))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(bits_g2)[rows].view(np.uint32), bits_o[rows])
    np.testing.assert_allclose(host(alpha_g2)[rows], alpha_o[rows], rtol=2e-7)
    # assignment of oracle-encoded points against decoded initial centroids: bit-exact
    idx = synth.init_indices(len(X), k)
    Po = {"fmt": "sign1", "bits": bits_o, "alpha": alpha_o, "m": m_o, "d": d}
    C = orc.init_centroids(Po, idx)
    P = km.points_sign1(to_dev(bits_o.view(np.int32), torch), to_dev(alpha_o, torch), to_dev(m_o, torch), d)
    say("c3 assign")
    a, sc, _ = km.kmeans_assign(P, to_dev(C, torch), score=True)
    torch.cuda.synchronize()
    a_o, sc_o, _ = orc.assign_sign1(bits_o[rows], alpha_o[rows], C, m_o)
    np.testing.assert_array_equal(host(a)[rows], a_o)
    np.testing.assert_array_equal(host(sc)[rows], sc_o)
    say("c3 update")
    a = host(a)
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), np.bincount(a, minlength=k))
    Cn = host(Cd)
    for j in np.random.default_rng(5).choice(np.nonzero(host(cnt))[0], 20, replace=False):
        members = np.nonzero(a == j)[0]
        mj, _ = orc.update_sign1(bits_o[members], alpha_o[members], d, m_o, np.zeros(len(members), np.int32), 1,
                                 C[j:j + 1], orc.EMPTY_KEEP)
        assert_centroids(Cn[j:j + 1], mj, f"cluster {j}")


@pytest.mark.timeout(300)
def test_c3_rabitq_sampled(km, torch, c3):
    """The RabitQ workload (1M x 1024, k = 1024): the GPU rotation and encoding of
    sampled rows against the oracle's (signs may differ only within rounding of 0);
    then, on oracle-encoded codes of every point (the codes of the centred rows; the
    assignment kernel does not depend on how they were rotated), the assignments and
    scores of sampled rows bit-exact, the counts exact and sampled clusters' means
    within the centroid tolerance."""
    cfg, X, Xd = c3
    import synth
    k, d = cfg["k"], cfg["spec"].d
    say("c3 rabitq encode")
    m_o = orc.col_mean(X)
    Rot = synth.random_rotation(d, 21)
    bits_g, _, alpha_g, Yg = km.rabitq_encode(Xd, to_dev(Rot, torch), center=to_dev(m_o, torch), want_rotated=True)
    torch.cuda.synchronize()
    rows = sample_rows(len(X), 8)
    Y = orc.project(X[rows], m_o, Rot)
    bits_o, alpha_o = orc.sign1_encode(Y, np.zeros(d, np.float32), 0)
    rn = np.linalg.norm(X[rows].astype(np.float64) - m_o.astype(np.float64), axis=1, keepdims=True)
    assert (np.abs(host(Yg)[rows].astype(np.float64) - Y) <= 2e-6 * rn + 1e-12).all()
    diff = unpack_bits(host(bits_g)[rows].view(np.uint32), d) != unpack_bits(bits_o, d)
    scale = np.abs(Y).max(1, keepdims=True) + 1e-30
    assert (np.abs(Y)[diff] <= 1e-5 * np.broadcast_to(scale, Y.shape)[diff]).all()
    np.testing.assert_allclose(host(alpha_g)[rows], alpha_o, rtol=2e-5, atol=1e-7)
    del bits_g, alpha_g, Yg
    # assignment and update on oracle codes of all points
    bits_a, alpha_a = orc.sign1_encode(X, m_o)
    Po = {"fmt": "rabitq", "bits": bits_a, "alpha": alpha_a, "d": d}
    idx = synth.init_indices(len(X), k)
    C = np.ascontiguousarray(X[idx] - m_o)
    P = km.points_rabitq(to_dev(bits_a.view(np.int32), torch), to_dev(alpha_a, torch), d)
    say("c3 rabitq assign")
    a, sc, _ = km.kmeans_assign(P, to_dev(C, torch), score=True)
    torch.cuda.synchronize()
    a, sc = host(a), host(sc)
    a_o, sc_o, _ = orc.assign_rabitq(bits_a[rows], alpha_a[rows], C)
    np.testing.assert_array_equal(a[rows], a_o)
    np.testing.assert_array_equal(sc[rows], sc_o)
    say("c3 rabitq update")
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    cnt = host(cnt)
    np.testing.assert_array_equal(cnt, np.bincount(a, minlength=k))
    Cn = host(Cd)
    for j in np.random.default_rng(9).choice(np.nonzero(cnt)[0], 20, replace=False):
        members = np.nonzero(a == j)[0]
        Pj = {"fmt": "rabitq", "bits": bits_a[members], "alpha": alpha_a[members], "d": d}
        mj, _ = orc.update(Pj, np.zeros(len(members), np.int32), 1, C[j:j + 1], orc.EMPTY_KEEP)
        assert_centroids(Cn[j:j + 1], mj, f"rabitq cluster {j}")


# --------------------------------------------------------------------------- 10M x 1024

@pytest.fixture(scope="module")
def c45(torch):
    import synth
    cfg = synth.config(4)
    X = generate(cfg["spec"])
    Xd = to_dev(X, torch)
    return cfg, X, Xd


@pytest.mark.timeout(600)
def test_hier_sq8_fine_full_size(km, torch, c45):
    """The hierarchical workload's FINE phase at its size (10M x 1024 SQ8 codes, 112
    meso-clusters from seeded labels, k = 12649 fine centroids; the segmented launches
    bench.py times): the fine counts exact, the STEP-1 fine centroids (members of each
    meso-cluster at the strided positions) exact, and the fine assignment of sampled
    rows bit-exact against the nearest centroid of their own meso-cluster's segment."""
    cfg, X, Xd = c45
    n = len(X)
    k_meso, k = 112, 12649
    say("hier fine: oracle SQ8 codes")
    lo, hi = orc.sq8_fit(X)
    codes_o = orc.sq8_encode(X, lo, hi)
    am = np.random.default_rng(12).integers(0, k_meso, n).astype(np.int32)
    say("hier fine: GPU fine phase")
    C, a, kf, _ = km.kmeans_fine(km.points_sq8(to_dev(codes_o, torch)), to_dev(am, torch), k_meso, k, 0)
    torch.cuda.synchronize()
    n_i = np.bincount(am, minlength=k_meso)
    kf_o = orc.fine_counts(n_i, k)
    np.testing.assert_array_equal(kf, kf_o)
    off = np.concatenate([[0], np.cumsum(kf_o)])
    start = np.concatenate([[0], np.cumsum(n_i)])
    order = np.argsort(am, kind="stable")
    C_o = np.empty((k, X.shape[1]), np.uint8)
    for i in range(k_meso):
        members = order[start[i]:start[i + 1]]
        C_o[off[i]:off[i + 1]] = codes_o[members[orc.fine_init_positions(int(n_i[i]), int(kf_o[i]))]]
    np.testing.assert_array_equal(host(C), C_o)
    a = host(a)
    rows = sample_rows(n, 14)
    for i in np.unique(am[rows]):
        ri = rows[am[rows] == i]
        a_o, _ = orc.assign_sq8(codes_o[ri], C_o[off[i]:off[i + 1]])
        np.testing.assert_array_equal(a[ri], a_o + off[i])


@pytest.mark.timeout(600)
def test_c4_pca_full_size(km, torch, c45):
    cfg, X, Xd = c45
    d, dout = cfg["spec"].d, cfg["d_out"]
    say("c4 pca_fit_cov")
    mean_g, cov_g = km.pca_fit_cov(Xd)
    torch.cuda.synchronize()
    mean_o = orc.col_mean64(X)
    np.testing.assert_allclose(host(mean_g), mean_o, rtol=1e-6, atol=1e-8)
    cov_h = host(cov_g).astype(np.float64)
    rng = np.random.default_rng(7)
    pairs = [(0, 0), (0, 1), (5, 700), (1023, 1023), (256, 255)] + [tuple(rng.integers(0, d, 2)) for _ in range(7)]
    for i, j in pairs:
        want = orc.pca_cov_entry(X, mean_o, int(i), int(j))
        assert abs(cov_h[i, j] - want) <= 1e-5 * abs(cov_h[0, 0]) + 1e-5 * abs(want), (i, j, cov_h[i, j], want)
    # projection with a seeded orthonormal basis (an input, not a HIP output)
    W = np.linalg.qr(np.random.default_rng(8).standard_normal((d, dout)))[0].astype(np.float32)
    mean32 = mean_o.astype(np.float32)
    say("c4 pca_project")
    Y = km.pca_project(Xd, to_dev(mean32, torch), to_dev(W, torch))
    torch.cuda.synchronize()
    rows = sample_rows(len(X), 6)
    Yo = orc.project(X[rows], mean32, W)
    np.testing.assert_allclose(host(Y[torch.from_numpy(rows).cuda()]), Yo, rtol=0, atol=2e-5 * np.abs(Yo).max())
    del Y


@pytest.mark.timeout(400)
def test_c4_assign_update_projected_shape(km, torch):
    """Assignment and update at the projected workload's shape: 10M x 256, k = 4096."""
    import synth
    spec = synth.MixtureSpec(10_000_000, 256, 4096, 0.15, True, power=0.5)
    X = generate(spec)
    Xd = to_dev(X, torch)
    idx = synth.init_indices(len(X), 4096)
    C = np.ascontiguousarray(X[idx])
    P = km.points_f32(Xd)
    say("c4 assign")
    a, _, _ = km.kmeans_assign(P, to_dev(C, torch), score=False)
    torch.cuda.synchronize()
    a = host(a)
    rows = sample_rows(len(X), 9)
    a_o, _ = orc.assign_f32(X[rows], C)
    assert_fp_assign(a[rows], a_o, lambda r, c: f32_dist(X[rows], C)(r, c), "10M x 256 sampled")
    say("c4 update")
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    cnt = host(cnt)
    np.testing.assert_array_equal(cnt, np.bincount(a, minlength=4096))
    Cn = host(Cd)
    for j in np.random.default_rng(2).choice(np.nonzero(cnt)[0], 10, replace=False):
        members = np.nonzero(a == j)[0].astype(np.int32)
        mj, _ = orc.update_f32(X[members], np.zeros(len(members), np.int32), 1, C[j:j + 1], orc.EMPTY_KEEP)
        assert_centroids(Cn[j:j + 1], mj, f"cluster {j}")


@pytest.mark.timeout(400)
def test_c5_hybrid_full_size(km, torch, c45):
    cfg5 = __import__("synth").config(5)
    _, X, Xd = c45
    import synth
    d, d0, k = cfg5["spec"].d, cfg5["d_front"], cfg5["k"]
    say("c5 encode (oracle)")
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m, d0)
    rows = sample_rows(len(X), 11)
    say("c5 quantize (gpu, given m)")
    bits_g, _, alpha_g, front_g = km.quantize_sign1(Xd, center=to_dev(m, torch), d_front=d0, want_front=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(bits_g)[rows].view(np.uint32), bits[rows])
    np.testing.assert_allclose(host(alpha_g)[rows], alpha[rows], rtol=2e-7)
    np.testing.assert_array_equal(host(front_g[torch.from_numpy(rows).cuda()]), X[rows, :d0])
    del bits_g, alpha_g
    front = np.ascontiguousarray(X[:, :d0])
    idx = synth.init_indices(len(X), k)
    Po = {"fmt": "hybrid", "front": front, "bits": bits, "alpha": alpha, "m": m, "d": d, "d0": d0}
    C = orc.init_centroids(Po, idx)
    P = km.points_hybrid(front_g, to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), to_dev(m, torch), d)
    say("c5 assign")
    a, _, _ = km.kmeans_assign(P, to_dev(C, torch), score=False)
    torch.cuda.synchronize()
    a = host(a)
    a_o, _ = orc.assign_hybrid(front[rows], bits[rows], alpha[rows], C, m, d0)
    q, sigma, _, _, _ = orc.sign1_prep(C, m, d0)
    sgn = np.where(unpack_bits(bits[rows], d)[:, d0:] > 0, 1.0, -1.0)

    def d_of(r, c):
        fr = ((front[rows][r].astype(np.float64) - C[c, :d0]) ** 2).sum(1)
        xt = alpha[rows][r, None].astype(np.float64) * sgn[r]
        ctl = sigma[c, None].astype(np.float64) * q[c]
        mag = (front[rows][r].astype(np.float64) ** 2).sum(1) + (C[c, :d0].astype(np.float64) ** 2).sum(1) + \
            (xt ** 2).sum(1) + (ctl ** 2).sum(1)
        return fr + ((xt - ctl) ** 2).sum(1), mag
    assert_fp_assign(a[rows], a_o, d_of, "c5 sampled")
    say("c5 update")
    Cd = to_dev(C, torch)
    _, cnt = km.kmeans_update(P, to_dev(a, torch), Cd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), np.bincount(a, minlength=k))
    Cn = host(Cd)
    for j in np.random.default_rng(4).choice(np.nonzero(host(cnt))[0], 10, replace=False):
        members = np.nonzero(a == j)[0]
        mj, _ = orc.update_sign1(bits[members], alpha[members], d, m, np.zeros(len(members), np.int32), 1,
                                 C[j:j + 1], orc.EMPTY_KEEP, front=front[members], d0=d0)
        assert_centroids(Cn[j:j + 1], mj, f"cluster {j}")
