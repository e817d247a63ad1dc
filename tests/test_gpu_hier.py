"""GPU parity of hierarchical k-means (Sec. 4.4, Table 7) against the CPU oracle:
the FINE-CLUSTERING phase on a given meso assignment (per format) and the whole
MESO -> FINE -> REFINE pipeline.  SQ8 runs are bit-exact end to end (integer
arithmetic throughout); the 1-bit, RabitQ and LVQ4 assignments are bit-exact given
the same centroids; fp formats follow the tolerances stated in gpu_util.py.
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import (OBJ_REL, assert_centroids, assert_fp_assign, f32_dist, host, say, to_dev, torch_cuda,
                      unpack_bits)

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


def formats(km, torch, fmt, X):
    """(oracle dict, GPU Points) of the same points in format fmt."""
    d = X.shape[1]
    if fmt == "f32":
        return {"fmt": "f32", "X": X}, km.points_f32(to_dev(X, torch))
    if fmt == "sq8":
        codes = orc.sq8_encode(X, *orc.sq8_fit(X))
        return {"fmt": "sq8", "codes": codes}, km.points_sq8(to_dev(codes, torch))
    if fmt == "bf16":
        codes = orc.bf16_round(X)
        return {"fmt": "bf16", "codes": codes}, km.points_bf16(to_dev(codes.view(np.int16), torch).view(torch.bfloat16))
    if fmt == "lvq4":
        codes, par = orc.lvq4_encode(X)
        return {"fmt": "lvq4", "codes": codes, "par": par}, km.points_lvq4(to_dev(orc.lvq4_pack(codes), torch),
                                                                         to_dev(par, torch), d)
    if fmt == "sign1":
        m = orc.col_mean(X)
        bits, alpha = orc.sign1_encode(X, m)
        return ({"fmt": "sign1", "bits": bits, "alpha": alpha, "m": m, "d": d},
                km.points_sign1(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), to_dev(m, torch), d))
    if fmt == "rabitq":
        import synth
        m = orc.col_mean(X)
        Y = orc.project(X, m, synth.random_rotation(d, 5))
        bits, alpha = orc.sign1_encode(Y, np.zeros(d, np.float32), 0)
        return ({"fmt": "rabitq", "bits": bits, "alpha": alpha, "d": d},
                km.points_rabitq(to_dev(bits.view(np.int32), torch), to_dev(alpha, torch), d))
    if fmt == "hybrid":
        d0 = d // 4
        m = orc.col_mean(X)
        bits, alpha = orc.sign1_encode(X, m, d0)
        front = np.ascontiguousarray(X[:, :d0])
        return ({"fmt": "hybrid", "front": front, "bits": bits, "alpha": alpha, "m": m, "d": d, "d0": d0},
                km.points_hybrid(to_dev(front, torch), to_dev(bits.view(np.int32), torch), to_dev(alpha, torch),
                                 to_dev(m, torch), d))
    raise ValueError(fmt)


def meso_labels(n, k_meso, seed, empty=None, invalid=0):
    rng = np.random.default_rng(seed)
    a = rng.integers(0, k_meso, n).astype(np.int32)
    if empty is not None:
        a[a == empty] = (empty + 1) % k_meso
    if invalid:
        idx = rng.choice(n, invalid, replace=False)
        a[idx[: invalid // 2]] = -1
        a[idx[invalid // 2:]] = k_meso + 2
    return a


# (n, d, k_meso, k, iters, empty meso-cluster, invalid ids); d = 1040 selects without
# packed keys; (700, 16, 5, 700) has meso-clusters on both sides of 128 fine
# centroids, so one pass runs both segment launches (128- and 256-centroid tiles)
SQ8_CASES = [(1, 16, 1, 1, 2, None, 0), (300, 16, 1, 17, 3, None, 0), (1000, 32, 4, 20, 3, None, 0),
             (5000, 64, 10, 100, 4, 3, 20), (3001, 768, 32, 1000, 2, None, 0), (2000, 48, 7, 7, 2, None, 0),
             (700, 16, 5, 700, 1, None, 0), (400, 1040, 3, 300, 1, None, 0), (600, 1040, 2, 400, 1, None, 0)]


@pytest.mark.parametrize("n,d,k_meso,k,iters,empty,invalid", SQ8_CASES)
def test_fine_sq8_bit_exact(km, torch, n, d, k_meso, k, iters, empty, invalid):
    say(f"fine sq8 n={n} d={d} k_meso={k_meso} k={k} iters={iters}")
    X = blobs(n, d, max(2, k // 3), seed=n + d + k)
    Po, Pg = formats(km, torch, "sq8", X)
    am = meso_labels(n, k_meso, seed=n + k, empty=empty, invalid=invalid)
    C_o, a_o, kf_o, J_o = orc.fit_fine(Po, am, k_meso, k, iters)
    C, a, kf, obj = km.kmeans_fine(Pg, to_dev(am, torch), k_meso, k, iters, objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, kf_o)
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(C), C_o)
    assert host(obj)[0] == J_o[-1]


@pytest.mark.parametrize("refine", [0, 1])
def test_hier_sq8_bit_exact(km, torch, refine):
    """The whole pipeline on SQ8 codes of the 768-dim embedding mixture (fewer rows)."""
    import synth
    spec = synth.config(2)["spec"].with_n(30000)
    X = synth.make_points(spec)
    Po, Pg = formats(km, torch, "sq8", X)
    k = 400
    init = synth.init_indices(len(X), orc.meso_count(k))
    say(f"hier sq8 refine={refine}")
    C_o, a_o, J_o, info = orc.fit_hier(Po, k, 4, 3, refine, init)
    C, a, kf, obj, ph = km.kmeans_fit_hier(Pg, k, init, 4, 3, refine, phases=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, info["k_fine"])
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(C), C_o)
    assert host(obj)[0] == J_o
    assert (ph[:2] > 0).all() and (ph >= 0).all()


@pytest.mark.parametrize("n,k_meso,cap", [(5000, 10, 300), (3000, 3, 95)])
def test_fine_sq8_sqrt_rule_bit_exact(km, torch, n, k_meso, cap):
    """The paper's fine counts (round(sqrt(n_i)) per meso-cluster) with C's capacity
    above or at their sum; a meso-cluster is left empty in the first case."""
    say(f"fine sq8 sqrt rule n={n} k_meso={k_meso}")
    X = blobs(n, 64, 30, seed=n + 91)
    Po, Pg = formats(km, torch, "sq8", X)
    am = meso_labels(n, k_meso, seed=n + 92, empty=3 if k_meso > 3 else None)
    C_o, a_o, kf_o, J_o = orc.fit_fine(Po, am, k_meso, cap, 3, sqrt_rule=True)
    assert kf_o.sum() <= cap
    C, a, kf, obj = km.kmeans_fine(Pg, to_dev(am, torch), k_meso, cap, 3, objective=True, sqrt_rule=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, kf_o)
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(C), C_o)
    assert host(obj)[0] == J_o[-1]


def test_fine_sqrt_rule_rejects_a_short_c(km, torch):
    n, k_meso = 2000, 4
    X = blobs(n, 32, 10, seed=93)
    Po, Pg = formats(km, torch, "sq8", X)
    am = meso_labels(n, k_meso, seed=94)
    need = int(orc.fine_counts_sqrt(np.bincount(am, minlength=k_meso)).sum())
    with pytest.raises(RuntimeError, match="fine counts sum"):
        km.kmeans_fine(Pg, to_dev(am, torch), k_meso, need - 1, 1, sqrt_rule=True)


def test_hier_sq8_sqrt_rule_bit_exact(km, torch):
    """The whole pipeline with the paper's fine counts and a refinement over the fine
    centroids made."""
    import synth
    spec = synth.config(2)["spec"].with_n(20000)
    X = synth.make_points(spec)
    Po, Pg = formats(km, torch, "sq8", X)
    k = 1000  # C's capacity: 32 meso-clusters of ~625 points take ~25 fine centroids each
    init = synth.init_indices(len(X), orc.meso_count(k))
    say("hier sq8 sqrt rule")
    C_o, a_o, J_o, info = orc.fit_hier(Po, k, 3, 2, 1, init, sqrt_rule=True)
    C, a, kf, obj, ph = km.kmeans_fit_hier(Pg, k, init, 3, 2, 1, sqrt_rule=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, info["k_fine"])
    np.testing.assert_array_equal(host(a), a_o)
    np.testing.assert_array_equal(host(C), C_o)
    assert host(obj)[0] == J_o


@pytest.mark.parametrize("fmt,d", [("sign1", 128), ("rabitq", 256), ("lvq4", 96), ("sign1", 1536)])
def test_fine_integer_formats_lockstep(km, torch, fmt, d):
    """Assignments bit-exact against the same fine centroids (STEP 1 gather exact as
    well); one fine iteration from the same centroids within the centroid tolerance."""
    n, k_meso, k = 3000, 6, 60
    X = blobs(n, d, 12, seed=d)
    Po, Pg = formats(km, torch, fmt, X)
    am = meso_labels(n, k_meso, seed=d + 1)
    C0_o, a0_o, kf_o, J0_o = orc.fit_fine(Po, am, k_meso, k, 0)
    C0, a0, kf, obj = km.kmeans_fine(Pg, to_dev(am, torch), k_meso, k, 0, objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, kf_o)
    np.testing.assert_array_equal(host(C0), C0_o)
    np.testing.assert_array_equal(host(a0), a0_o)
    assert abs(host(obj)[0] - J0_o[-1]) <= 1e-5 * abs(J0_o[-1])
    C_start = C0_o
    for t in range(2):
        say(f"fine lockstep {fmt} d={d} step {t}")
        C1_o, a1_o, _, _ = orc.fit_fine(Po, am, k_meso, k, 1, C0=C_start)
        C1, a1, _, _ = km.kmeans_fine(Pg, to_dev(am, torch), k_meso, k, 1, C=to_dev(C_start, torch))
        torch.cuda.synchronize()
        assert_centroids(host(C1), C1_o, f"{fmt} fine step {t}")
        # the final pass of the two runs used slightly different centroids: compare it
        # bit-exactly against the oracle's assignment to the GPU's centroids
        Cg = host(C1)
        _, a_chk, _, _ = orc.fit_fine(Po, am, k_meso, k, 0, C0=Cg)
        np.testing.assert_array_equal(host(a1), a_chk)
        C_start = C1_o


@pytest.mark.parametrize("fmt,d", [("lvq4", 32), ("hybrid", 128)])
def test_fine_per_cluster_launch_groups(km, torch, fmt, d):
    """Per-meso-cluster launches (every format but fp32, SQ8 and bf16) whose centroid
    tiles split over groups while the launch over all points would not: 131072
    points and k = 1028 take one group on a 256-CU device (five 256-centroid tiles;
    two groups' rounds tie with one), but each of the four meso-clusters of 32768
    points and 257 fine centroids takes two, so the fine phase must supply the
    per-point merge keys that the preparation for all points leaves out.  LVQ4
    bit-exact against the oracle; the hybrid (32-dim front, 96-dim 1-bit tail: the
    direct-copy hybrid kernel) within the fp tolerance."""
    n, k_meso, k = 131072, 4, 1028
    X = blobs(n, d, 64, seed=7)
    Po, Pg = formats(km, torch, fmt, X)
    am = np.repeat(np.arange(k_meso, dtype=np.int32), n // k_meso)
    say(f"fine {fmt} per-cluster launch groups")
    C0_o, a0_o, kf_o, _ = orc.fit_fine(Po, am, k_meso, k, 0)
    C0, a0, kf, _ = km.kmeans_fine(Pg, to_dev(am, torch), k_meso, k, 0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, kf_o)
    assert (np.asarray(kf) == k // k_meso).all()
    np.testing.assert_array_equal(host(C0), C0_o)
    if fmt == "lvq4":
        np.testing.assert_array_equal(host(a0), a0_o)
    else:
        assert_fp_assign(host(a0), a0_o, hybrid_d_of(Po, C0_o), f"{fmt} per-cluster groups")


def hybrid_d_of(Po, C):
    front, bits, alpha, m, d, d0 = Po["front"], Po["bits"], Po["alpha"], Po["m"], Po["d"], Po["d0"]
    q, sigma, _, _, _ = orc.sign1_prep(C, m, d0)
    sgn = np.where(unpack_bits(bits, d)[:, d0:] > 0, 1.0, -1.0)

    def d_of(rows, cands):
        fr = ((front[rows].astype(np.float64) - C[cands, :d0]) ** 2).sum(1)
        xt = alpha[rows, None].astype(np.float64) * sgn[rows]
        ct = sigma[cands, None].astype(np.float64) * q[cands]
        mag = (front[rows].astype(np.float64) ** 2).sum(1) + (C[cands, :d0].astype(np.float64) ** 2).sum(1) + \
            (xt ** 2).sum(1) + (ct ** 2).sum(1)
        return fr + ((xt - ct) ** 2).sum(1), mag
    return d_of


def fp_d_of(fmt, Po, C):
    if fmt == "f32":
        return f32_dist(Po["X"], C)
    if fmt == "bf16":
        return f32_dist(orc.bf16_decode(Po["codes"]), orc.bf16_decode(orc.bf16_round(C)))
    return hybrid_d_of(Po, C)


@pytest.mark.parametrize("fmt,d", [("f32", 64), ("f32", 768), ("bf16", 256), ("hybrid", 512)])
def test_fine_fp_formats_lockstep(km, torch, fmt, d):
    """STEP 1 gather exact; then, from the same fine centroids at every step, the
    final fine assignment within the fp tolerance (mismatches only at near ties),
    its objective within OBJ_REL, and one fine iteration's centroids within the
    centroid tolerance whenever the two first assignments agree (a near-tie flip
    legitimately moves a centroid, so that step is compared from the next start)."""
    n, k_meso, k = 4000, 8, 96
    X = blobs(n, d, 16, seed=d + 7)
    Po, Pg = formats(km, torch, fmt, X)
    am = meso_labels(n, k_meso, seed=d + 8, empty=5)
    amd = to_dev(am, torch)
    C0_o, _, kf_o, _ = orc.fit_fine(Po, am, k_meso, k, 0)
    C0, _, kf, _ = km.kmeans_fine(Pg, amd, k_meso, k, 0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, kf_o)
    assert kf[5] == 0
    np.testing.assert_array_equal(host(C0), C0_o)
    C_t = C0_o
    compared = 0
    for t in range(4):
        say(f"fine {fmt} d={d} lockstep step {t}")
        _, a_o, _, J_o = orc.fit_fine(Po, am, k_meso, k, 0, C0=C_t)
        _, a, _, obj = km.kmeans_fine(Pg, amd, k_meso, k, 0, C=to_dev(C_t, torch), objective=True)
        torch.cuda.synchronize()
        agree = assert_fp_assign(host(a), a_o, fp_d_of(fmt, Po, C_t), f"{fmt} step {t}")
        assert abs(host(obj)[0] - J_o[-1]) <= OBJ_REL * abs(J_o[-1])
        C_n, _, _, _ = orc.fit_fine(Po, am, k_meso, k, 1, C0=C_t)
        if agree == 1.0:
            C1, _, _, _ = km.kmeans_fine(Pg, amd, k_meso, k, 1, C=to_dev(C_t, torch))
            torch.cuda.synchronize()
            assert_centroids(host(C1), C_n, f"{fmt} fine update {t}")
            compared += 1
        C_t = C_n
    assert compared >= 2


@pytest.mark.parametrize("fmt", ["f32", "bf16"])
def test_fine_large_segments(km, torch, fmt):
    """Meso-clusters of ~200 fine centroids (128 < k_i <= 256): the segmented launch
    takes 256-centroid tiles (bf16: the 16-wave kernel).  From the oracle's STEP-1
    centroids, the fine assignment within the fp tolerance and its objective within
    OBJ_REL."""
    n, d, k_meso, k = 6000, 64, 4, 800
    X = blobs(n, d, 24, seed=31)
    Po, Pg = formats(km, torch, fmt, X)
    am = meso_labels(n, k_meso, seed=32)
    amd = to_dev(am, torch)
    C0_o, _, kf_o, _ = orc.fit_fine(Po, am, k_meso, k, 0)
    assert all(128 < kf_o[i] <= 256 for i in range(k_meso))
    _, a_o, _, J_o = orc.fit_fine(Po, am, k_meso, k, 0, C0=C0_o)
    _, a, kf, obj = km.kmeans_fine(Pg, amd, k_meso, k, 0, C=to_dev(C0_o, torch), objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, kf_o)
    assert_fp_assign(host(a), a_o, fp_d_of(fmt, Po, C0_o), f"{fmt} large segments")
    assert abs(host(obj)[0] - J_o[-1]) <= OBJ_REL * abs(J_o[-1])


def test_hier_pipeline_is_its_phases(km, torch):
    """kmeans_fit_hier equals, bit for bit, its phases called one by one (kmeans_fit for
    MESO, kmeans_fine, kmeans_fit from the fine centroids for REFINE); the fine phase
    on the GPU's meso partition starts from the oracle's rows and its first pass
    agrees with the oracle's within the fp tolerance.  fp32 points of the 768-dim
    mixture (fewer rows)."""
    import synth
    spec = synth.config(2)["spec"].with_n(20000)
    X = synth.make_points(spec)
    Po, Pg = formats(km, torch, "f32", X)
    k = 256
    kmeso = orc.meso_count(k)
    init = synth.init_indices(len(X), kmeso)
    say("hier f32 pipeline")
    C, a, kf, obj, ph, am_h = km.kmeans_fit_hier(Pg, k, init, 5, 4, 1, phases=True, meso=True)
    _, am, _ = km.kmeans_fit(Pg, kmeso, 5, init, objective=False)
    Cf, af, kf2, _ = km.kmeans_fine(Pg, am, kmeso, k, 4)
    Cr, ar, Jr = km.kmeans_fit(Pg, k, 1, None, C=Cf.clone())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(kf, kf2)
    np.testing.assert_array_equal(host(C), host(Cr))
    np.testing.assert_array_equal(host(a), host(ar))
    assert host(obj)[0] == host(Jr)[-1]
    assert (ph > 0).all()
    np.testing.assert_array_equal(host(am_h), host(am))
    am_h = host(am)
    np.testing.assert_array_equal(kf, orc.fine_counts(np.bincount(am_h, minlength=kmeso), k))
    C0_o, a0_o, _, J0_o = orc.fit_fine(Po, am_h, kmeso, k, 0)
    C0, a0, _, obj0 = km.kmeans_fine(Pg, am, kmeso, k, 0, objective=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(C0), C0_o)
    assert_fp_assign(host(a0), a0_o, f32_dist(X, C0_o), "fine pass 0 on the GPU meso partition")
    assert abs(host(obj0)[0] - J0_o[-1]) <= OBJ_REL * J0_o[-1]


def test_fine_split_donor_stays_in_meso_cluster(km, torch):
    """Six identical rows in meso-cluster 0 with three fine centroids (two come out
    empty) next to a 20-member cluster in meso-cluster 1: the split donors are taken
    inside meso-cluster 0, as in the oracle."""
    rng = np.random.default_rng(73)
    v0 = np.array([1.0, 2.0, 3.0, 4.0], np.float32)
    w = np.array([-5.0, 1.0, 0.0, 2.0], np.float32)
    X = np.concatenate([np.repeat(v0[None], 6, 0), np.repeat(w[None], 20, 0),
                        (w + rng.standard_normal((10, 4)) * 0.5).astype(np.float32)])
    am = np.array([0] * 6 + [1] * 30, np.int32)
    C_o, a_o, kf_o, _ = orc.fit_fine({"fmt": "f32", "X": X}, am, 2, 16, 1)
    C, a, kf, _ = km.kmeans_fine(km.points_f32(to_dev(X, torch)), to_dev(am, torch), 2, 16, 1)
    torch.cuda.synchronize()
    assert kf.tolist() == [3, 13] == kf_o.tolist()
    np.testing.assert_array_equal(host(C)[:3], C_o[:3])
    assert_centroids(host(C), C_o, "split donor")
    np.testing.assert_array_equal(host(a)[:6], a_o[:6])
    assert_fp_assign(host(a), a_o, f32_dist(X, C_o), "split donor")
