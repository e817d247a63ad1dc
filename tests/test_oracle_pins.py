"""Pins for the CPU oracle: hand-computed examples, closed forms, invariants and
brute force on tiny inputs.  Each check is independent of the oracle's own code
path (numpy evaluations of a different formula, or values worked out by hand),
so a dropped term, a wrong sign or index, or a transposed operand fails one.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from conftest import load_golden

EPS = 2.0 ** -10


# --------------------------------------------------------------------------
# Hand-computed examples (tests/golden)

def test_lloyd_1d_example(orc):
    g = load_golden("lloyd_1d.json")
    X = np.array(g["X"], np.float32)
    P = {"fmt": "f32", "X": X}
    a0, dist0 = orc.assign(P, X[g["init_idx"]])
    assert a0.tolist() == g["assign0"]
    assert dist0.sum() == g["J0"]
    C, a, J = orc.fit(P, 2, g["iters"], g["init_idx"], orc.EMPTY_KEEP)
    np.testing.assert_array_equal(C, np.array(g["C1"], np.float32))
    assert a.tolist() == g["assign1"]
    assert J == [g["J0"], g["J1"]]


def test_tie_goes_to_smallest_index(orc):
    g = load_golden("tie_smallest_index.json")
    a, _ = orc.assign_f32(np.array(g["X"], np.float32), np.array(g["C"], np.float32))
    assert a.tolist() == g["assign"]
    a, dist = orc.assign_sq8(np.array(g["sq8_codes"], np.uint8), np.array(g["sq8_C"], np.uint8))
    assert a.tolist() == g["sq8_assign"] and dist.tolist() == [25]
    # identical centroids: every point goes to the first copy
    rng = np.random.default_rng(3)
    X = rng.standard_normal((50, 8)).astype(np.float32)
    C = np.repeat(rng.standard_normal((1, 8)).astype(np.float32), 4, axis=0)
    assert (orc.assign_f32(X, C)[0] == 0).all()


def test_sign1_identity_example(orc):
    g = load_golden("sign1_identity.json")
    # a 32-dim vector whose first word is the fixture's; remaining bits 0, remaining q 0
    d = 32
    bits = np.array([[g["bits_word"]]], np.uint32)
    q = np.zeros(d, np.int64)
    q[:4] = g["centroid_residual"]
    b = np.array([(g["bits_word"] >> i) & 1 for i in range(d)])
    assert int(q[b == 1].sum()) == g["set_bit_sum"] and int(q.sum()) == g["total_sum"]
    assert int(np.dot(2 * b - 1, q)) == g["signed_dot"]
    # The oracle's 1-bit score must equal sigma^2 Q - 2 alpha sigma <2b-1, q>.
    # Centroid residual with max |.| = 127 gives sigma = 1 and q = residual exactly.
    m = np.zeros(d, np.float32)
    C = np.zeros((1, d), np.float32)
    C[0, :4] = g["centroid_residual"]
    C[0, 4] = 127.0
    q[4] = 127
    alpha = np.array([0.5], np.float32)
    a, score, _ = orc.assign_sign1(bits, alpha, C, m)
    expect = float((q * q).sum()) - 2 * 0.5 * 1.0 * float(np.dot(2 * b - 1, q))
    assert score[0] == np.float32(expect)


def test_sign1_encode_example(orc):
    g = load_golden("sign1_encode.json")
    d = g["d"]
    x = np.zeros((1, d), np.float32)
    x[0, :4] = g["x_head"]
    bits, alpha = orc.sign1_encode(x, np.zeros(d, np.float32))
    assert bits[0, 0] == g["bits_word"]
    assert alpha[0] == np.float32(g["alpha_num"] / g["alpha_den"])
    dec = orc.sign1_decode(bits, alpha, d, np.zeros(d, np.float32))
    r = x[0].astype(np.float64)
    # <xhat - m, r> = ||r||^2 (the quantisation error is orthogonal to r)
    assert np.dot(dec[0].astype(np.float64), r) == pytest.approx(float(r @ r), rel=1e-6)
    # radius alpha sqrt(d) >= ||r|| (Cauchy-Schwarz)
    assert np.linalg.norm(dec[0]) >= np.linalg.norm(r)


def test_sq8_codes_example(orc):
    g = load_golden("sq8_codes.json")
    X = np.array(g["column"], np.float32)[:, None]
    lo, hi = orc.sq8_fit(X)
    assert lo[0] == g["lo"] and hi[0] == g["hi"]
    assert np.float32(255.0) / (hi[0] - lo[0]) == g["inv"]
    assert orc.sq8_encode(X, lo, hi)[:, 0].tolist() == g["codes"]
    Xc = np.array(g["constant_column"], np.float32)[:, None]
    lo, hi = orc.sq8_fit(Xc)
    assert orc.sq8_encode(Xc, lo, hi)[:, 0].tolist() == g["constant_codes"]


def test_sq8_centroid_rounding_example(orc):
    g = load_golden("sq8_centroid_round.json")
    for case in g["cases"]:
        codes = np.array(case["members"], np.uint8)[:, None]
        a = np.zeros(len(case["members"]), np.int32)
        C, cnt = orc.update_sq8(codes, a, 1, np.zeros((1, 1), np.uint8))
        assert int(C[0, 0]) == case["centroid"], case
        assert cnt.tolist() == [len(case["members"])]


def test_empty_split_example(orc):
    g = load_golden("empty_split.json")
    X = np.array(g["X"], np.float32)
    C, cnt = orc.update_f32(X, np.array(g["assign"], np.int32), g["k"], np.array(g["C_old"], np.float32))
    np.testing.assert_array_equal(C, np.array(g["C_new"], np.float32))
    assert cnt.tolist() == g["counts"]
    # KEEP leaves the empty centroid untouched
    C, _ = orc.update_f32(X, np.array(g["assign"], np.int32), g["k"], np.array(g["C_old"], np.float32),
                          orc.EMPTY_KEEP)
    np.testing.assert_array_equal(C[2], np.array(g["C_old"][2], np.float32))


def test_empty_split_donor_sequence(orc):
    # two empties: the first takes half of cluster 0 (count 8 -> 4/4), the second then
    # sees counts (4, 3, 4, 0): largest is 4, smallest index 0 again.
    X = np.arange(11 * 2, dtype=np.float32).reshape(11, 2)
    a = np.array([0] * 8 + [1] * 3, np.int32)
    C, cnt = orc.update_f32(X, a, 4, np.zeros((4, 2), np.float32))
    mean0 = X[:8].mean(0)
    up, dn = np.float32(1 + EPS), np.float32(1 - EPS)
    p_up = np.array([up, dn], np.float32)
    p_dn = np.array([dn, up], np.float32)
    c0 = mean0.astype(np.float32)
    c2 = c0 * p_up
    c0 = c0 * p_dn
    c3 = c0 * p_up
    c0 = c0 * p_dn
    np.testing.assert_array_equal(C[2], c2)
    np.testing.assert_array_equal(C[3], c3)
    np.testing.assert_array_equal(C[0], c0)
    assert cnt.tolist() == [8, 3, 0, 0]


def test_empty_split_sq8_steps(orc):
    codes = np.array([[0, 255, 10], [0, 255, 10]], np.uint8)
    a = np.zeros(2, np.int32)
    C, _ = orc.update_sq8(codes, a, 2, np.full((2, 3), 77, np.uint8))
    # p = (+1, -1, +1): new = clamp(c + p), donor = clamp(c - p)
    assert C[1].tolist() == [1, 254, 11]
    assert C[0].tolist() == [0, 255, 9]


# --------------------------------------------------------------------------
# Closed forms and invariants

def _blobs(n=600, d=16, comps=6, seed=0, sigma=0.2):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((comps, d)) * 2
    lab = rng.integers(0, comps, n)
    return (mu[lab] + sigma * rng.standard_normal((n, d))).astype(np.float32)


def test_centroid_is_member_mean(orc):
    X = _blobs()
    rng = np.random.default_rng(1)
    k = 7
    a = rng.integers(0, k, len(X)).astype(np.int32)
    C, cnt = orc.update_f32(X, a, k, np.zeros((k, X.shape[1]), np.float32))
    onehot = np.zeros((len(X), k))
    onehot[np.arange(len(X)), a] = 1
    expect = (onehot.T @ X.astype(np.float64)) / onehot.sum(0)[:, None]
    np.testing.assert_allclose(C, expect, rtol=1e-6, atol=1e-7)
    assert cnt.tolist() == np.bincount(a, minlength=k).tolist()


@pytest.mark.parametrize("fmt", ["f32", "sq8"])
def test_lloyd_monotone(orc, fmt):
    X = _blobs(n=800, d=32, comps=10)
    if fmt == "f32":
        P = {"fmt": "f32", "X": X}
    else:
        lo, hi = orc.sq8_fit(X)
        P = {"fmt": "sq8", "codes": orc.sq8_encode(X, lo, hi)}
    idx = np.random.default_rng(5).choice(len(X), 12, replace=False)
    _, _, J = orc.fit(P, 12, 8, idx, orc.EMPTY_KEEP)
    for j0, j1 in zip(J, J[1:]):
        if fmt == "sq8":
            assert j1 <= j0  # exact integers: rounding the mean to the nearest code keeps descent
        else:
            assert j1 <= j0 * (1 + 1e-9)
    assert J[-1] < J[0]


def test_sign1_lloyd_roughly_monotone(orc):
    X = _blobs(n=800, d=64, comps=8, sigma=0.5)
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m)
    P = {"fmt": "sign1", "bits": bits, "alpha": alpha, "m": m, "d": 64}
    idx = np.random.default_rng(2).choice(len(X), 8, replace=False)
    _, _, J = orc.fit(P, 8, 6, idx, orc.EMPTY_KEEP)
    # int8 centroid rounding makes this approximate; it must not drift upward materially
    assert J[-1] <= J[0]
    for j0, j1 in zip(J, J[1:]):
        assert j1 <= j0 * 1.01


def test_k1_is_global_mean_and_kn_is_zero(orc):
    X = _blobs(n=40, d=8)
    P = {"fmt": "f32", "X": X}
    C, a, J = orc.fit(P, 1, 3, [7])
    np.testing.assert_allclose(C[0], X.astype(np.float64).mean(0), rtol=1e-6, atol=1e-7)
    C, a, J = orc.fit(P, len(X), 2, np.arange(len(X)))
    assert J[-1] == 0.0 and a.tolist() == list(range(len(X)))


def test_alpha_matches_rabitq_factor(orc):
    # alpha = (1/sqrt d) ||r|| / <x_bar, x> with x_bar = sign(r)/sqrt d, x = r/||r||
    rng = np.random.default_rng(4)
    d = 96
    X = rng.standard_normal((50, d)).astype(np.float32)
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m)
    r = X.astype(np.float64) - m.astype(np.float64)
    xbar = np.where(r > 0, 1.0, -1.0) / np.sqrt(d)
    cosine = np.einsum("ij,ij->i", xbar, r / np.linalg.norm(r, axis=1, keepdims=True))
    np.testing.assert_allclose(alpha, np.linalg.norm(r, axis=1) / cosine / np.sqrt(d), rtol=2e-6)
    # bits: bit i of row in word i//32 at position i%32
    b = (bits[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1
    np.testing.assert_array_equal(b.reshape(len(X), d).astype(bool), (X - m) > 0)
    # decoded residual: orthogonal error and radius >= ||r||
    dec = orc.sign1_decode(bits, alpha, d, m).astype(np.float64) - m
    np.testing.assert_allclose(np.einsum("ij,ij->i", dec, r), np.einsum("ij,ij->i", r, r), rtol=1e-5)
    assert (np.linalg.norm(dec, axis=1) >= np.linalg.norm(r, axis=1) * (1 - 1e-6)).all()


def test_sign1_alpha_zero_at_mean(orc):
    m = np.linspace(-1, 1, 32).astype(np.float32)
    X = np.tile(m, (3, 1))
    bits, alpha = orc.sign1_encode(X, m)
    assert (alpha == 0).all() and (bits == 0).all()


def test_sign1_tail_alpha(orc):
    rng = np.random.default_rng(9)
    X = rng.standard_normal((20, 64)).astype(np.float32)
    m = orc.col_mean(X)
    bits_full, _ = orc.sign1_encode(X, m, 0)
    bits, alpha = orc.sign1_encode(X, m, 32)
    np.testing.assert_array_equal(bits, bits_full)
    r = (X - m).astype(np.float64)[:, 32:]
    np.testing.assert_allclose(alpha, (r * r).sum(1) / np.abs(r).sum(1), rtol=1e-6)


def test_sq8_codes_match_definition(orc):
    rng = np.random.default_rng(11)
    X = rng.standard_normal((300, 24)).astype(np.float32) * rng.uniform(0.1, 3, 24).astype(np.float32)
    lo, hi = orc.sq8_fit(X)
    np.testing.assert_array_equal(lo, X.min(0))
    np.testing.assert_array_equal(hi, X.max(0))
    codes = orc.sq8_encode(X, lo, hi)
    s = (hi.astype(np.float64) - lo) / 255.0
    approx = np.clip(np.round((X - lo) / s), 0, 255)
    # fp32 (x-lo)*inv vs fp64 (x-lo)/s may differ only at exact .5 boundaries: at most one code
    assert np.abs(codes.astype(int) - approx).max() <= 1
    assert (codes.astype(int) == approx).mean() > 0.999
    assert codes.min(0).tolist() == [0] * 24 and codes.max(0).tolist() == [255] * 24
    # reconstruction error within half a step
    rec = codes * s + lo
    assert (np.abs(rec - X) <= s * 0.5 + 1e-6).all()


def test_pca_cov_and_basis(orc):
    rng = np.random.default_rng(12)
    d = 24
    lam = np.arange(1, d + 1) ** -0.5
    X = (rng.standard_normal((500, d)) * np.sqrt(lam) + 3.0).astype(np.float32)
    mean, cov = orc.pca_cov(X)
    np.testing.assert_allclose(mean, X.astype(np.float64).mean(0), rtol=1e-12)
    np.testing.assert_allclose(cov, np.cov(X.astype(np.float64).T, bias=True), rtol=1e-10, atol=1e-12)
    assert orc.pca_cov_entry(X, mean, 3, 5) == pytest.approx(cov[3, 5], rel=1e-12)
    W, w = orc.pca_basis(cov, d)
    np.testing.assert_allclose(W.T.astype(np.float64) @ W, np.eye(d), atol=1e-5)
    assert (w >= -1e-12).all() and (np.diff(w) <= 0).all()
    # each column: A w = lambda w and largest-|.| entry positive
    for c in range(d):
        np.testing.assert_allclose(cov @ W[:, c], w[c] * W[:, c], atol=1e-5)
        assert W[np.argmax(np.abs(W[:, c])), c] > 0
    Y = orc.project(X, mean.astype(np.float32), W[:, :5])
    np.testing.assert_allclose(Y, (X.astype(np.float64) - mean.astype(np.float32)) @ W[:, :5].astype(np.float64),
                               rtol=1e-5, atol=1e-6)
    # variance captured by the first components is the eigenvalue sum
    assert Y.astype(np.float64).var(0).sum() == pytest.approx(w[:5].sum(), rel=1e-4)


def test_full_rank_pca_keeps_partition(orc):
    # rotation + translation preserve every distance, so Lloyd partitions agree
    X = _blobs(n=500, d=12, comps=5, sigma=0.3)
    mean, cov = orc.pca_cov(X)
    W, _ = orc.pca_basis(cov, 12)
    Y = orc.project(X, mean.astype(np.float32), W)
    idx = np.random.default_rng(7).choice(500, 5, replace=False)
    _, a1, J1 = orc.fit({"fmt": "f32", "X": X}, 5, 6, idx)
    _, a2, J2 = orc.fit({"fmt": "f32", "X": Y}, 5, 6, idx)
    np.testing.assert_array_equal(a1, a2)
    np.testing.assert_allclose(J1, J2, rtol=1e-5)


def test_partition_cost(orc):
    X = _blobs(n=100, d=6)
    a = (np.arange(100) % 4).astype(np.int32)
    mu = np.stack([X[a == j].astype(np.float64).mean(0) for j in range(4)])
    expect = sum(((X[a == j] - mu[j]) ** 2).sum() for j in range(4))
    assert orc.partition_cost(X, a, 4) == pytest.approx(expect, rel=1e-10)
    C = mu.astype(np.float32)
    assert orc.cost_f32(X, C, a) == pytest.approx(
        float(((X.astype(np.float64) - C.astype(np.float64)[a]) ** 2).sum()), rel=1e-12)


def test_hybrid_segment_decomposition(orc):
    # front part exact L2, tail the 1-bit decoded distance: dist = ||x'-c'||^2 + tail
    rng = np.random.default_rng(13)
    n, d, d0, k = 60, 96, 32, 5
    X = rng.standard_normal((n, d)).astype(np.float32)
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m, d0)
    front = np.ascontiguousarray(X[:, :d0])
    C = rng.standard_normal((k, d)).astype(np.float32) * 0.5
    a, dist = orc.assign_hybrid(front, bits, alpha, C, m, d0)
    q, sigma, T, Q, u = orc.sign1_prep(C, m, d0)
    sgn = np.where(((bits[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(n, d), 1.0, -1.0)[:, d0:]
    xt = alpha[:, None].astype(np.float64) * sgn
    ct = sigma[:, None].astype(np.float64) * q
    full = ((front[:, None, :].astype(np.float64) - C[None, :, :d0]) ** 2).sum(-1) + \
        ((xt[:, None, :] - ct[None]) ** 2).sum(-1)
    np.testing.assert_array_equal(a, full.argmin(1))
    np.testing.assert_allclose(dist, full.min(1), rtol=1e-9)


def test_sign1_prep_definition(orc):
    rng = np.random.default_rng(14)
    k, d = 6, 64
    C = rng.standard_normal((k, d)).astype(np.float32)
    m = rng.standard_normal(d).astype(np.float32) * 0.1
    C[3] = m  # a centroid at the mean: sigma 1, q 0
    q, sigma, T, Q, u = orc.sign1_prep(C, m, 0)
    res = C - m
    for j in range(k):
        mx = np.abs(res[j]).max()
        if mx == 0:
            assert sigma[j] == 1 and (q[j] == 0).all()
            continue
        assert sigma[j] == np.float32(mx) / np.float32(127)
        assert np.abs(q[j]).max() == 127
        np.testing.assert_allclose(q[j] * np.float64(sigma[j]), res[j], atol=float(sigma[j]) * 0.5 + 1e-7)
    assert T.tolist() == q.sum(1).tolist() and Q.tolist() == (q.astype(int) ** 2).sum(1).tolist()
    assert u.tolist() == [np.float32(np.float32(s * s) * np.float32(qq)) for s, qq in zip(sigma, Q)]


# --------------------------------------------------------------------------
# Brute force on tiny inputs (hypothesis)

@settings(max_examples=40, deadline=None)
@given(n=st.integers(1, 64), d=st.integers(1, 64), k=st.integers(1, 8), seed=st.integers(0, 2**31 - 1))
def test_assign_f32_bruteforce(orc, n, d, k, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    C = rng.standard_normal((k, d)).astype(np.float32)
    a, dist = orc.assign_f32(X, C)
    D = ((X[:, None, :].astype(np.float64) - C[None].astype(np.float64)) ** 2).sum(-1)
    np.testing.assert_array_equal(a, D.argmin(1))
    np.testing.assert_allclose(dist, D.min(1), rtol=1e-12, atol=1e-12)


@settings(max_examples=40, deadline=None)
@given(n=st.integers(1, 64), d=st.integers(1, 64), k=st.integers(1, 8), seed=st.integers(0, 2**31 - 1))
def test_assign_sq8_bruteforce(orc, n, d, k, seed):
    rng = np.random.default_rng(seed)
    X = rng.integers(0, 256, (n, d)).astype(np.uint8)
    C = rng.integers(0, 256, (k, d)).astype(np.uint8)
    if k > 1 and seed % 3 == 0:
        C[-1] = C[0]  # exact ties must resolve to the smallest index
    a, dist = orc.assign_sq8(X, C)
    D = ((X[:, None, :].astype(np.int64) - C[None].astype(np.int64)) ** 2).sum(-1)
    np.testing.assert_array_equal(a, D.argmin(1))
    np.testing.assert_array_equal(dist, D.min(1))


@settings(max_examples=40, deadline=None)
@given(n=st.integers(1, 64), w=st.integers(1, 2), k=st.integers(1, 8), seed=st.integers(0, 2**31 - 1))
def test_assign_sign1_bruteforce(orc, n, w, k, seed):
    d = 32 * w
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m)
    C = (m + rng.standard_normal((k, d)) * 0.3).astype(np.float32)
    a, score, dist = orc.assign_sign1(bits, alpha, C, m)
    q, sigma, T, Q, u = orc.sign1_prep(C, m)
    sgn = np.where(((bits[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(n, d), 1.0, -1.0)
    xhat = alpha[:, None].astype(np.float64) * sgn      # decoded residual of the point
    chat = sigma[:, None].astype(np.float64) * q         # decoded residual of the centroid
    D = ((xhat[:, None, :] - chat[None]) ** 2).sum(-1)
    # the fp32 score is the decoded distance minus the point-only term alpha^2 d
    S = D - (alpha.astype(np.float64) ** 2 * d)[:, None]
    best = S.min(1)
    np.testing.assert_allclose(score, best, rtol=1e-5, atol=1e-5 * (1 + np.abs(S).max()))
    # the oracle's choice is optimal up to fp32 rounding of the score
    chosen = S[np.arange(n), a]
    assert (chosen <= best + 1e-5 * (1 + np.abs(S).max(1))).all()
    np.testing.assert_allclose(dist, D[np.arange(n), a], rtol=1e-12)


@settings(max_examples=25, deadline=None)
@given(n=st.integers(1, 40), d=st.integers(1, 16), k=st.integers(1, 6), seed=st.integers(0, 2**31 - 1))
def test_update_f32_bruteforce(orc, n, d, k, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    a = rng.integers(0, k, n).astype(np.int32)
    C0 = rng.standard_normal((k, d)).astype(np.float32)
    C, cnt = orc.update_f32(X, a, k, C0, orc.EMPTY_KEEP)
    for j in range(k):
        if (a == j).any():
            np.testing.assert_allclose(C[j], X[a == j].astype(np.float64).mean(0), rtol=1e-6, atol=1e-7)
        else:
            np.testing.assert_array_equal(C[j], C0[j])
    assert cnt.tolist() == np.bincount(a, minlength=k).tolist()


@settings(max_examples=25, deadline=None)
@given(n=st.integers(1, 40), w=st.integers(1, 2), k=st.integers(1, 6), seed=st.integers(0, 2**31 - 1))
def test_update_sign1_bruteforce(orc, n, w, k, seed):
    d = 32 * w
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    m = orc.col_mean(X)
    bits, alpha = orc.sign1_encode(X, m)
    a = rng.integers(0, k, n).astype(np.int32)
    C0 = rng.standard_normal((k, d)).astype(np.float32)
    C, cnt = orc.update_sign1(bits, alpha, d, m, a, k, C0, orc.EMPTY_KEEP)
    dec = m.astype(np.float64) + alpha[:, None].astype(np.float64) * (2 * _unpack_bits(bits, d) - 1)  # m + alpha(2b-1)
    for j in range(k):
        if (a == j).any():
            # fused decode-average == average of decoded points (m is common)
            np.testing.assert_allclose(C[j], dec[a == j].mean(0), rtol=1e-5, atol=1e-6)
        else:
            np.testing.assert_array_equal(C[j], C0[j])


def _unpack_bits(bits, d):
    """{0, 1} matrix (n x d) of LSB-first uint32 sign words, by numpy shifts."""
    n = bits.shape[0]
    return ((bits[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(n, d).astype(np.int64)


def _padded_front(front, d):
    """The front rows (n x d0) as the leading rows of a larger contiguous buffer
    whose other rows hold 1e6: a read with the row stride of the whole vector
    stays inside memory and returns values far from every real one."""
    n, d0 = front.shape
    buf = np.full((n * (d // d0 + 1) + 1, d0), 1e6, np.float32)
    buf[:n] = front
    return buf[:n]


def _split_reference(Z, cnt):
    """Empty-cluster rule (Sec. 2.3 STEP 3 reading): ascending empty j, donor the
    largest working count (first on ties), halves of the donor's count."""
    k, d = Z.shape
    Z = Z.copy()
    work = cnt.copy()
    fresh = cnt > 0
    p = np.where(np.arange(d) % 2 == 0, 1.0, -1.0)
    for j in range(k):
        if cnt[j] != 0:
            continue
        b = int(np.argmax(work))
        if work[b] < 2:
            continue
        Z[j] = Z[b] * (1.0 + EPS * p)
        Z[b] = Z[b] * (1.0 - EPS * p)
        work[j] = work[b] // 2
        work[b] -= work[j]
        fresh[j] = True
    return Z, fresh


def _golden_rows(g, part, rows, d, d0):
    out = np.empty((rows, d), np.float64)
    even = np.arange(d) % 2 == 0
    for r in range(rows):
        out[r, :d0] = np.where(even[:d0], part["front_even"][r], part["front_odd"][r])
        out[r, d0:] = np.where(even[d0:], part["tail_even"][r], part["tail_odd"][r])
    return out


def _golden_hybrid_inputs(g):
    d, d0 = g["d"], g["d0"]
    n = len(g["alpha"])
    front = np.repeat(np.array(g["front_value"], np.float32)[:, None], d0, axis=1)
    bits = np.array(g["words"], np.uint32)
    alpha = np.array(g["alpha"], np.float32)
    m = np.concatenate([np.full(d0, g["m_front"]), np.full(d - d0, g["m_tail"])]).astype(np.float32)
    C_old = np.repeat(np.array(g["C_old_value"], np.float32)[:, None], d, axis=1)
    return n, d, d0, front, bits, alpha, m, C_old


def test_update_hybrid_example(orc):
    g = load_golden("hybrid_update.json")
    n, d, d0, front, bits, alpha, m, C_old = _golden_hybrid_inputs(g)
    a = np.array(g["assign"], np.int32)
    for policy, key in ((orc.EMPTY_KEEP, "keep"), (orc.EMPTY_SPLIT, "split")):
        C, cnt = orc.update_sign1(bits, alpha, d, m, a, g["k"], C_old, policy,
                                  front=_padded_front(front, d), d0=d0)
        np.testing.assert_array_equal(C, _golden_rows(g, g[key], g["k"], d, d0).astype(np.float32), err_msg=key)
        assert cnt.tolist() == g["counts"]


def test_init_hybrid_example(orc):
    g = load_golden("hybrid_update.json")
    n, d, d0, front, bits, alpha, m, _ = _golden_hybrid_inputs(g)
    P = {"fmt": "hybrid", "front": front, "bits": bits, "alpha": alpha, "m": m, "d": d, "d0": d0}
    C = orc.init_centroids(P, g["init_idx"])
    np.testing.assert_array_equal(C, _golden_rows(g, g["init"], len(g["init_idx"]), d, d0).astype(np.float32))


@settings(max_examples=40, deadline=None)
@given(n=st.integers(1, 40), shape=st.sampled_from([(64, 32), (128, 32), (416, 384), (448, 384)]),
       k=st.integers(1, 6), split=st.booleans(), seed=st.integers(0, 2**31 - 1))
def test_update_hybrid_bruteforce(orc, n, shape, k, split, seed):
    d, d0 = shape
    rng = np.random.default_rng(seed)
    front = rng.standard_normal((n, d0)).astype(np.float32)
    bits = rng.integers(0, 2**32, (n, d // 32), dtype=np.uint64).astype(np.uint32)
    alpha = rng.uniform(0.05, 2.0, n).astype(np.float32)
    m = (rng.standard_normal(d) * 0.5).astype(np.float32)
    a = rng.integers(0, max(1, k - (seed % 3)), n).astype(np.int32)  # some draws leave clusters empty
    C0 = rng.standard_normal((k, d)).astype(np.float32)
    policy = orc.EMPTY_SPLIT if split else orc.EMPTY_KEEP
    C, cnt = orc.update_sign1(bits, alpha, d, m, a, k, C0, policy, front=_padded_front(front, d), d0=d0)
    # clustering-space members: front values, and tail residuals alpha (2b - 1)
    V = np.concatenate([front.astype(np.float64),
                        alpha[:, None].astype(np.float64) * (2 * _unpack_bits(bits, d)[:, d0:] - 1)], axis=1)
    counts = np.bincount(a, minlength=k)
    Z = np.zeros((k, d))
    for j in range(k):
        if counts[j]:
            Z[j] = V[a == j].mean(0)
    fresh = counts > 0
    if split:
        Z, fresh = _split_reference(Z, counts)
    expect = C0.astype(np.float64).copy()
    for j in range(k):
        if fresh[j]:
            expect[j, :d0] = Z[j, :d0]
            expect[j, d0:] = m[d0:].astype(np.float64) + Z[j, d0:]
    np.testing.assert_allclose(C, expect, rtol=1e-6, atol=1e-6)
    assert cnt.tolist() == counts.tolist()


@settings(max_examples=20, deadline=None)
@given(n=st.integers(1, 30), shape=st.sampled_from([(64, 32), (416, 384)]), seed=st.integers(0, 2**31 - 1))
def test_init_hybrid_bruteforce(orc, n, shape, seed):
    d, d0 = shape
    rng = np.random.default_rng(seed)
    front = rng.standard_normal((n, d0)).astype(np.float32)
    bits = rng.integers(0, 2**32, (n, d // 32), dtype=np.uint64).astype(np.uint32)
    alpha = rng.uniform(0.05, 2.0, n).astype(np.float32)
    m = (rng.standard_normal(d) * 0.5).astype(np.float32)
    idx = rng.permutation(n)[: max(1, n // 2)]
    P = {"fmt": "hybrid", "front": front, "bits": bits, "alpha": alpha, "m": m, "d": d, "d0": d0}
    C = orc.init_centroids(P, idx)
    sgn = 2 * _unpack_bits(bits, d)[:, d0:] - 1
    np.testing.assert_array_equal(C[:, :d0], front[idx])
    np.testing.assert_allclose(C[:, d0:], m[d0:].astype(np.float64) + alpha[idx, None].astype(np.float64) * sgn[idx],
                               rtol=1e-7, atol=1e-7)


def test_hybrid_fit_with_constant_tail_is_front_lloyd(orc):
    # every row's tail equals the column mean: residuals are zero, so alpha = 0, the
    # tail adds nothing to any distance and every centroid's tail stays m; the
    # hybrid fit is then plain Lloyd on the front dims (numpy, fp64)
    rng = np.random.default_rng(31)
    n, d, d0, k, T = 300, 96, 32, 5, 6
    centers = rng.standard_normal((k, d0)) * 3
    Xf = (centers[rng.integers(0, k, n)] + rng.standard_normal((n, d0)) * 0.5).astype(np.float32)
    tail = rng.standard_normal(d - d0).astype(np.float32)
    X = np.concatenate([Xf, np.repeat(tail[None], n, axis=0)], axis=1)
    m = orc.col_mean(X)
    assert np.array_equal(m[d0:], tail)
    bits, alpha = orc.sign1_encode(X, m, d0)
    assert (alpha == 0).all()
    idx = rng.choice(n, k, replace=False)
    P = {"fmt": "hybrid", "front": _padded_front(Xf, d), "bits": bits, "alpha": alpha, "m": m, "d": d, "d0": d0}
    C, a, J = orc.fit(P, k, T, idx)
    Cr = Xf[idx].astype(np.float64)
    Xd = Xf.astype(np.float64)
    Jr = []
    for t in range(T + 1):
        D = ((Xd[:, None, :] - Cr[None]) ** 2).sum(-1)
        ar = D.argmin(1)
        Jr.append(D.min(1).sum())
        if t < T:
            for j in range(k):
                if (ar == j).any():
                    Cr[j] = Xd[ar == j].mean(0)
    np.testing.assert_array_equal(a, ar)
    np.testing.assert_allclose(C[:, :d0], Cr, rtol=1e-5, atol=1e-6)
    np.testing.assert_array_equal(C[:, d0:], np.repeat(tail[None], k, axis=0))
    np.testing.assert_allclose(J, Jr, rtol=1e-6)


def test_col_mean_and_sq8_fit_special_cases(orc):
    rng = np.random.default_rng(21)
    X = (rng.standard_normal((513, 40)) * 3 + 1).astype(np.float32)
    np.testing.assert_allclose(orc.col_mean(X), X.astype(np.float64).mean(0), rtol=1e-6, atol=1e-7)
    # a single row is its own mean and its own (lo, hi)
    x1 = X[:1]
    np.testing.assert_array_equal(orc.col_mean(x1), x1[0])
    lo, hi = orc.sq8_fit(x1)
    np.testing.assert_array_equal(lo, x1[0])
    np.testing.assert_array_equal(hi, x1[0])


# --------------------------------------------------------------------------
# bfloat16 storage (16-bit full-precision vectors, Sec. 2.4)

def _f32(bits):
    return np.array([bits], np.uint32).view(np.float32)[0]


def test_bf16_rounding_hand_examples(orc):
    """Nearest bfloat16 with ties to the even significand, worked out by hand:
    bfloat16 keeps the top 16 bits of the fp32 pattern, so the discarded half is
    compared with 0x8000 (exactly 0x8000 = a tie)."""
    cases = [
        (1.0, 0x3F80),
        (1.0 + 2.0 ** -8, 0x3F80),            # tie, 0x3F80 is even
        (1.0 + 3 * 2.0 ** -8, 0x3F82),        # tie between 0x3F81 (odd) and 0x3F82
        (1.0 + 2.0 ** -8 + 2.0 ** -23, 0x3F81),  # just above the tie
        (-2.5, 0xC020),
        (-0.0, 0x8000),
        (2.0 ** -133, 0x0001),                # smallest bfloat16 subnormal
        (3 * 2.0 ** -134, 0x0002),            # tie between 1 and 2 units of 2^-133
        (2.0 ** -134, 0x0000),                # tie between 0 and 1 unit
        (2.0 ** -149, 0x0000),
        (_f32(0x7F7F7FFF), 0x7F7F),           # below the tie: largest finite bfloat16
        (_f32(0x7F7FFFFF), 0x7F80),           # largest fp32 rounds past it: +inf
        (np.inf, 0x7F80),
        (-np.inf, 0xFF80),
    ]
    X = np.array([c[0] for c in cases], np.float32)
    got = orc.bf16_round(X)
    assert [int(g) for g in got] == [c[1] for c in cases]
    nan = orc.bf16_round(np.array([np.nan], np.float32))[0]
    assert (int(nan) & 0x7F80) == 0x7F80 and (int(nan) & 0x7F) != 0


def test_bf16_rounding_matches_library(orc):
    """Special case that reduces to a library routine: torch's fp32 -> bfloat16
    conversion on the CPU (round to nearest, ties to even) on values spanning the
    whole exponent range, exact ties included."""
    import torch
    rng = np.random.default_rng(31)
    u = rng.integers(0, 2 ** 32, 200_000, dtype=np.uint64).astype(np.uint32)
    u = u[(u & 0x7F800000) != 0x7F800000]                   # finite patterns, subnormals included
    ties = (u & 0xFFFF0000) | 0x8000                          # exact ties
    X = np.concatenate([u, ties]).view(np.float32)
    ref = torch.from_numpy(X.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(orc.bf16_round(X), ref)


def test_bf16_steps_on_representable_data_equal_f32(orc):
    """Points and centroids that are already bfloat16 values: the bfloat16 steps
    must give exactly the fp32 steps (rounding is the identity on them), and the
    rounding error bound |x - bf16(x)| <= 2^-8 |x| (unit roundoff of 8 significant
    bits) holds on normal values."""
    rng = np.random.default_rng(32)
    X = rng.standard_normal((300, 48)).astype(np.float32)
    codes = orc.bf16_round(X)
    Xb = orc.bf16_decode(codes)
    assert np.all(np.abs(Xb.astype(np.float64) - X) <= 2.0 ** -8 * np.abs(X.astype(np.float64)))
    np.testing.assert_array_equal(orc.bf16_round(Xb), codes)  # idempotent
    C = Xb[[3, 70, 150, 220, 299]].copy()
    a16, d16 = orc.assign_bf16(codes, C)
    a32, d32 = orc.assign_f32(Xb, C)
    np.testing.assert_array_equal(a16, a32)
    np.testing.assert_array_equal(d16, d32)
    C16, n16 = orc.update_bf16(codes, a16, 5, C)
    C32, n32 = orc.update_f32(Xb, a32, 5, C)
    np.testing.assert_array_equal(C16, C32)
    np.testing.assert_array_equal(n16, n32)
    # a cluster whose members all hold one value keeps exactly that value
    same = np.repeat(codes[:1], 7, axis=0)
    Cm, _ = orc.update_bf16(same, np.zeros(7, np.int32), 1, np.zeros((1, 48), np.float32))
    np.testing.assert_array_equal(Cm[0], Xb[0])


# --------------------------------------------------------------------------
# RabitQ with SQ4 centroid codes (Sec. 3.1, Eq. 3-5) and the raw-vector last update

def test_rabitq_eq5_example(orc):
    """Hand-worked Eq. 5 example: codes, sums and the estimator, evaluated directly as
    sum_i (2 xbar_i - 1)(b + s ybar_i) over the 32 dims."""
    g = load_golden("rabitq_eq5.json")
    d = g["d"]
    C = np.zeros((1, d), np.float32)
    C[0, :4] = g["centroid_residual_head"]
    q, s, b, T, N = orc.rabitq_prep(C)
    s32 = np.float32(g["scale_fraction"][0]) / np.float32(g["scale_fraction"][1])
    assert b[0] == g["bias"] and s[0] == s32
    assert q[0, :4].tolist() == g["codes_head"] and (q[0, 4:] == g["code_of_zero"]).all()
    assert int(T[0]) == g["T"] and float(N[0]) == g["centroid_norm_sq"]
    bits = np.zeros((1, 1), np.uint32)
    bits[0, 0] = g["bits_word"]
    xb = np.array([(g["bits_word"] >> i) & 1 for i in range(d)])
    assert int(q[0][xb == 1].sum()) == g["D"] and int(xb.sum()) == g["popcount"]
    direct = float(np.sum((2.0 * xb - 1.0) * (float(b[0]) + float(s[0]) * q[0].astype(np.float64))))
    hand = g["estimator_constant"] + g["estimator_s_coefficient"] * float(s[0])
    assert abs(direct - hand) < 1e-6
    alpha = np.array([0.5], np.float32)
    a, score, dist = orc.assign_rabitq(bits, alpha, C)
    # score = N - 2 alpha <2xbar - 1, b + s q>, to fp32 rounding
    assert abs(float(score[0]) - (g["centroid_norm_sq"] - 2 * 0.5 * hand)) < 1e-5
    assert abs(dist[0] - (0.25 * d + float(score[0]))) < 1e-9


def test_rabitq_sq4_code_properties(orc):
    """Per-centroid SQ4: bias = min, 15 s = max - min, codes in [0, 15] with the min
    at 0 and the max at 15, reconstruction within half a step; a constant centroid
    codes to 0 with s = 1 and reconstructs exactly."""
    rng = np.random.default_rng(41)
    C = (rng.standard_normal((20, 64)) * rng.uniform(0.1, 3.0, (20, 1))).astype(np.float32)
    C[3] = 0.75
    q, s, b, T, N = orc.rabitq_prep(C)
    C64 = C.astype(np.float64)
    np.testing.assert_array_equal(b, C.min(1))
    live = np.arange(20) != 3
    np.testing.assert_allclose(15.0 * s[live], C64.max(1)[live] - C64.min(1)[live], rtol=1e-6)
    assert q.min() >= 0 and q.max() <= 15
    assert (q[live].min(1) == 0).all() and (q[live].max(1) == 15).all()
    rec = b[:, None].astype(np.float64) + s[:, None].astype(np.float64) * q
    assert (np.abs(rec - C64) <= 0.5 * s[:, None] * (1 + 1e-5)).all()
    assert s[3] == 1.0 and (q[3] == 0).all() and rec[3, 0] == 0.75
    np.testing.assert_array_equal(T, q.astype(np.int64).sum(1))
    np.testing.assert_allclose(N, (C64 ** 2).sum(1), rtol=1e-6)


def test_rabitq_estimator_unbiased_over_rotations(orc):
    """RabitQ's estimator of <x_r - m, y_r - m> (Eq. 4-5) is unbiased over random
    rotations: averaging alpha <2 xbar - 1, SQ4(P y)> over many seeded rotations P
    recovers the exact inner product within a few standard errors (the SQ4 rounding
    of the rotated centroid behaves as zero-mean noise).  A dropped bias term, a
    wrong sign or a wrong scale of alpha moves the mean far outside."""
    import synth
    d = 64
    rng = np.random.default_rng(43)
    r = rng.standard_normal(d).astype(np.float32)
    y = (0.6 * r + 0.8 * rng.standard_normal(d)).astype(np.float32)
    exact = float(np.dot(r.astype(np.float64), y.astype(np.float64)))
    est = []
    for t in range(3000):
        P = synth.random_rotation(d, seed=1000 + t)
        rp = (r.astype(np.float64) @ P.astype(np.float64)).astype(np.float32)[None, :]
        yp = (y.astype(np.float64) @ P.astype(np.float64)).astype(np.float32)[None, :]
        bits, alpha = orc.sign1_encode(rp, np.zeros(d, np.float32), 0)
        _, score, _ = orc.assign_rabitq(bits, alpha, yp)
        _, _, _, _, N = orc.rabitq_prep(yp)
        est.append((float(N[0]) - float(score[0])) / 2.0)  # alpha * <2xbar - 1, b + s q>
    est = np.array(est)
    se = est.std() / np.sqrt(len(est))
    assert abs(est.mean() - exact) < 5 * se + 1e-3 * abs(exact), (est.mean(), exact, se)


@settings(max_examples=25, deadline=None)
@given(n=st.integers(1, 40), w=st.integers(1, 2), k=st.integers(1, 7), seed=st.integers(0, 10_000))
def test_assign_rabitq_bruteforce(orc, n, w, k, seed):
    """Against an explicit fp64 evaluation of N_j - 2 alpha <2 xbar - 1, b_j + s_j q_j>
    over the decoded sign vectors; disagreements only at fp32 near-ties."""
    d = 32 * w
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    C = rng.standard_normal((k, d)).astype(np.float32)
    bits, alpha = orc.sign1_encode(X, np.zeros(d, np.float32), 0)
    a, score, _ = orc.assign_rabitq(bits, alpha, C)
    q, s, b, T, N = orc.rabitq_prep(C)
    sgn = ((bits[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(n, d).astype(np.float64) * 2 - 1
    rec = b[:, None].astype(np.float64) + s[:, None].astype(np.float64) * q
    est = N[None, :].astype(np.float64) - 2 * alpha[:, None].astype(np.float64) * (sgn @ rec.T)
    ref = est.argmin(1)
    gap = est[np.arange(n), a] - est[np.arange(n), ref]
    assert (gap <= 1e-4 * (1 + np.abs(est).max())).all()


def test_fit_raw_last_update(orc):
    """With raw rows given, the last Lloyd update averages them: the final centroids
    are the raw-row means of the clusters of the last-but-one assignment pass
    (explicit one-hot means), and the final pass assigns against them."""
    import synth
    rng = np.random.default_rng(47)
    d, n, k, T = 64, 600, 6, 3
    Xr = rng.standard_normal((n, d)).astype(np.float32)
    P = synth.random_rotation(d, seed=5)
    Y = (Xr.astype(np.float64) @ P.astype(np.float64)).astype(np.float32)
    bits, alpha = orc.sign1_encode(Y, np.zeros(d, np.float32), 0)
    Pd = {"fmt": "rabitq", "bits": bits, "alpha": alpha, "d": d, "raw": Y}
    idx = rng.choice(n, k, replace=False)
    C, a, J = orc.fit(Pd, k, T, idx)
    C2, a2, J2 = orc.fit({k_: v for k_, v in Pd.items() if k_ != "raw"}, k, T - 1, idx)
    a_last, _ = orc.assign(Pd, C2)
    for j in range(k):
        mem = Y[a_last == j].astype(np.float64)
        if len(mem):
            np.testing.assert_allclose(C[j], mem.mean(0), rtol=1e-6, atol=1e-6)
    a_fin, _ = orc.assign(Pd, C)
    np.testing.assert_array_equal(a, a_fin)


# --------------------------------------------------------------------------
# LVQ4 (Sec. 3.1 LVQ, Eq. 1-2)

def test_lvq4_hand_example(orc):
    """Codes, per-vector terms and the Eq. 2 distance of a hand-worked example with
    exact scales; the winning score plus N_x is the decoded squared distance."""
    g = load_golden("lvq4_eq2.json")
    V = np.array(g["vectors"], np.float32)
    codes, par = orc.lvq4_encode(V)
    assert codes.tolist() == g["codes"]
    assert par[:, 0].tolist() == g["scale"] and par[:, 1].tolist() == g["bias"]
    assert par[:, 2].tolist() == g["A"] and par[:, 3].tolist() == g["N"]
    p = g["point"]
    assert int(codes[p].astype(np.int64) @ codes[2].astype(np.int64)) == g["dot_point_centroid2"]
    C = V[g["centroids"]]
    a, score, dist = orc.assign_lvq4(codes[p:p + 1], par[p:p + 1], C)
    assert int(a[0]) == g["assign"] and float(score[0]) == g["scores"][g["assign"]]
    assert dist[0] == g["decoded_distance"]


def test_lvq4_cached_terms_and_eq2_identity(orc):
    """A_x is the sum and N_x the squared norm of the decoded vector, and N_x + score is
    the squared distance between decoded point and decoded centroid (Eq. 2), checked
    against explicit fp64 evaluations on the decoded vectors."""
    rng = np.random.default_rng(51)
    X = (rng.standard_normal((200, 96)) * rng.uniform(0.2, 3, (200, 1)) + rng.normal(0, 1, (200, 1))).astype(np.float32)
    codes, par = orc.lvq4_encode(X)
    dec = orc.lvq4_decode(codes, par).astype(np.float64)
    np.testing.assert_allclose(par[:, 2], dec.sum(1), rtol=2e-6, atol=1e-4)
    np.testing.assert_allclose(par[:, 3], (dec ** 2).sum(1), rtol=2e-6)
    assert (np.abs(dec - X) <= 0.5 * par[:, :1] * (1 + 1e-5)).all()  # within half a step
    C = X[:7] * 1.1
    a, score, dist = orc.assign_lvq4(codes, par, C)
    cdec = orc.lvq4_decode(*orc.lvq4_encode(C)).astype(np.float64)
    full = ((dec[:, None, :] - cdec[None, :, :]) ** 2).sum(-1)
    np.testing.assert_allclose(dist, full[np.arange(len(X)), a], rtol=1e-5, atol=1e-3)
    gap = full[np.arange(len(X)), a] - full.min(1)
    assert (gap <= 1e-5 * (1 + full.max())).all()


def test_lvq4_update_is_decoded_mean(orc):
    rng = np.random.default_rng(53)
    X = rng.standard_normal((500, 64)).astype(np.float32)
    codes, par = orc.lvq4_encode(X)
    dec = orc.lvq4_decode(codes, par).astype(np.float64)
    k = 9
    a = rng.integers(0, k - 1, 500).astype(np.int32)  # cluster k-1 stays empty
    C0 = rng.standard_normal((k, 64)).astype(np.float32)
    C, cnt = orc.update_lvq4(codes, par, a, k, C0, orc.EMPTY_KEEP)
    for j in range(k - 1):
        np.testing.assert_allclose(C[j], dec[a == j].mean(0), rtol=1e-6, atol=1e-6)
    np.testing.assert_array_equal(C[k - 1], C0[k - 1])
    np.testing.assert_array_equal(cnt, np.bincount(a, minlength=k))


# --------------------------------------------------------------------------
# Hierarchical k-means (Sec. 4.4, Table 7)

def test_hier_meso_count_and_fine_counts_hand_examples(orc):
    g = load_golden("hier_fine_counts.json")
    for k, m in g["meso_count"].items():
        assert orc.meso_count(int(k)) == m
    for k in list(range(1, 2000)) + [4096, 10000, 12649, 40000]:
        assert orc.meso_count(k) == int(np.floor(np.sqrt(k) + 0.5)), k
    for case in g["cases"]:
        assert orc.fine_counts(case["n"], case["k"]).tolist() == case["k_fine"], case


def test_fine_counts_sqrt_rule(orc):
    """The paper's fine counts: hand values, then for every n up to 20000 the count is
    the unique integer within 1/2 of sqrt(n) (floating point decides nothing here:
    (c - 1/2)^2 < n < (c + 1/2)^2 in integers is 4c^2 - 4c + 1 < 4n < 4c^2 + 4c + 1)."""
    g = load_golden("hier_fine_counts.json")["sqrt_rule"]
    assert orc.fine_counts_sqrt(g["n"]).tolist() == g["k_fine"]
    ks = orc.fine_counts_sqrt(range(20001))
    assert ks[0] == 0
    for v in range(1, 20001):
        c = int(ks[v])
        assert 1 <= c <= v and 4 * c * c - 4 * c + 1 < 4 * v < 4 * c * c + 4 * c + 1, (v, c)


def test_fine_sqrt_rule_fit(orc):
    """fit_fine with the paper's counts: k_i = fine_counts_sqrt(n_i), C holds their sum,
    each meso-cluster's points keep to its own segment of centroids, and a larger k
    than needed changes nothing; fit_hier refines over the fine centroids made."""
    X = _blob_rows(500, 8, 83)
    a_meso = np.random.default_rng(84).integers(0, 4, 500).astype(np.int32)
    a_meso[a_meso == 2] = 3  # an empty meso-cluster
    P = {"fmt": "f32", "X": X}
    n_i = np.bincount(a_meso, minlength=4)
    C, a, ks, J = orc.fit_fine(P, a_meso, 4, 60, 2, sqrt_rule=True)
    assert ks.tolist() == orc.fine_counts_sqrt(n_i).tolist() and ks[2] == 0 and len(C) == ks.sum()
    off = np.concatenate([[0], np.cumsum(ks)])
    np.testing.assert_array_equal(np.searchsorted(off, a, side="right") - 1, a_meso)
    C2, a2, ks2, J2 = orc.fit_fine(P, a_meso, 4, int(ks.sum()), 2, sqrt_rule=True)
    np.testing.assert_array_equal(C, C2)
    np.testing.assert_array_equal(a, a2)
    with pytest.raises(ValueError):
        orc.fit_fine(P, a_meso, 4, int(ks.sum()) - 1, 2, sqrt_rule=True)
    init = np.random.default_rng(85).choice(500, 4, replace=False)
    Ch, ah, Jh, info = orc.fit_hier(P, 64, 2, 2, 1, init, k_meso=4, sqrt_rule=True)
    assert len(Ch) == info["k_fine"].sum() and info["k_fine"].tolist() == orc.fine_counts_sqrt(
        np.bincount(info["a_meso"], minlength=info["k_meso"])).tolist()
    a_exp, d = _nearest(X, Ch, list(range(len(Ch))))
    np.testing.assert_array_equal(ah, a_exp)


@settings(max_examples=200, deadline=None)
@given(n=st.lists(st.integers(0, 40), min_size=1, max_size=12), seed=st.integers(0, 10 ** 6))
def test_fine_counts_properties(orc, n, seed):
    m, N = sum(v > 0 for v in n), sum(n)
    if m == 0:
        return
    k = m + seed % (N - m + 1)
    ks = orc.fine_counts(n, k)
    assert ks.sum() == k
    for v, kv in zip(n, ks):
        assert (kv > 0) == (v > 0) and kv <= v
        if v > 0 and N > m:  # within one of the exact proportional share
            assert abs(kv - 1 - (k - m) * (v - 1) / (N - m)) < 1
    # order-independence of the shares up to the tie rule: a larger meso-cluster never gets fewer
    for i in range(len(n)):
        for j in range(len(n)):
            if n[i] > n[j]:
                assert ks[i] >= ks[j]


def _blob_rows(n, d, seed, comps=6):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((comps, d)) * 3
    return (mu[rng.integers(0, comps, n)] + rng.standard_normal((n, d))).astype(np.float32)


@pytest.mark.parametrize("fmt", ["f32", "sq8"])
def test_fine_with_one_meso_cluster_is_plain_lloyd(orc, fmt):
    """All points in one meso-cluster: the fine phase is Lloyd with k centroids started
    from the rows floor(j n / k)."""
    X = _blob_rows(300, 16, 61)
    P = {"fmt": "f32", "X": X} if fmt == "f32" else {"fmt": "sq8", "codes": orc.sq8_encode(X, *orc.sq8_fit(X))}
    k, T = 13, 3
    C, a, ks, J = orc.fit_fine(P, np.zeros(300, np.int32), 1, k, T)
    idx = np.array([j * 300 // k for j in range(k)])
    C2, a2, J2 = orc.fit(P, k, T, idx)
    assert ks.tolist() == [k]
    np.testing.assert_array_equal(C, C2)
    np.testing.assert_array_equal(a, a2)
    assert list(J) == J2


def _nearest(X, C, cand):
    D = ((X[:, None, :].astype(np.float64) - C[None, cand, :].astype(np.float64)) ** 2).sum(-1)
    return np.asarray(cand)[D.argmin(1)], D.min(1)


def test_fine_first_update_brute_force(orc):
    """One fine iteration (KEEP) worked out with explicit numpy: each meso-cluster's
    members (ascending index) start from the rows at positions floor(j n_i / k_i),
    are assigned to the nearest centroid of their own meso-cluster, the centroids
    become member means (global ids offset by the counts before), and the final
    assignment is again the nearest within the meso-cluster."""
    X = _blob_rows(240, 8, 67)
    rng = np.random.default_rng(68)
    a_meso = rng.integers(0, 4, 240).astype(np.int32)
    a_meso[a_meso == 3] = 2  # meso-cluster 3 is empty
    k = 17
    C, a, ks, J = orc.fit_fine({"fmt": "f32", "X": X}, a_meso, 4, k, 1, orc.EMPTY_KEEP)
    n_i = np.bincount(a_meso, minlength=4)
    assert ks.tolist() == orc.fine_counts(n_i, k).tolist() and ks[3] == 0
    off = np.concatenate([[0], np.cumsum(ks)])
    C_exp = np.zeros((k, 8))
    a_exp = np.zeros(240, np.int64)
    J_exp = 0.0
    for i in range(3):
        rows = np.nonzero(a_meso == i)[0]
        seg = list(range(off[i], off[i + 1]))
        C0 = np.zeros((k, 8), np.float32)
        C0[seg] = X[rows[(np.arange(ks[i]) * len(rows)) // ks[i]]]
        a0, _ = _nearest(X[rows], C0, seg)
        for j in seg:
            C_exp[j] = X[rows[a0 == j]].astype(np.float64).mean(0) if (a0 == j).any() else C0[j]
        a1, d1 = _nearest(X[rows], C_exp.astype(np.float32), seg)
        a_exp[rows] = a1
        J_exp += d1.sum()
    np.testing.assert_allclose(C, C_exp, rtol=1e-6, atol=1e-6)
    np.testing.assert_array_equal(a, a_exp)
    assert abs(J[-1] - J_exp) <= 1e-9 * J_exp


def test_hier_refine_ends_at_the_global_nearest(orc):
    """With refinement the returned assignment is the nearest of all k centroids and
    J its in-space objective; without it every point stays in its meso-cluster's
    segment of centroids (on unclustered data, where the two differ)."""
    X = np.random.default_rng(71).standard_normal((400, 8)).astype(np.float32)
    P = {"fmt": "f32", "X": X}
    init = np.random.default_rng(72).choice(400, 4, replace=False)
    C, a, J, info = orc.fit_hier(P, 16, 3, 2, 1, init)
    a_exp, d = _nearest(X, C, list(range(16)))
    np.testing.assert_array_equal(a, a_exp)
    assert abs(J - d.sum()) <= 1e-9 * d.sum()
    C0, a0, J0, info0 = orc.fit_hier(P, 16, 3, 2, 0, init)
    assert info0["k_meso"] == 4 and info0["k_fine"].sum() == 16
    off = np.concatenate([[0], np.cumsum(info0["k_fine"])])
    seg_of = np.searchsorted(off, a0, side="right") - 1
    np.testing.assert_array_equal(seg_of, info0["a_meso"])
    assert (_nearest(X, C0, list(range(16)))[0] != a0).any()


def test_fine_split_donor_stays_in_its_meso_cluster(orc):
    """Meso-cluster 0: six identical rows and three fine centroids that start equal, so
    two fine clusters come out empty; meso-cluster 1 holds a 20-member cluster.  The
    split must take its donor inside meso-cluster 0 (the largest cluster overall is
    in meso-cluster 1), so all three centroids of meso-cluster 0 stay at the row."""
    rng = np.random.default_rng(73)
    v0 = np.array([1.0, 2.0, 3.0, 4.0], np.float32)
    w = np.array([-5.0, 1.0, 0.0, 2.0], np.float32)
    X = np.concatenate([np.repeat(v0[None], 6, 0), np.repeat(w[None], 20, 0),
                        (w + rng.standard_normal((10, 4)) * 0.5).astype(np.float32)])
    a_meso = np.array([0] * 6 + [1] * 30, np.int32)
    C, a, ks, J = orc.fit_fine({"fmt": "f32", "X": X}, a_meso, 2, 16, 1, orc.EMPTY_SPLIT)
    assert ks.tolist() == [3, 13]
    assert np.all(np.abs(C[:3] - v0) <= 2.0 ** -8 * np.abs(v0))
    assert set(a[:6].tolist()) <= {0, 1, 2}


def test_hier_one_fine_cluster_per_meso_cluster(orc):
    """k = k_meso with every meso-cluster non-empty: each fine centroid is the mean of
    its meso-cluster's members and the partition is the meso partition."""
    X = _blob_rows(300, 8, 79)
    init = np.random.default_rng(80).choice(300, 5, replace=False)
    C, a, J, info = orc.fit_hier({"fmt": "f32", "X": X}, 5, 4, 2, 0, init, k_meso=5)
    am = info["a_meso"]
    assert info["k_fine"].tolist() == [1] * 5
    np.testing.assert_array_equal(a, am)
    for j in range(5):
        np.testing.assert_allclose(C[j], X[am == j].astype(np.float64).mean(0), rtol=1e-6, atol=1e-6)


# --------------------------------------------------------------------------
# Dimension pruning inside STEP 2 (Sec. 3.1 SuperKMeans, ADSampling test)

def test_prune_hand_example(orc):
    g = load_golden("prune_adsampling.json")
    d, D0, step, eps0 = g["d"], g["d_front"], g["step"], g["eps0"]
    for D, lim in g["thresholds_tau8"].items():
        assert abs(8.0 * orc.prune_factor(int(D), d, eps0) - lim) <= 1e-12 * lim
    for fmt in ("f32", "sq8"):
        e = g[fmt]
        if fmt == "f32":
            P = {"fmt": "f32", "X": np.array(e["points"], np.float32)}
            C = np.array(e["centroids"], np.float32)
        else:
            P = {"fmt": "sq8", "codes": np.array(e["points"], np.uint8)}
            C = np.array(e["centroids"], np.uint8)
        a, dist, cnt = orc.assign_pruned(P, C, np.array(e["prev"], np.int32), eps0, D0, step)
        assert a.tolist() == e["assign"], fmt
        assert dist.tolist() == e["dist"], fmt
        assert cnt.tolist() == e["counters"], fmt
    a_exact, _ = orc.assign_f32(np.array(g["f32"]["points"], np.float32), np.array(g["f32"]["centroids"], np.float32))
    assert a_exact.tolist() == g["f32"]["exact_nearest"]


def _prune_numpy(Xd, Cd, prev, eps0, D0, step, sq8):
    """The pruned assignment evaluated with numpy: prefix sums of the squared
    differences (cumsum), the survivor matrix over all checkpoints, then the argmin of
    the full distance over the survivors and the previous centroid."""
    n, d = Xd.shape
    k = len(Cd)
    sq = (Xd[:, None, :] - Cd[None, :, :]) ** 2
    pre = np.cumsum(sq, axis=2)
    full = pre[:, :, -1]
    tau = full[np.arange(n), prev]
    alive = np.ones((n, k), bool)
    alive[np.arange(n), prev] = False
    cps = list(range(D0, d, step))
    tested = passed = 0
    for m, D in enumerate(cps):
        g = (1.0 + eps0 / np.sqrt(D)) ** 2 * D / d
        if sq8:
            keep = pre[:, :, D - 1].astype(np.float32) <= (tau.astype(np.float32)[:, None] * np.float32(g))
        else:
            keep = pre[:, :, D - 1] <= tau[:, None] * g
        if m == 0:
            tested = int(alive.sum())
            passed = int((alive & keep).sum())
        alive &= keep
    cand = alive.copy()
    cand[np.arange(n), prev] = True
    score = np.where(cand, full, np.inf)
    a = score.argmin(1)
    return a, score[np.arange(n), a], [tested, passed, int(alive.sum())]


@settings(max_examples=40, deadline=None)
@given(n=st.integers(1, 30), d=st.sampled_from([8, 16, 40, 64]), k=st.integers(1, 9),
       seed=st.integers(0, 2**31 - 1), sq8=st.booleans())
def test_prune_brute_force(orc, n, d, k, seed, sq8):
    rng = np.random.default_rng(seed)
    D0, step = max(1, d // 8), max(1, d // 4)
    prev = rng.integers(0, k, n).astype(np.int32)
    if sq8:
        X = rng.integers(0, 256, (n, d)).astype(np.uint8)
        C = rng.integers(0, 256, (k, d)).astype(np.uint8)
        C[k // 2] = C[0]  # equal centroids: ties to the smaller index
        P = {"fmt": "sq8", "codes": X}
        Xd, Cd = X.astype(np.int64), C.astype(np.int64)
    else:
        X = rng.standard_normal((n, d)).astype(np.float32)
        C = (X[rng.integers(0, n, k)] + 0.7 * rng.standard_normal((k, d))).astype(np.float32)
        P = {"fmt": "f32", "X": X}
        Xd, Cd = X.astype(np.float64), C.astype(np.float64)
    eps0 = float(rng.uniform(0.2, 3.0))
    a, dist, cnt = orc.assign_pruned(P, C, prev, eps0, D0, step)
    a2, dist2, cnt2 = _prune_numpy(Xd, Cd, prev, eps0, D0, step, sq8)
    np.testing.assert_array_equal(a, a2)
    np.testing.assert_array_equal(dist, dist2.astype(np.float64))
    assert cnt.tolist() == cnt2
    # never worse than the previous centroid
    assert (dist <= ((Xd - Cd[prev]) ** 2).sum(1) + 1e-9).all()


@pytest.mark.parametrize("fmt", ["f32", "sq8"])
def test_prune_with_huge_eps_is_exact_assignment(orc, fmt):
    rng = np.random.default_rng(81)
    X = rng.standard_normal((300, 64)).astype(np.float32)
    C = X[rng.choice(300, 17, replace=False)].copy()
    C[5] = C[2]
    if fmt == "f32":
        P = {"fmt": "f32", "X": X}
    else:
        lo, hi = orc.sq8_fit(X)
        P = {"fmt": "sq8", "codes": orc.sq8_encode(X, lo, hi)}
        C = orc.sq8_encode(C, lo, hi)
    prev = rng.integers(0, 17, 300).astype(np.int32)
    a, dist, cnt = orc.assign_pruned(P, C, prev, 1e12)
    a_ex, dist_ex = orc.assign(P, C)
    np.testing.assert_array_equal(a, a_ex)
    np.testing.assert_allclose(dist, dist_ex, rtol=1e-12)
    assert cnt[0] == cnt[1] == cnt[2] == 300 * 16


def test_prune_on_rotated_mixture_keeps_the_partition(orc):
    """On randomly rotated, unit-normalised clustered data the test drops most
    candidates at d' and the pruned Lloyd ends at (nearly) the exact partition."""
    import synth
    rng = np.random.default_rng(83)
    d, n, comps = 256, 3000, 24
    mu = rng.standard_normal((comps, d))
    X = mu[rng.integers(0, comps, n)] + 0.35 * rng.standard_normal((n, d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    X = (X @ synth.random_rotation(d, 4)).astype(np.float32)
    P = {"fmt": "f32", "X": X}
    idx = rng.choice(n, comps, replace=False)
    C, a, J, cnt = orc.fit_pruned(P, comps, 6, idx)
    C2, a2, J2 = orc.fit(P, comps, 6, idx)
    assert (a == a2).mean() >= 0.995
    assert cnt[1] <= 0.2 * cnt[0]
    assert cnt[2] <= cnt[1]
    assert abs(J[-1] - J2[-1]) <= 1e-3 * J2[-1]
