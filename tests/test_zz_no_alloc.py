"""kmeans_assign_noalloc: the assignment entry point for callers that cannot
allocate, with its scratch in the library's static device array.  Checked
through the C ABI against kmeans_assign on the same inputs, on two calls in a
row (the second with fewer points, so the static array still holds the first
call's contents), in fp32, SQ8, bfloat16, LVQ4 and 1-bit formats, with the objective.
"""
import numpy as np
import pytest

import synth
from gpu_util import host, say, to_dev, torch_cuda

pytestmark = pytest.mark.gpu

K = 1000
N_FIRST, N_SECOND = 40_000, 25_000  # both large enough for the centroid-tile groups and their keys


def _inputs(torch, km, fmt, n):
    spec = synth.MixtureSpec(n, 256, 64, 0.15, True, seed=5)
    X = to_dev(synth.make_points(spec), torch)
    idx = to_dev(synth.init_indices(n, K, seed=6), torch)
    if fmt == "f32":
        return km.points_f32(X), X[idx].contiguous()
    if fmt == "sq8":
        codes, _ = km.quantize_sq8(X)
        return km.points_sq8(codes), codes[idx].contiguous()
    if fmt == "bf16":
        return km.points_bf16(km.quantize_bf16(X)), X[idx].contiguous()
    if fmt == "lvq4":
        codes, par = km.quantize_lvq4(X)
        return km.points_lvq4(codes, par, spec.d), X[idx].contiguous()
    bits, m, alpha, _ = km.quantize_sign1(X)
    return km.points_sign1(bits, alpha, m, spec.d), X[idx].contiguous()


@pytest.mark.parametrize("fmt", ["f32", "sq8", "bf16", "lvq4", "sign1"])
def test_noalloc_matches_kmeans_assign(fmt):
    torch = torch_cuda()
    import paper_2608_14648_amd as km
    for n in (N_FIRST, N_SECOND):
        say(f"noalloc {fmt}: n={n} k={K}")
        P, C = _inputs(torch, km, fmt, n)
        a_ref, s_ref, o_ref = km.kmeans_assign(P, C, score=True, objective=True)
        a = torch.full((n,), -7, dtype=torch.int32, device="cuda")
        s = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
        o = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
        km.kmeans_assign_noalloc(P, C, a, s, o)
        torch.cuda.synchronize()
        # same kernels on the same inputs: identical assignments, scores and objective
        np.testing.assert_array_equal(host(a), host(a_ref))
        np.testing.assert_array_equal(host(s), host(s_ref))
        assert host(o)[0] == host(o_ref)[0]
        # and without score or objective
        a2 = torch.full((n,), -7, dtype=torch.int32, device="cuda")
        km.kmeans_assign_noalloc(P, C, a2)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(a2), host(a_ref))


def test_noalloc_rejects_what_the_static_array_cannot_hold():
    torch = torch_cuda()
    import paper_2608_14648_amd as km
    n, d = 5_000_000, 16  # 16 bytes of scratch per point with the objective: more than 64 MiB
    say(f"noalloc oversize: n={n} d={d} k={K}")
    X = torch.zeros((n, d), dtype=torch.float32, device="cuda")
    C = torch.zeros((K, d), dtype=torch.float32, device="cuda")
    a = torch.empty(n, dtype=torch.int32, device="cuda")
    o = torch.empty(1, dtype=torch.float64, device="cuda")
    with pytest.raises(km.KmqError) as e:
        km.kmeans_assign_noalloc(km.points_f32(X), C, a, None, o)
    assert e.value.status == -1 and "static buffer" in str(e.value)
