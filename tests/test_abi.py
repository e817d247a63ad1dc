"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/kmq.h, and rejects bad arguments on the host with the
documented status before touching the device.  No compute call is made here.
"""
import ctypes as ct
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kmq.h")
LIB = os.path.join(ROOT, "paper_2608_14648_amd", "libkmq.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libkmq.so not built (run __graft_entry__.build())")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:km_status|const char \*)\s*(\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("quantize", "pca_fit_cov", "pca_project", "kmeans_assign", "kmeans_update", "kmeans_fit",
              "kmeans_cost", "km_last_error", "km_release"):
        assert n in names


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    L = ct.CDLL(LIB)
    for n in declared_functions():
        assert hasattr(L, n)


def test_header_compiles_as_c():
    src = '#include "kmq.h"\nint main(void){ km_points p = {0}; (void)p; return (int)sizeof(km_points); }\n'
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER), "-x", "c", "-", "-o",
                        "/dev/null"], input=src, text=True, capture_output=True)
    assert r.returncode == 0, r.stderr


@pytest.fixture(scope="module")
def kmq():
    from paper_2608_14648_amd import _kmq
    return _kmq


def _pts(kmq, **kw):
    base = dict(fmt=kmq.KM_F32, d=128, n=100, data=0x1000, ld=128, alpha=None, center=None, front=None, d_front=0,
                reserved=0, raw=None, raw_ld=0, vparams=None)
    base.update(kw)
    return kmq.KmPoints(base["fmt"], base["d"], base["n"], base["data"], base["ld"], base["alpha"], base["center"],
                        base["front"], base["d_front"], base["reserved"], base["raw"], base["raw_ld"],
                        base["vparams"])


FAKE = ct.c_void_p(0x10000)  # never dereferenced: validation fails first


@pytest.mark.parametrize("kw,status,msg", [
    (dict(fmt=7), -2, "format"),
    (dict(n=0), -1, "n ="),
    (dict(d=0), -1, "d ="),
    (dict(d=126, ld=128), -1, "d % 4"),
    (dict(ld=64), -1, "ld"),
    (dict(data=None), -1, "NULL"),
    (dict(data=0x1004), -1, "aligned"),
    (dict(reserved=1), -1, "reserved"),
    (dict(fmt=2, d=40, ld=48), -1, "d % 16"),
    (dict(fmt=1, d=12, ld=16), -1, "d % 8"),
    (dict(fmt=1, d=64, ld=68), -1, "ld % 8"),
    (dict(fmt=1, d=64, ld=64, d_front=32), -1, "d_front"),
    (dict(fmt=3, d=100, alpha=0x2000, center=0x3000), -1, "d % 32"),
    (dict(fmt=3, d=128, alpha=None, center=0x3000), -1, "alpha"),
    (dict(fmt=3, d=128, alpha=0x2000, center=None), -1, "center"),
    (dict(fmt=4, d=128, alpha=0x2000, center=0x3000, front=0x4000, d_front=0), -1, "d_front"),
    (dict(fmt=4, d=128, alpha=0x2000, center=0x3000, front=0x4000, d_front=48), -1, "d_front"),
    (dict(fmt=4, d=128, alpha=0x2000, center=0x3000, front=None, d_front=64), -1, "front"),
    (dict(fmt=0, d_front=32), -1, "d_front"),
    (dict(fmt=5, d=128, alpha=0x2000, center=0x3000), -1, "center must be NULL"),
    (dict(fmt=5, d=100, alpha=0x2000), -1, "d % 32"),
    (dict(fmt=5, d=128, alpha=None), -1, "alpha"),
    (dict(fmt=2, d=128, ld=128, raw=0x5000, raw_ld=128), -1, "not allowed for SQ8"),
    (dict(fmt=5, d=128, alpha=0x2000, raw=0x5004, raw_ld=128), -1, "raw rows"),
    (dict(fmt=5, d=128, alpha=0x2000, raw=0x5000, raw_ld=64), -1, "raw rows"),
    (dict(fmt=6, d=128, ld=64), -1, "vparams"),
    (dict(fmt=0, vparams=0x6000), -1, "vparams"),
    (dict(fmt=6, d=112, ld=64, vparams=0x6000), -1, "d % 32"),
    (dict(fmt=6, d=128, ld=48, vparams=0x6000), -1, "ld >= d/2"),
    (dict(fmt=6, d=128, ld=72, vparams=0x6000), -1, "ld % 16"),
    (dict(fmt=6, d=128, ld=64, vparams=0x6000, center=0x3000), -1, "no center"),
    (dict(fmt=6, d=128, ld=64, vparams=0x6004), -1, "vparams must be 16-byte"),
    (dict(fmt=0, d=128, ld=1 << 21), -1, "too large"),
    (dict(fmt=1, d=128, ld=1 << 22), -1, "too large"),
    (dict(fmt=2, d=128, ld=1 << 23), -1, "too large"),
    (dict(fmt=6, d=128, ld=1 << 23, vparams=0x6000), -1, "too large"),
])
def test_points_validation(kmq, kw, status, msg):
    L = kmq.lib()
    P = _pts(kmq, **kw)
    st = L.kmeans_assign(ct.byref(P), FAKE, 4, FAKE, None, None, None)
    assert st == status
    assert msg in L.km_last_error().decode()
    st = L.kmeans_update(ct.byref(P), FAKE, 4, FAKE, None, 0, None)
    assert st == status


def test_entry_point_argument_checks(kmq):
    L = kmq.lib()
    P = _pts(kmq)
    assert L.kmeans_assign(None, FAKE, 4, FAKE, None, None, None) == -1
    assert L.kmeans_assign(ct.byref(P), FAKE, 0, FAKE, None, None, None) == -1
    assert L.kmeans_assign(ct.byref(P), None, 4, FAKE, None, None, None) == -1
    assert L.kmeans_assign(ct.byref(P), ct.c_void_p(0x10004), 4, FAKE, None, None, None) == -1
    assert L.kmeans_assign(ct.byref(P), FAKE, 4, None, None, None, None) == -1
    assert L.kmeans_update(ct.byref(P), FAKE, 4, FAKE, None, 5, None) == -1
    assert "policy" in L.km_last_error().decode()
    # fit: k > n, negative iters, bad init indices (host memory)
    assert L.kmeans_fit(ct.byref(P), 101, 3, None, FAKE, FAKE, None, 0, None, None) == -1
    assert L.kmeans_fit(ct.byref(P), 4, -1, None, FAKE, FAKE, None, 0, None, None) == -1
    dup = (ct.c_int64 * 4)(0, 5, 5, 7)
    assert L.kmeans_fit(ct.byref(P), 4, 3, dup, FAKE, FAKE, None, 0, None, None) == -1
    assert "duplicates" in L.km_last_error().decode()
    oob = (ct.c_int64 * 4)(0, 5, 100, 7)
    assert L.kmeans_fit(ct.byref(P), 4, 3, oob, FAKE, FAKE, None, 0, None, None) == -1
    neg = (ct.c_int64 * 4)(0, -1, 2, 7)
    assert L.kmeans_fit(ct.byref(P), 4, 3, neg, FAKE, FAKE, None, 0, None, None) == -1


def test_rabitq_encode_argument_checks(kmq):
    L = kmq.lib()
    ok = (FAKE, 10, 64, 64, FAKE, FAKE, FAKE, FAKE, None, 1, None)
    bad = [
        ((None,) + ok[1:], "NULL"),
        (ok[:2] + (48, 48) + ok[4:], "d % 32"),
        (ok[:3] + (60,) + ok[4:], "ldx"),
        (ok[:4] + (None,) + ok[5:], "NULL"),
        ((ct.c_void_p(0x10004),) + ok[1:], "aligned"),
        (ok[:9] + (4,) + ok[10:], "flags"),
        (ok[:8] + (ct.c_void_p(0x10008),) + ok[9:], "aligned"),
        (ok[:1] + (0,) + ok[2:], "n ="),
    ]
    for args, msg in bad:
        assert L.rabitq_encode(*args) == -1, msg
        assert msg in L.km_last_error().decode(), (msg, L.km_last_error())


def test_quantize_and_pca_argument_checks(kmq):
    L = kmq.lib()
    # unsupported format, bad d, misaligned, unknown flags
    assert L.quantize(FAKE, 10, 64, 64, 0, FAKE, FAKE, FAKE, 0, None, 1, None) == -2
    assert L.quantize(FAKE, 10, 40, 40, 2, FAKE, FAKE, None, 0, None, 1, None) == -1
    assert L.quantize(FAKE, 10, 64, 64, 3, FAKE, FAKE, None, 0, None, 1, None) == -1  # alpha NULL
    assert L.quantize(FAKE, 10, 64, 64, 3, FAKE, FAKE, FAKE, 16, None, 1, None) == -1  # d_front % 32
    assert L.quantize(FAKE, 10, 64, 64, 3, FAKE, FAKE, FAKE, 64, None, 1, None) == -1  # d_front == d
    assert L.quantize(FAKE, 10, 64, 64, 2, FAKE, FAKE, None, 0, None, 4, None) == -1  # flags
    assert L.quantize(ct.c_void_p(0x10002), 10, 64, 64, 2, FAKE, FAKE, None, 0, None, 1, None) == -1
    assert L.quantize(FAKE, 0, 64, 64, 2, FAKE, FAKE, None, 0, None, 1, None) == -1
    assert L.quantize(FAKE, 10, 64, 64, 3, FAKE, ct.c_void_p(0x10008), FAKE, 0, None, 1, None) == -1  # params
    assert L.quantize(FAKE, 10, 12, 12, 1, FAKE, None, None, 0, None, 0, None) == -1  # bf16: d % 8
    assert "d % 8" in L.km_last_error().decode()
    assert L.quantize(FAKE, 10, 64, 64, 1, FAKE, None, None, 32, None, 0, None) == -1  # bf16: no front
    assert L.quantize(FAKE, 10, 64, 64, 1, None, None, None, 0, None, 0, None) == -1  # bf16: codes NULL
    assert L.quantize(FAKE, 10, 48, 48, 6, FAKE, FAKE, None, 0, None, 0, None) == -1  # lvq4: d % 32
    assert "d % 32" in L.km_last_error().decode()
    assert L.quantize(FAKE, 10, 64, 64, 6, FAKE, None, None, 0, None, 0, None) == -1  # lvq4: params NULL
    assert L.quantize(FAKE, 10, 64, 64, 6, FAKE, ct.c_void_p(0x10008), None, 0, None, 0, None) == -1
    assert L.pca_fit_cov(FAKE, 10, 30, FAKE, FAKE, None) == -1
    assert L.pca_fit_cov(None, 10, 32, FAKE, FAKE, None) == -1
    assert L.pca_project(FAKE, 10, 32, FAKE, FAKE, 0, FAKE, None) == -1
    assert L.pca_project(FAKE, 10, 32, FAKE, None, 8, FAKE, None) == -1
    assert L.kmeans_cost(FAKE, 10, 32, 16, FAKE, 4, FAKE, FAKE, None) == -1
    assert L.kmeans_cost(FAKE, 10, 32, 32, FAKE, 0, FAKE, FAKE, None) == -1


def test_last_error_is_per_thread(kmq):
    import threading
    L = kmq.lib()
    P = _pts(kmq, n=0)
    assert L.kmeans_assign(ct.byref(P), FAKE, 4, FAKE, None, None, None) == -1
    seen = {}

    def other():
        seen["msg"] = L.km_last_error().decode()

    th = threading.Thread(target=other)
    th.start()
    th.join()
    assert seen["msg"] == ""
    assert "n =" in L.km_last_error().decode()


def test_binding_rejects_host_tensors(kmq):
    import torch
    with pytest.raises(ValueError):
        kmq.points_f32(torch.zeros(4, 8))


def test_hierarchical_argument_checks(kmq):
    """kmeans_fine / kmeans_fit_hier reject bad arguments on the host, before any HIP call."""
    L = kmq.lib()
    P = _pts(kmq)
    ok = (ct.byref(P), FAKE, 4, 10, 2, 0, FAKE, FAKE, None, None, 0, None)
    bad = [
        (ok[:1] + (None,) + ok[2:], "NULL"),
        (ok[:2] + (0,) + ok[3:], "k_meso"),
        (ok[:4] + (-1,) + ok[5:], "iters"),
        (ok[:5] + (4,) + ok[6:], "flags"),  # 1 and 2 (KM_FINE_C_GIVEN, KM_FINE_SQRT) are known
        (ok[:10] + (5,) + ok[11:], "policy"),
        (ok[:6] + (None,) + ok[7:], "centroids"),
        (ok[:7] + (None,) + ok[8:], "NULL"),
    ]
    for args, msg in bad:
        assert L.kmeans_fine(*args) == -1, msg
        assert msg in L.km_last_error().decode(), (msg, L.km_last_error())
    init = (ct.c_int64 * 3)(0, 5, 9)
    hp = kmq.KmHierParams(3, 2, 2, 0)
    base = [ct.byref(P), 10, ct.byref(hp), init, FAKE, FAKE, None, None, None, 0, None, None, None]
    for i, v, msg in [(2, None, "NULL"), (3, None, "NULL"), (1, 101, "exceeds"), (9, 7, "policy")]:
        args = list(base)
        args[i] = v
        assert L.kmeans_fit_hier(*args) == -1, msg
        assert msg in L.km_last_error().decode(), (msg, L.km_last_error())
    for params, msg in [((11, 2, 2, 0), "k_meso"), ((3, -1, 2, 0), "iteration"), ((3, 2, 2, -2), "iteration"),
                        ((3, 2, 2, 0, 4), "flags")]:
        hp2 = kmq.KmHierParams(*params)
        args = list(base)
        args[2] = ct.byref(hp2)
        assert L.kmeans_fit_hier(*args) == -1, msg
        assert msg in L.km_last_error().decode(), (msg, L.km_last_error())
    dup = (ct.c_int64 * 3)(0, 5, 5)
    args = list(base)
    args[3] = dup
    assert L.kmeans_fit_hier(*args) == -1
    assert "duplicates" in L.km_last_error().decode()
    # k_meso = 0 means round(sqrt(k)): 3 for k = 10, so three initial rows are needed and checked
    hp0 = kmq.KmHierParams(0, 1, 1, 0)
    oob = (ct.c_int64 * 3)(0, 5, 100)
    args = list(base)
    args[2], args[3] = ct.byref(hp0), oob
    assert L.kmeans_fit_hier(*args) == -1
    assert "outside" in L.km_last_error().decode()


def test_pruned_argument_checks(kmq):
    """kmeans_assign_pruned / kmeans_fit_pruned reject bad arguments on the host."""
    L = kmq.lib()
    P = _pts(kmq, d=768, ld=768)
    pr = kmq.KmPrune(2.1, 0, 0)
    ok = [ct.byref(P), FAKE, 4, FAKE, FAKE, None, None, ct.byref(pr), None, None]
    cases = [(3, None, -1, "NULL"), (7, None, -1, "NULL")]
    for i, v, code, msg in cases:
        args = list(ok)
        args[i] = v
        assert L.kmeans_assign_pruned(*args) == code, msg
        assert msg in L.km_last_error().decode()
    for params, code, msg in [((0.0, 0, 0), -1, "eps0"), ((2.1, 0, 1), -1, "reserved"), ((2.1, 6, 0), -1, "d_front"),
                              ((2.1, 36, 0), -1, "d_front"),
                              ((2.1, 512, 0), -2, "d_front"), ((2.1, 800, 0), -1, "d_front")]:
        pr2 = kmq.KmPrune(*params)
        args = list(ok)
        args[7] = ct.byref(pr2)
        assert L.kmeans_assign_pruned(*args) == code, msg
        assert msg in L.km_last_error().decode(), (msg, L.km_last_error())
    # formats other than fp32 / SQ8, and rows too long after d'
    P1 = _pts(kmq, fmt=3, d=128, alpha=0x2000, center=0x3000)
    args = list(ok)
    args[0] = ct.byref(P1)
    assert L.kmeans_assign_pruned(*args) == -2
    Pw = _pts(kmq, d=4096, ld=4096)
    args = list(ok)
    args[0] = ct.byref(Pw)
    assert L.kmeans_assign_pruned(*args) == -2
    # fp32 rows must hold whole groups of 8 dims
    P8 = _pts(kmq, d=132, ld=132)
    args = list(ok)
    args[0] = ct.byref(P8)
    assert L.kmeans_assign_pruned(*args) == -2
    # SQ8: d' must be a multiple of 16
    Ps = _pts(kmq, fmt=2, d=256, ld=256)
    pr3 = kmq.KmPrune(2.1, 40, 0)
    args = list(ok)
    args[0], args[7] = ct.byref(Ps), ct.byref(pr3)
    assert L.kmeans_assign_pruned(*args) == -1
    # the fit: k > n, negative iterations, policy
    fit_ok = [ct.byref(P), 4, 3, None, FAKE, FAKE, None, 0, ct.byref(pr), None, None, None]
    for i, v, msg in [(1, 101, "exceeds"), (2, -1, "iters"), (7, 4, "policy"), (8, None, "NULL")]:
        args = list(fit_ok)
        args[i] = v
        assert L.kmeans_fit_pruned(*args) == -1, msg
        assert msg in L.km_last_error().decode(), (msg, L.km_last_error())


def test_allocation_failure_is_reported(kmq):
    # KMQ_FAIL_ALLOC=1 refuses every scratch allocation before any HIP call; a valid
    # call then returns KM_ENOMEM with nothing launched (checked in a child process,
    # since the library reads the variable on every allocation)
    code = (
        "import ctypes as ct, sys\n"
        f"sys.path.insert(0, {ROOT!r})\n"
        "from paper_2608_14648_amd import _kmq as k\n"
        "L = k.lib()\n"
        "P = k.KmPoints(k.KM_F32, 128, 100, ct.c_void_p(0x10000), 128, None, None, None, 0, 0, None, 0, None)\n"
        "F = ct.c_void_p(0x10000)\n"
        "st = [L.kmeans_assign(ct.byref(P), F, 4, F, None, None, None),\n"
        "      L.kmeans_update(ct.byref(P), F, 4, F, None, 0, None),\n"
        "      L.quantize(F, 100, 128, 128, k.KM_SQ8, F, F, None, 0, None, 1, None),\n"
        "      L.pca_fit_cov(F, 100, 128, F, F, None)]\n"
        "print(st, L.km_last_error().decode())\n"
    )
    env = dict(os.environ, KMQ_FAIL_ALLOC="1")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("[-3, -3, -3, -3]"), r.stdout
    assert "KMQ_FAIL_ALLOC" in r.stdout
    # the noalloc entry point never allocates, so the variable cannot make it fail
    # that way: it still validates its arguments on the host
    L = kmq.lib()
    assert L.kmeans_assign_noalloc(None, FAKE, 4, FAKE, None, None, None) == -1
