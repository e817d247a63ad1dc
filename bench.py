#!/usr/bin/env python3
"""Benchmark of the hot path on one MI355X: Lloyd k-means on compressed vectors.

One JSON line per run, for one workload and one point format.  The default
workload (`c4`) is the largest single-GPU configuration: 10,000,000 x 1024
unit-normalised Gaussian mixture of 4,096 components with decaying per-dim
variance (lambda_i = i^-0.5), PCA projection to 256 dims, then k = 4,096 and 10
Lloyd iterations.  One step =
  pca_fit_cov (mean, covariance) + host eigensolve of the 1024 x 1024 covariance
  + pca_project (10M x 1024 -> 10M x 256)
  + kmeans_fit (init gather, 10 x (assign, update), final assign, objectives)
  + full-precision partition cost of the final partition (raw-vector means).
Inputs are resident in HBM before the timed region; `value` is Lloyd iterations
per second over the whole step (iterations of the step / seconds per step).

Other workloads (`--workload NAME`; the old numbers still work):
  c1 (1)        20k x 128, k = 64, 10 iterations, fp32
  c2-f32 (2)    1M x 768, k = 1000, 20 iterations, fp32
  c2-sq8 (11)   the same data as per-dimension SQ8 codes (quantisation in the step)
  c3 (3)        1M x 1024, k = 1024, 20 iterations, 1-bit sign codes + alpha
  c4 (4)        the default (above)
  c5 (5)        the 10M x 1024 data as fp32 front 384 dims + 1-bit codes of the
                tail, k = 4096, 10 iterations (quantisation in the step)
  bf16 (6)      c2's data stored as bfloat16
  rabitq (7)    c3's data through random rotation, SQ4 centroid codes, raw last update
  lvq4 (8)      c2's data as LVQ4 codes
  hier-f32 (9), hier-sq8 (12)      hierarchical k-means on c4's data, k = 4 sqrt(N)
  pruned-f32 (10), pruned-sq8 (13) c2's data rotated, dimension pruning after pass 1

The line carries:
* `roofline`: the dominant kernel (the fused assignment kernel; the line names
  it), its algorithmic work per launch over its average launch time, measured
  from HIP events that the library records on its stream around each launch,
  against MI355X's peak for the arithmetic it issues.  `traffic` is the HBM
  bytes per launch from the committed rocprofv3 counter record of the same
  workload (FETCH_SIZE and WRITE_SIZE scaled by a copy kernel of known size),
  or null when there is none or the kernel's sources changed since.
* `update_hbm`: bytes the update step must move per iteration over its time.
* `cpu_baseline`: the plain CPU oracle timed on this host's cores on a bounded
  sample of the same workload, every stage once, scaled to the whole step.
* `quality` (after the timed region; --no-quality skips it): full-precision
  cost of the final partition (raw-vector member means), the cost with the
  centroids the method itself leaves (reconstructed from codes, or unprojected),
  cluster-size spread, and the ratio to fp32 Lloyd on the raw vectors from the
  same initial rows.

--copy-probe runs a 1 GiB fill and a 1 GiB negating copy before the workload:
kernels of known traffic against which FETCH_SIZE / WRITE_SIZE are scaled.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np
import scipy.linalg

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Lloyd iters/s + point×centroid distances/s; objective ratio vs fp32 oracle"
PEAK = {"fp32": 157.3, "bf16": 2500.0, "int8": 5000.0, "hbm_gbs": 8000.0}
PEAK_UNIT = {"fp32": "TFLOP/s", "bf16": "TFLOP/s", "int8": "TOP/s"}
ASSIGN_SOURCES = ("paper_2608_14648_amd/csrc/assign.hip", "paper_2608_14648_amd/csrc/common.hpp")
COPY_PROBE_FLOATS = 256 << 20  # 1 GiB of fp32


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def upload(spec, torch):
    """Generate the mixture chunk by chunk straight into a device tensor."""
    import synth
    X = torch.empty((spec.n, spec.d), dtype=torch.float32, device="cuda")

    def put(r0, blk):
        X[r0:r0 + blk.shape[0]].copy_(torch.from_numpy(blk), non_blocking=False)
    synth.for_each_chunk(spec, put)
    torch.cuda.synchronize()
    return X


class Timer:
    def __init__(self):
        self.stats = {}
        self.host_ms = {}

    def add(self, name, st):
        d = self.stats.setdefault(name, {"assign_ms": 0.0, "prep_ms": 0.0, "update_ms": 0.0, "other_ms": 0.0,
                                         "assign_passes": 0, "updates": 0})
        for key, v in st.as_dict().items():
            d[key] += v

    def host(self, name, ms):
        self.host_ms[name] = self.host_ms.get(name, 0.0) + ms


def stage_summary(s):
    return {"assign_ms_per_pass": s["assign_ms"] / max(1, s["assign_passes"]),
            "update_ms_per_iter": s["update_ms"] / max(1, s["updates"]),
            "prep_ms_per_pass": s["prep_ms"] / max(1, s["assign_passes"]),
            "other_ms_total": s["other_ms"]}


def source_hash(paths):
    h = hashlib.sha256()
    for rel in paths:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def counted_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` on `workload` from the committed counter
    record profiles/counters__<workload>.md (its JSON block), or None when the
    record is missing, holds no entry for the kernel, or was taken from other
    sources of the kernel than the ones here."""
    try:
        with open(os.path.join(ROOT, "profiles", f"counters__{workload}.md")) as f:
            text = f.read()
    except OSError:
        return None
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if m is None:
        return None
    rec = json.loads(m.group(1))
    if rec.get("workload") != workload:
        return None
    ent = rec.get("kernels", {}).get(kernel)
    if ent is None or ent.get("source_sha256") != source_hash(ent.get("sources", ASSIGN_SOURCES)):
        return None
    return ent.get("traffic_bytes_per_launch")


def copy_probe(torch):
    """Kernels of known traffic for counter calibration: a fill that writes
    1 GiB, then a negating copy that reads 1 GiB and writes 1 GiB."""
    src = torch.ones(COPY_PROBE_FLOATS, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst
    log(f"copy probe done ({COPY_PROBE_FLOATS * 4} bytes)")


def roofline(workload, stats, work_per_launch, peak, kernel, kernel_key):
    a_ms = stats["assign_ms"] / max(1, stats["assign_passes"])
    ach = work_per_launch / (a_ms * 1e-3) / 1e12
    return {"bound": "mfma", "kernel": kernel, "achieved": ach, "peak": PEAK[peak], "unit": PEAK_UNIT[peak],
            "frac": ach / PEAK[peak], "traffic": counted_traffic(workload, kernel_key),
            "avg_launch_ms": a_ms, "work_per_launch": work_per_launch,
            "work": "2 d multiply-adds' operations per (point, centroid) pair"}


def update_hbm(stats, bytes_per_update, what):
    u_ms = stats["update_ms"] / max(1, stats["updates"])
    gbs = bytes_per_update / (u_ms * 1e-3) / 1e9
    return {"bytes_per_update": bytes_per_update, "bytes": what, "ms_per_update": u_ms, "achieved_gbs": gbs,
            "peak_gbs": PEAK["hbm_gbs"], "frac": gbs / PEAK["hbm_gbs"]}


def partition_stats(km, X, a, mu):
    """Full-precision cost of a partition (raw-vector member means) and the spread
    of its cluster sizes."""
    _, cnt = km.kmeans_update(km.points_f32(X), a, mu, km.KM_EMPTY_KEEP, counts=True)
    cost = float(km.kmeans_cost(X, mu, a).item())
    c = cnt.cpu().numpy()
    return {"cost": cost, "cluster_size_std": float(c.std()), "empty_clusters": int((c == 0).sum())}


def quality_vs_f32(km, X, k, T, idx, mu, name, a, own_centroids=None):
    """Partition quality of `name` next to fp32 Lloyd on the raw vectors (same init, T).
    own_centroids: fp32 centroids in the original space that the method itself
    produces (decoded from its codes, or unprojected); their cost is reported too."""
    q = {name: partition_stats(km, X, a, mu)}
    if own_centroids is not None:
        q[name]["cost_own_centroids"] = float(km.kmeans_cost(X, own_centroids.contiguous(), a).item())
    log("quality: fp32 reference fit (outside the timed region)")
    _, a32, _ = km.kmeans_fit(km.points_f32(X), k, T, idx, objective=False)
    q["f32"] = partition_stats(km, X, a32, mu)
    q[f"objective_ratio_{name}_vs_f32"] = q[name]["cost"] / q["f32"]["cost"]
    if own_centroids is not None:
        q[f"objective_ratio_{name}_own_centroids_vs_f32"] = q[name]["cost_own_centroids"] / q["f32"]["cost"]
    return q


# ------------------------------------------------------------------ CPU oracle baseline

def _timed(fn):
    t0 = time.perf_counter()
    r = fn()
    return time.perf_counter() - t0, r


def oracle_baseline(run, N, T, budget_s, n_probe, n_cap, what, unit="Lloyd iters/s", per_step=None):
    """Time the oracle's stages on the first ns rows of the workload and scale each
    by N over the rows it ran on and by how often it runs in one step.  run(ns)
    returns a list of (stage, seconds, runs per step, rows the stage ran on, or
    None for a stage whose cost does not grow with N).  A probe at n_probe rows
    sizes ns so that the timed sample takes about budget_s."""
    import oracle as orc
    t_probe = sum(s for _, s, _, _ in run(n_probe))
    ns = int(min(n_cap, max(n_probe, n_probe * budget_s / max(t_probe, 1e-6))))
    stages = run(ns)
    per = {name: sec * reps * (N / rows if rows else 1.0) for name, sec, reps, rows in stages}
    step_s = sum(per.values())
    timed = sum(s for _, s, _, _ in stages)
    value = (per_step if per_step is not None else T) / step_s
    return {"value": value, "unit": unit, "cores": orc.num_threads(), "kind": "oracle",
            "sample": f"{what}: every stage of the step once on the first {ns} of the {N} points (timed {timed:.1f} s), "
                      f"each scaled by N over the rows it ran on and by its count per step; "
                      f"{step_s:.1f} s per step extrapolated",
            "rows": {name: rows for name, _, _, rows in stages},
            "stage_seconds_per_step": per}


def sample_rows(spec, ns, extra=0):
    import synth
    return synth.make_points(spec.with_n(max(ns, extra)))


# ------------------------------------------------------------------------- workloads

def fit_step(km, P, k, T, idx, timer, name):
    st = km.KmFitStats()
    C, a, J = km.kmeans_fit(P, k, T, idx, stats=st)
    if timer is not None:
        timer.add(name, st)
    return C, a, J


def final_cost(km, P32, X, a, mu):
    km.kmeans_update(P32, a, mu, km.KM_EMPTY_KEEP, counts=False)
    return km.kmeans_cost(X, mu, a)


def line(value, unit, dtype, config, **extra):
    out = {"value": value, "unit": unit, "dtype": dtype, "config": config}
    out.update(extra)
    return out


def wl_c1(cfg, torch, km, args):
    spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
    import synth
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        C, a, J = fit_step(km, P, k, T, idx, timer, "f32")
        return {"a": a, "cost": final_cost(km, P, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["f32"]
        return line(T * K / elapsed, "Lloyd iters/s", "f32",
                    {"workload": cfg["name"], "N": spec.n, "d": spec.d, "k": k, "iters": T, "format": "f32"},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    roofline=roofline(cfg["name"], s, 2.0 * spec.n * k * spec.d, "fp32",
                                      "assign_f32_kernel", "assign_f32_kernel"),
                    update_hbm=update_hbm(s, spec.n * (4 * spec.d + 4), "4d+4 per point"),
                    stages={"f32": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc
        Xh = synth.make_points(spec)
        t, _ = _timed(lambda: orc.fit({"fmt": "f32", "X": Xh}, k, T, idx))
        return {"value": T / t, "unit": "Lloyd iters/s", "cores": orc.num_threads(), "kind": "oracle",
                "sample": f"the whole fit ({T} iterations, {spec.n} points, k={k}) timed in full: {t:.2f} s"}

    def quality(out):
        return {"f32": partition_stats(km, X, out["a"], mu)}

    return step, finish, cpu_baseline, quality


def wl_c2_f32(cfg, torch, km, args):
    spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    wname = "gmm1m_d768_k1000_f32"

    def step(timer):
        C, a, J = fit_step(km, P, k, T, idx, timer, "f32")
        return {"a": a, "cost": final_cost(km, P, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["f32"]
        return line(T * K / elapsed, "Lloyd iters/s", "f32",
                    {"workload": wname, "N": spec.n, "d": spec.d, "k": k, "iters": T, "format": "f32",
                     "components": spec.components, "sigma": spec.sigma},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=roofline(wname, s, 2.0 * spec.n * k * spec.d, "fp32", "assign_f32_kernel",
                                      "assign_f32_kernel"),
                    update_hbm=update_hbm(s, spec.n * (4 * spec.d + 4), "4d+4 per point"),
                    stages={"f32": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs, C = Xs[:ns], np.ascontiguousarray(Xs[:k])
            ta, (a, _) = _timed(lambda: orc.assign_f32(xs, C))
            tu, _ = _timed(lambda: orc.update_f32(xs, a, k, C))
            tc, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("assign", ta, T + 1, ns), ("update", tu, T, ns), ("partition_cost", tc, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 1000, spec.n, f"fp32 Lloyd, k={k}, d={spec.d}")

    def quality(out):
        return {"f32": partition_stats(km, X, out["a"], mu)}

    return step, finish, cpu_baseline, quality


def wl_c2_sq8(cfg, torch, km, args):
    spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    wname = "gmm1m_d768_k1000_sq8"

    def step(timer):
        codes, params = km.quantize_sq8(X)
        C, a, J = fit_step(km, km.points_sq8(codes), k, T, idx, timer, "sq8")
        return {"a": a, "C": C, "params": params, "cost": final_cost(km, P32, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["sq8"]
        return line(T * K / elapsed, "Lloyd iters/s", "u8",
                    {"workload": wname, "N": spec.n, "d": spec.d, "k": k, "iters": T, "format": "sq8",
                     "components": spec.components, "sigma": spec.sigma},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=roofline(wname, s, 2.0 * spec.n * k * spec.d, "int8", "assign_q8_kernel<sq8>",
                                      "assign_q8_kernel"),
                    update_hbm=update_hbm(s, spec.n * (spec.d + 4), "d+4 per point"),
                    stages={"sq8": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs = Xs[:ns]
            tq, (lo, hi) = _timed(lambda: orc.sq8_fit(xs))
            te, codes = _timed(lambda: orc.sq8_encode(xs, lo, hi))
            C = orc.sq8_encode(np.ascontiguousarray(Xs[:k]), lo, hi)
            ta, (a, _) = _timed(lambda: orc.assign_sq8(codes, C))
            tu, _ = _timed(lambda: orc.update_sq8(codes, a, k, C))
            tc, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("sq8_fit", tq, 1, ns), ("sq8_encode", te, 1, ns), ("assign", ta, T + 1, ns),
                    ("update", tu, T, ns), ("partition_cost", tc, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 1000, spec.n, f"SQ8 Lloyd, k={k}, d={spec.d}")

    def quality(out):
        lo, hi = out["params"][:spec.d], out["params"][spec.d:]
        own = lo + out["C"].float() * ((hi - lo) / 255.0)  # centroids reconstructed from their codes
        return quality_vs_f32(km, X, k, T, idx, mu, "sq8", out["a"], own)

    return step, finish, cpu_baseline, quality


def wl_c3(cfg, torch, km, args):
    spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        bits, m, alpha, _ = km.quantize_sign1(X)
        C, a, J = fit_step(km, km.points_sign1(bits, alpha, m, spec.d), k, T, idx, timer, "sign1")
        return {"a": a, "C": C, "cost": final_cost(km, P32, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["sign1"]
        return line(T * K / elapsed, "Lloyd iters/s", "i8",
                    {"workload": cfg["name"], "N": spec.n, "d": spec.d, "k": k, "iters": T, "format": "sign1"},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=roofline(cfg["name"], s, 2.0 * spec.n * k * spec.d, "int8", "assign_bits_kernel<sign1>",
                                      "assign_bits_kernel"),
                    update_hbm=update_hbm(s, spec.n * (spec.d // 8 + 8), "d/8+8 per point"),
                    stages={"sign1": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs = Xs[:ns]
            tm, m = _timed(lambda: orc.col_mean(xs))
            te, (bits, alpha) = _timed(lambda: orc.sign1_encode(xs, m))
            C = np.ascontiguousarray(Xs[:k])
            ta, (a, _, _) = _timed(lambda: orc.assign_sign1(bits, alpha, C, m))
            tu, _ = _timed(lambda: orc.update_sign1(bits, alpha, spec.d, m, a, k, C))
            tc, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("col_mean", tm, 1, ns), ("sign1_encode", te, 1, ns), ("assign", ta, T + 1, ns),
                    ("update", tu, T, ns), ("partition_cost", tc, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 1000, spec.n, f"1-bit Lloyd, k={k}, d={spec.d}")

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "sign1", out["a"], out["C"])

    return step, finish, cpu_baseline, quality


def wl_c4(cfg, torch, km, args):
    spec, k, T, dout = cfg["spec"], cfg["k"], cfg["iters"], cfg["d_out"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    Y = torch.empty((spec.n, dout), dtype=torch.float32, device="cuda")
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    keep = {}

    def step(timer):
        mean, cov = km.pca_fit_cov(X)
        cov_h = cov.cpu().numpy()  # waits for the covariance
        t0 = time.perf_counter()
        # host eigensolve of the d x d covariance in its own precision (fp32),
        # LAPACK's divide and conquer
        w, V = scipy.linalg.eigh(cov_h, driver="evd", check_finite=False)
        w = w.astype(np.float64)
        order = np.argsort(w)[::-1][:dout]
        W = torch.from_numpy(np.ascontiguousarray(V[:, order], dtype=np.float32)).cuda()
        if timer is not None:
            timer.host("eigensolve", 1e3 * (time.perf_counter() - t0))
        km.pca_project(X, mean, W, out=Y)
        C, a, J = fit_step(km, km.points_f32(Y), k, T, idx, timer, "pca")
        keep.update(W=W, mean=mean, C=C, J=J, w=w[order], wsum=float(w.sum()))
        return {"a": a, "cost": final_cost(km, P32, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["pca"]
        return line(T * K / elapsed, "Lloyd iters/s", "f32",
                    {"workload": cfg["name"], "N": spec.n, "d": spec.d, "d_out": dout, "k": k, "iters": T,
                     "format": "f32 (PCA-projected)"},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=roofline(cfg["name"], s, 2.0 * spec.n * k * dout, "fp32", "assign_f32_kernel",
                                      "assign_f32_kernel"),
                    update_hbm=update_hbm(s, spec.n * (4 * dout + 4), "4d'+4 per point"),
                    host_eigensolve_ms_per_step=timer.host_ms.get("eigensolve", 0.0) / K,
                    stages={"pca": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs = Xs[:ns]
            # the oracle's covariance walks columns with the row stride: timed on at most
            # 2000 rows (where its per-row cost is that of a cached walk) and scaled from there
            ncov = min(ns, 2000)
            tc, (mean64, cov) = _timed(lambda: orc.pca_cov(xs[:ncov]))
            te, (W, _) = _timed(lambda: orc.pca_basis(cov, dout))
            mean = mean64.astype(np.float32)
            tp, Ys = _timed(lambda: orc.project(xs, mean, W))
            C = orc.project(np.ascontiguousarray(Xs[:k]), mean, W)
            ta, (a, _) = _timed(lambda: orc.assign_f32(Ys, C))
            tu, _ = _timed(lambda: orc.update_f32(Ys, a, k, C))
            tq, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("pca_cov", tc, 1, ncov), ("eigensolve", te, 1, None), ("project", tp, 1, ns),
                    ("assign", ta, T + 1, ns), ("update", tu, T, ns), ("partition_cost", tq, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 500, 200_000,
                               f"PCA-{dout} then fp32 Lloyd, k={k}, d={spec.d}")

    def quality(out):
        # Table 6: the recomputed cost (raw-vector means) is the main figure; the
        # unprojected centroids C W^T + mean and the preserved variance come with it
        own = keep["C"] @ keep["W"].t() + keep["mean"]
        q = quality_vs_f32(km, X, k, T, idx, mu, "pca", out["a"], own)
        q["preserved_variance"] = float(keep["w"].sum() / keep["wsum"])
        return q

    return step, finish, cpu_baseline, quality


def wl_c5(cfg, torch, km, args):
    spec, k, T, d0 = cfg["spec"], cfg["k"], cfg["iters"], cfg["d_front"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        bits, m, alpha, front = km.quantize_sign1(X, d_front=d0, want_front=True)
        P = km.points_hybrid(front, bits, alpha, m, spec.d)
        C, a, J = fit_step(km, P, k, T, idx, timer, "hybrid")
        del front
        return {"a": a, "C": C, "cost": final_cost(km, P32, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["hybrid"]
        return line(T * K / elapsed, "Lloyd iters/s", "f32+i8",
                    {"workload": cfg["name"], "N": spec.n, "d": spec.d, "d_front": d0, "k": k, "iters": T,
                     "format": "hybrid (fp32 front + 1-bit tail)"},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=dict(roofline(cfg["name"], s, 2.0 * spec.n * k * d0, "fp32", "assign_hyb_kernel",
                                           "assign_hyb_kernel"),
                                  work="2 d_front operations per (point, centroid) pair on fp32 MFMA (the front "
                                       "contraction; the 1-bit tail's int8 work rides in the same launch)"),
                    update_hbm=update_hbm(s, spec.n * (4 * d0 + (spec.d - d0) // 8 + 8),
                                          "4 d_front + (d - d_front)/8 + 8 per point"),
                    stages={"hybrid": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs = Xs[:ns]
            tm, m = _timed(lambda: orc.col_mean(xs))
            te, (bits, alpha) = _timed(lambda: orc.sign1_encode(xs, m, d0))
            tf, front = _timed(lambda: np.ascontiguousarray(xs[:, :d0]))
            C = np.ascontiguousarray(Xs[:k])
            ta, (a, _) = _timed(lambda: orc.assign_hybrid(front, bits, alpha, C, m, d0))
            tu, _ = _timed(lambda: orc.update_sign1(bits, alpha, spec.d, m, a, k, C, front=front, d0=d0))
            tc, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("col_mean", tm, 1, ns), ("sign1_encode", te, 1, ns), ("front_copy", tf, 1, ns),
                    ("assign", ta, T + 1, ns), ("update", tu, T, ns), ("partition_cost", tc, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 500, 200_000,
                               f"hybrid Lloyd (fp32 front {d0} + 1-bit tail), k={k}, d={spec.d}")

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "hybrid", out["a"], out["C"])

    return step, finish, cpu_baseline, quality


def wl_bf16(cfg, torch, km, args):
    """The 1M x 768, k=1000 mixture stored as bfloat16 (conversion in the step)."""
    spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    wname = "gmm1m_d768_k1000_bf16"

    def step(timer):
        Xb = km.quantize_bf16(X)
        C, a, J = fit_step(km, km.points_bf16(Xb), k, T, idx, timer, "bf16")
        return {"a": a, "C": C, "cost": final_cost(km, P32, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["bf16"]
        return line(T * K / elapsed, "Lloyd iters/s", "bf16",
                    {"workload": wname, "N": spec.n, "d": spec.d, "k": k, "iters": T, "format": "bf16"},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=roofline(wname, s, 2.0 * spec.n * k * spec.d, "bf16", "assign_q8_kernel<bf16>",
                                      "assign_q8_kernel<bf16>"),
                    update_hbm=update_hbm(s, spec.n * (2 * spec.d + 4), "2d+4 per point"),
                    stages={"bf16": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs = Xs[:ns]
            tr, codes = _timed(lambda: orc.bf16_round(xs))
            C = orc.bf16_decode(orc.bf16_round(np.ascontiguousarray(Xs[:k])))
            ta, (a, _) = _timed(lambda: orc.assign_bf16(codes, C))
            tu, _ = _timed(lambda: orc.update_bf16(codes, a, k, C))
            tc, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("bf16_round", tr, 1, ns), ("assign", ta, T + 1, ns), ("update", tu, T, ns),
                    ("partition_cost", tc, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 1000, spec.n, f"bf16 Lloyd, k={k}, d={spec.d}")

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "bf16", out["a"], out["C"])

    return step, finish, cpu_baseline, quality


def wl_lvq4(cfg, torch, km, args):
    """The 1M x 768, k=1000 mixture as LVQ4 codes.  One step: encode (per-vector bias,
    scale, packed 4-bit codes, cached A and N), kmeans_fit on the codes (centroids
    LVQ4-coded per pass, decode-averaging update), partition cost."""
    spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    wname = "gmm1m_d768_k1000_lvq4"

    def step(timer):
        codes, par = km.quantize_lvq4(X)
        C, a, J = fit_step(km, km.points_lvq4(codes, par, spec.d), k, T, idx, timer, "lvq4")
        return {"a": a, "C": C, "cost": final_cost(km, P32, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["lvq4"]
        return line(T * K / elapsed, "Lloyd iters/s", "u4+i8",
                    {"workload": wname, "N": spec.n, "d": spec.d, "k": k, "iters": T, "format": "lvq4"},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=roofline(wname, s, 2.0 * spec.n * k * spec.d, "int8", "assign_q8_kernel<lvq4>",
                                      "assign_q8_kernel<lvq4>"),
                    update_hbm=update_hbm(s, spec.n * (spec.d // 2 + 20), "d/2+20 per point"),
                    stages={"lvq4": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs = Xs[:ns]
            te, (codes, par) = _timed(lambda: orc.lvq4_encode(xs))
            C = np.ascontiguousarray(Xs[:k])
            ta, (a, _, _) = _timed(lambda: orc.assign_lvq4(codes, par, C))
            tu, _ = _timed(lambda: orc.update_lvq4(codes, par, a, k, C))
            tc, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("lvq4_encode", te, 1, ns), ("assign", ta, T + 1, ns), ("update", tu, T, ns),
                    ("partition_cost", tc, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 1000, spec.n, f"LVQ4 Lloyd, k={k}, d={spec.d}")

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "lvq4", out["a"], out["C"])

    return step, finish, cpu_baseline, quality


def wl_rabitq(cfg, torch, km, args):
    """The 1M x 1024, k=1024 mixture through the paper's RabitQ pipeline: centre, random
    rotation, 1-bit codes; SQ4 centroid codes; last update from the rotated raw rows."""
    spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    rot_np = synth.random_rotation(spec.d)
    rot = torch.from_numpy(rot_np).cuda()
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    keep = {}

    def step(timer):
        bits, m, alpha, Yr = km.rabitq_encode(X, rot, want_rotated=True)
        C, a, J = fit_step(km, km.points_rabitq(bits, alpha, spec.d, raw=Yr), k, T, idx, timer, "rabitq")
        keep.update(bits=bits, alpha=alpha, m=m, C=C)
        return {"a": a, "cost": final_cost(km, P32, X, a, mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["rabitq"]
        return line(T * K / elapsed, "Lloyd iters/s", "i8",
                    {"workload": "gmm1m_d1024_k1024_rabitq", "N": spec.n, "d": spec.d, "k": k, "iters": T,
                     "format": "rabitq", "raw_last_update": True},
                    distances_per_s=(T + 1) * spec.n * k * K / elapsed,
                    partition_cost=float(out["cost"].item()),
                    roofline=roofline("gmm1m_d1024_k1024_rabitq", s, 2.0 * spec.n * k * spec.d, "int8",
                                      "assign_bits_kernel<rabitq>", "assign_bits_kernel<rabitq>"),
                    stages={"rabitq": stage_summary(s)})

    def cpu_baseline():
        import oracle as orc

        def run(ns):
            Xs = sample_rows(spec, ns, k)
            xs = Xs[:ns]
            tm, m = _timed(lambda: orc.col_mean(xs))
            tp, Ys = _timed(lambda: orc.project(xs, m, rot_np))
            zero = np.zeros(spec.d, np.float32)
            te, (bits, alpha) = _timed(lambda: orc.sign1_encode(Ys, zero))
            C = orc.project(np.ascontiguousarray(Xs[:k]), m, rot_np)
            ta, (a, _, _) = _timed(lambda: orc.assign_rabitq(bits, alpha, C))
            tu, _ = _timed(lambda: orc.update_sign1(bits, alpha, spec.d, zero, a, k, C))
            tr, _ = _timed(lambda: orc.update_f32(Ys, a, k, C))
            tc, _ = _timed(lambda: orc.partition_cost(xs, a, k))
            return [("col_mean", tm, 1, ns), ("rotate", tp, 1, ns), ("sign1_encode", te, 1, ns),
                    ("assign", ta, T + 1, ns), ("update", tu, T - 1, ns), ("raw_last_update", tr, 1, ns),
                    ("partition_cost", tc, 1, ns)]
        return oracle_baseline(run, spec.n, T, args.cpu_seconds, 1000, spec.n, f"RabitQ Lloyd, k={k}, d={spec.d}")

    def quality(out):
        own = keep["C"] @ rot.t() + keep["m"]  # centroids back in the original space
        q = quality_vs_f32(km, X, k, T, idx, mu, "rabitq", out["a"], own)
        _, a2, _ = km.kmeans_fit(km.points_rabitq(keep["bits"], keep["alpha"], spec.d), k, T, idx, objective=False)
        q["rabitq_codes_only"] = partition_stats(km, X, a2, mu)
        q["objective_ratio_rabitq_codes_only_vs_f32"] = q["rabitq_codes_only"]["cost"] / q["f32"]["cost"]
        return q

    return step, finish, cpu_baseline, quality


def wl_hier(fmt):
    def build(cfg, torch, km, args):
        """Hierarchical k-means on the 10M x 1024 mixture with the paper's k = 4 sqrt(N)
        = 12649 (Table 7): MESO (round(sqrt(k)) = 112 centroids) and FINE phases of 10
        Lloyd iterations each, no refinement (SQ8: quantisation inside the step)."""
        spec = cfg["spec"]
        import synth
        k = int(round(4 * math.sqrt(spec.n)))
        Tm = Tf = 10
        log(f"generating {spec.n} x {spec.d} mixture")
        X = upload(spec, torch)
        P32 = km.points_f32(X)
        kmeso = int(np.floor(np.sqrt(k) + 0.5))
        init = synth.init_indices(spec.n, kmeso)
        mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
        wname = f"gmm{spec.n // 1000000}m_d{spec.d}_k{k}_hier_{fmt}"
        res = {}

        def step(timer):
            st = km.KmFitStats()
            P = P32 if fmt == "f32" else km.points_sq8(km.quantize_sq8(X)[0])
            C, a, kf, J, ph, am = km.kmeans_fit_hier(P, k, init, Tm, Tf, 0, stats=st, phases=True, meso=True)
            if timer is not None:
                timer.add(fmt, st)
                res.update(ph=ph, kf=kf, am=am)
            return {"a": a, "cost": final_cost(km, P32, X, a, mu)}

        def finish(out, timer, elapsed, K):
            s = timer.stats[fmt]
            n_i = torch.bincount(res["am"].long(), minlength=kmeso).cpu().numpy().astype(np.float64)
            work_meso = 2.0 * spec.n * kmeso * spec.d
            work_fine = 2.0 * spec.d * float((n_i * res["kf"]).sum())
            work = K * ((Tm + 1) * work_meso + (Tf + 1) * work_fine)
            ach = work / (s["assign_ms"] * 1e-3) / 1e12
            peak = "fp32" if fmt == "f32" else "int8"
            kern = "assign_f32_kernel" if fmt == "f32" else "assign_q8_kernel<sq8>"
            return line(K / elapsed, "fits/s", "f32" if fmt == "f32" else "u8",
                        {"workload": wname, "N": spec.n, "d": spec.d, "k": k, "k_meso": kmeso, "iters_meso": Tm,
                         "iters_fine": Tf, "iters_refine": 0, "format": fmt},
                        metric="hierarchical k-means fits/s (build time of Table 7)",
                        partition_cost=float(out["cost"].item()),
                        ms_per_fit=float(res["ph"].sum()),
                        phase_ms={"meso": res["ph"][0], "fine": res["ph"][1]},
                        roofline={"bound": "mfma", "kernel": f"{kern} (meso launches and segmented fine launches)",
                                  "achieved": ach, "peak": PEAK[peak], "unit": PEAK_UNIT[peak],
                                  "frac": ach / PEAK[peak], "traffic": None,
                                  "algorithmic_work_per_fit": work / K},
                        stages={fmt: stage_summary(s)})

        def cpu_baseline():
            import oracle as orc

            def run(ns):
                Xs = sample_rows(spec, ns)
                ks = int(round(4 * math.sqrt(ns)))
                P = {"fmt": "f32", "X": Xs}
                tq = 0.0
                if fmt == "sq8":
                    tq, (lo, hi) = _timed(lambda: orc.sq8_fit(Xs))
                    te, codes = _timed(lambda: orc.sq8_encode(Xs, lo, hi))
                    tq += te
                    P = {"fmt": "sq8", "codes": codes}
                init_s = synth.init_indices(ns, orc.meso_count(ks))
                t, _ = _timed(lambda: orc.fit_hier(P, ks, Tm, Tf, 0, init_s))
                return [("quantize", tq, 1, ns), ("fit_hier", t, 1, None)]
            # meso work N k_meso d and fine work sum n_i k_i d both grow as N sqrt(k) = 2 N^1.25 d:
            # the sample's fit is scaled by (N / ns)^1.25, its quantisation by N / ns
            r = oracle_baseline(lambda ns: run(ns), spec.n, 1, args.cpu_seconds, 4000, 400_000,
                                f"hierarchical {fmt}, k = 4 sqrt(N)", unit="fits/s", per_step=1)
            ns = int(re.search(r"first (\d+) of", r["sample"]).group(1))
            fit_s = r["stage_seconds_per_step"]["fit_hier"] * (spec.n / ns) ** 1.25
            step_s = fit_s + r["stage_seconds_per_step"]["quantize"]
            r["stage_seconds_per_step"]["fit_hier"] = fit_s
            r["value"] = 1.0 / step_s
            r["sample"] += (f"; the fit itself (k = 4 sqrt(ns) on the sample) scaled by (N/ns)^1.25 instead, "
                            f"since meso and fine work grow as N sqrt(k); {step_s:.1f} s per fit extrapolated")
            return r

        def quality(out):
            q = {fmt: partition_stats(km, X, out["a"], mu)}
            log("quality: one vanilla fp32 pass at full k (outside the timed region)")
            C = mu.clone()
            km.kmeans_assign(P32, C, score=False)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            a, _, _ = km.kmeans_assign(P32, C, score=False)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            km.kmeans_update(P32, a, C, counts=False)
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            vanilla_ms = 1e3 * (11 * (t1 - t0) + 10 * (t2 - t1))
            q["vanilla_f32_T10_ms_estimate"] = vanilla_ms
            q["speedup_vs_vanilla_f32"] = vanilla_ms / float(res["ph"].sum())
            # Sec. 4.4 taken literally: round(sqrt(n_i)) fine clusters per meso-cluster
            # (the same meso partition: the meso phase is deterministic), C sized to their sum
            n_i = torch.bincount(res["am"].long(), minlength=kmeso).cpu().numpy().astype(np.int64)
            r = np.floor(np.sqrt(n_i.astype(np.float64))).astype(np.int64)
            r -= (r * r > n_i)
            r += ((r + 1) * (r + 1) <= n_i)
            cap = int(np.where(n_i > 0, np.where(n_i - r * r > r, r + 1, r), 0).sum())
            log(f"quality: the paper's literal fine counts ({cap} fine clusters), outside the timed region")
            P = P32 if fmt == "f32" else km.points_sq8(km.quantize_sq8(X)[0])
            C2, a2, kf2, _, ph2 = km.kmeans_fit_hier(P, cap, init, Tm, Tf, 0, k_meso=kmeso, objective=False,
                                                     phases=True, sqrt_rule=True)
            mu2 = torch.empty((len(C2), spec.d), dtype=torch.float32, device="cuda")
            lit = partition_stats(km, X, a2, mu2)
            lit.update(k_fine_total=int(kf2.sum()), ms_per_fit=float(ph2.sum()),
                       phase_ms={"meso": float(ph2[0]), "fine": float(ph2[1])})
            lit["meso_sizes"] = {"min": int(n_i.min()), "max": int(n_i.max()),
                                 "cv": float(n_i.std() / max(n_i.mean(), 1e-30))}
            q["sqrt_rule"] = lit
            q["objective_ratio_sqrt_rule_vs_reading"] = lit["cost"] / q[fmt]["cost"]
            return q

        return step, finish, cpu_baseline, quality
    return build


def wl_pruned(fmt):
    def build(cfg, torch, km, args):
        """The 1M x 768, k=1000 mixture under a random rotation, clustered with
        dimension pruning in every assignment pass after the first (SuperKMeans with
        the ADSampling test, eps0 = 2.1, d' = 96).  One step: rotation (projection
        with an orthogonal matrix), SQ8 encode for SQ8, pruned fit, partition cost."""
        spec, k, T = cfg["spec"], cfg["k"], cfg["iters"]
        import synth
        log(f"generating {spec.n} x {spec.d} mixture")
        X = upload(spec, torch)
        idx = synth.init_indices(spec.n, k)
        R_np = synth.random_rotation(spec.d, 11)
        R = torch.from_numpy(R_np).cuda()
        zero = torch.zeros(spec.d, dtype=torch.float32, device="cuda")
        Y = torch.empty_like(X)
        P32 = km.points_f32(X)
        mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
        wname = f"gmm{spec.n // 1000000}m_d{spec.d}_k{k}_pruned_{fmt}"
        res = {}

        def points():
            if fmt == "f32":
                return km.points_f32(Y)
            codes, _ = km.quantize_sq8(Y)
            res["codes"] = codes
            return km.points_sq8(codes)

        def step(timer):
            km.pca_project(X, zero, R, out=Y)
            st = km.KmFitStats()
            C, a, J, cnt = km.kmeans_fit_pruned(points(), k, T, idx, stats=st, counters=True)
            if timer is not None:
                timer.add(fmt, st)
                res["cnt"] = cnt
            return {"a": a, "cost": final_cost(km, P32, X, a, mu)}  # the rotation keeps distances

        def finish(out, timer, elapsed, K):
            s = timer.stats[fmt]
            c = res["cnt"].astype(np.float64)
            # the MFMA work of the assignment passes of one fit: the first, full pass,
            # then T pruned passes (the d'-dim front on every pair, the full distance on
            # the survivors), against the whole assignment stage's time (front, tau and
            # refinement kernels alike)
            d_front = 32 * ((spec.d + 255) // 256)
            work = K * (2.0 * spec.n * k * spec.d + T * 2.0 * spec.n * k * d_front + 2.0 * spec.d * c[2])
            ach = work / (s["assign_ms"] * 1e-3) / 1e12
            peak = "fp32" if fmt == "f32" else "int8"
            return line(T * K / elapsed, "Lloyd iters/s", "f32" if fmt == "f32" else "u8",
                        {"workload": wname, "N": spec.n, "d": spec.d, "k": k, "iters": T, "format": fmt,
                         "eps0": 2.1, "d_front": 32 * ((spec.d + 255) // 256), "rotation": "random orthogonal"},
                        partition_cost=float(out["cost"].item()),
                        survivors={"front_pass": c[1] / max(1.0, c[0]), "full_distance": c[2] / max(1.0, c[0]),
                                   "candidates_tested_per_pass": c[0] / T},
                        roofline={"bound": "mfma", "kernel": "all assignment launches (first full pass, then the "
                                  "pruned front, threshold and refinement kernels)",
                                  "achieved": ach, "peak": PEAK[peak], "unit": PEAK_UNIT[peak],
                                  "frac": ach / PEAK[peak], "traffic": None,
                                  "algorithmic_work_per_fit": work / K},
                        stages={fmt: stage_summary(s)})

        def cpu_baseline():
            import oracle as orc

            def run(ns):
                Xs = sample_rows(spec, ns, k)
                zero_h = np.zeros(spec.d, np.float32)
                tp, Ys = _timed(lambda: orc.project(Xs, zero_h, R_np))
                tq = 0.0
                P = {"fmt": "f32", "X": Ys[:ns]}
                if fmt == "sq8":
                    tq, (lo, hi) = _timed(lambda: orc.sq8_fit(Ys[:ns]))
                    te, codes = _timed(lambda: orc.sq8_encode(Ys, lo, hi))
                    tq += te
                    P = {"fmt": "sq8", "codes": codes[:ns]}
                    C = np.ascontiguousarray(codes[:k])
                else:
                    C = np.ascontiguousarray(Ys[:k])
                ta, (a, _) = _timed(lambda: orc.assign(P, C))
                tu, (C1, _) = _timed(lambda: orc.update(P, a, k, C))
                tpr, _ = _timed(lambda: orc.assign_pruned(P, C1, a))
                tc, _ = _timed(lambda: orc.partition_cost(Xs[:ns], a, k))
                return [("rotate", tp, 1, ns), ("quantize", tq, 1, ns), ("assign_full", ta, 1, ns),
                        ("update", tu, T, ns), ("assign_pruned", tpr, T, ns), ("partition_cost", tc, 1, ns)]
            r = oracle_baseline(run, spec.n, T, args.cpu_seconds, 1000, spec.n,
                                f"pruned {fmt} Lloyd, k={k}, d={spec.d}")
            r["sample"] += " (the pruned pass is timed right after the first update, before the partition settles)"
            return r

        def quality(out):
            log("quality: exact fit on the rotated rows (outside the timed region)")
            _, a_ex, _ = km.kmeans_fit(points(), k, T, idx, objective=False)
            q = {f"{fmt}_exact": partition_stats(km, X, a_ex, mu), f"{fmt}_pruned": partition_stats(km, X, out["a"], mu)}
            q["objective_ratio_pruned_vs_exact"] = q[f"{fmt}_pruned"]["cost"] / q[f"{fmt}_exact"]["cost"]
            return q

        return step, finish, cpu_baseline, quality
    return build


# name -> (builder, configuration whose data it uses)
WORKLOADS = {
    "c1": (wl_c1, 1), "c2-f32": (wl_c2_f32, 2), "c2-sq8": (wl_c2_sq8, 2), "c3": (wl_c3, 3), "c4": (wl_c4, 4),
    "c5": (wl_c5, 5), "bf16": (wl_bf16, 2), "rabitq": (wl_rabitq, 3), "lvq4": (wl_lvq4, 2),
    "hier-f32": (wl_hier("f32"), 4), "hier-sq8": (wl_hier("sq8"), 4),
    "pruned-f32": (wl_pruned("f32"), 2), "pruned-sq8": (wl_pruned("sq8"), 2),
}
ALIASES = {"1": "c1", "2": "c2-f32", "3": "c3", "4": "c4", "5": "c5", "6": "bf16", "7": "rabitq", "8": "lvq4",
           "9": "hier-f32", "10": "pruned-f32", "11": "c2-sq8", "12": "hier-sq8", "13": "pruned-sq8"}
DEFAULT_WORKLOAD = "c4"


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(WORKLOADS) + sorted(ALIASES))
    ap.add_argument("--n", type=int, default=None, help="override the number of points (measurement only)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle's CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true", help="run the counter-calibration copy kernels first")
    ap.add_argument("--no-quality", action="store_true",
                    help="skip the partition-quality figures computed after the timed region")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (points would be sharded "
              "by rows, one shard per GPU, with an all-reduce of the per-cluster sums); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_14648_amd as km
    import synth
    km.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    name = ALIASES.get(args.workload, args.workload)
    builder, cfg_id = WORKLOADS[name]
    cfg = dict(synth.config(cfg_id))
    if args.n is not None:
        cfg["spec"] = cfg["spec"].with_n(args.n)
    if args.copy_probe:
        copy_probe(torch)
    step, finish, cpu_baseline, quality = builder(cfg, torch, km, args)
    for i in range(args.warmup):
        step(None)
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")
    timer = Timer()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    out = None
    for i in range(args.steps):
        out = step(timer)
        log(f"timed step {i + 1}/{args.steps} issued")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    res = finish(out, timer, elapsed, args.steps)
    if args.n is not None:
        res["config"]["N_override"] = args.n
        if isinstance(res.get("roofline"), dict):
            res["roofline"]["traffic"] = None
    rec = {"metric": res.pop("metric", METRIC), "value": res.pop("value"), "unit": res.pop("unit"), "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": res.pop("dtype"),
           "data": "synthetic (seeded Gaussian mixture shaped like the paper's embedding workloads)",
           "config": res.pop("config")}
    rec.update(res)
    if quality is not None and not args.no_quality:
        rec["quality"] = quality(out)
    if cpu_baseline is not None and not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        rec["cpu_baseline"] = cpu_baseline()
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
