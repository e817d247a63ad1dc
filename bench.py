#!/usr/bin/env python3
"""Benchmark of the hot path on one MI355X: Lloyd k-means on compressed vectors.

Default workload (N=1): 1,000,000 x 768 unit-normalised Gaussian mixture of
1,000 components (sigma 0.15), k = 1,000, 20 Lloyd iterations, clustered twice:
as fp32 vectors and as per-dimension SQ8 codes.  One step =
  quantize (SQ8 parameters + codes)
  + kmeans_fit fp32 (init, 20 x (assign, update), final assign, objectives)
  + kmeans_fit SQ8  (same)
  + full-precision partition cost of both final partitions (raw-vector means).
Inputs are resident in HBM before the timed region.  `value` is Lloyd
iterations per second over the whole step (20 fp32 + 20 SQ8 iterations).

Other workloads (--workload 1|3|4|5) time the other configurations for
measurement; they are not the headline line.  --workload 6 runs the default
workload's data stored as bfloat16; --workload 7 runs the 1-bit workload's data
through the paper's RabitQ pipeline (random rotation, SQ4 centroid codes with
bias, last update from the raw rotated rows); --workload 8 runs the default
workload's data as LVQ4 codes; --workload 9 runs hierarchical k-means (meso,
then fine clustering inside each meso-cluster) on the 10M x 1024 data with
k = 4 sqrt(N), fp32 and SQ8, and reports fits per second; --workload 10 runs
the default workload's data under a random rotation with dimension pruning in
the assignment passes (fp32 and SQ8).

After the timed region, `quality` reports each final partition's full-precision
cost (raw-vector member means), its cluster-size spread and, for the compressed
formats other than SQ8, the ratio to an fp32 Lloyd run on the raw vectors with
the same initial centroids and iteration count (--no-quality skips it).

The JSON line carries the roofline of the dominant kernel (the fused fp32
assignment kernel, on fp32 MFMA), measured from HIP events recorded by the
library around each launch of that kernel on its stream, and the oracle timed on
this host on a bounded sample of the same workload.  `roofline.traffic` (bytes
the kernel moves between L2 and memory per launch) comes from the committed
rocprofv3 counter summary under profiles/; it is null when that summary is
missing, covers another workload, or was taken from a different source of the
kernel than the one built here.

--copy-probe runs a 1 GiB fill and a 1 GiB negating copy before the workload:
kernels of known traffic against which FETCH_SIZE / WRITE_SIZE are scaled.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Lloyd iters/s + point×centroid distances/s; objective ratio vs fp32 oracle"
PEAK = {"fp32_mfma_tflops": 157.3, "bf16_mfma_tflops": 2500.0, "int8_mfma_tops": 5000.0, "hbm_gbs": 8000.0}
COUNTERS = os.path.join(ROOT, "profiles", "counters__assign_f32_kernel__gmm1m_d768_k1000.md")
KERNEL_SOURCES = ("paper_2608_14648_amd/csrc/assign.hip", "paper_2608_14648_amd/csrc/common.hpp")
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

    def add(self, name, st):
        d = self.stats.setdefault(name, {"assign_ms": 0.0, "prep_ms": 0.0, "update_ms": 0.0, "other_ms": 0.0,
                                         "assign_passes": 0, "updates": 0})
        for key, v in st.as_dict().items():
            d[key] += v


def stage_summary(s):
    return {"assign_ms_per_pass": s["assign_ms"] / max(1, s["assign_passes"]),
            "update_ms_per_iter": s["update_ms"] / max(1, s["updates"]),
            "prep_ms_per_pass": s["prep_ms"] / max(1, s["assign_passes"]),
            "other_ms_total": s["other_ms"]}


def kernel_source_hash():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def counted_traffic(workload):
    """Calibrated L2<->memory bytes per launch of the fp32 assignment kernel.

    Read from the JSON block of the committed counter summary; None when the
    summary is absent, was taken on another workload, or the kernel's sources
    have changed since the counters were collected."""
    try:
        with open(COUNTERS) as f:
            text = f.read()
    except OSError:
        return None
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if m is None:
        return None
    rec = json.loads(m.group(1))
    if rec.get("workload") != workload or rec.get("source_sha256") != kernel_source_hash():
        return None
    return rec.get("traffic_bytes_per_launch")


def copy_probe(torch):
    """Kernels of known traffic for counter calibration: a fill that writes
    1 GiB, then a negating copy that reads 1 GiB and writes 1 GiB."""
    src = torch.ones(COPY_PROBE_FLOATS, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst
    log(f"copy probe done ({COPY_PROBE_FLOATS * 4} bytes)")


def partition_stats(km, X, a, mu):
    """Full-precision cost of a partition (raw-vector member means) and the spread
    of its cluster sizes."""
    _, cnt = km.kmeans_update(km.points_f32(X), a, mu, km.KM_EMPTY_KEEP, counts=True)
    cost = float(km.kmeans_cost(X, mu, a).item())
    c = cnt.cpu().numpy()
    return {"cost": cost, "cluster_size_std": float(c.std()), "empty_clusters": int((c == 0).sum())}


def f32_reference(km, X, k, T, idx, mu):
    """The quality baseline: fp32 Lloyd on the raw vectors, same init and T."""
    _, a, _ = km.kmeans_fit(km.points_f32(X), k, T, idx, objective=False)
    return partition_stats(km, X, a, mu)


def quality_vs_f32(km, X, k, T, idx, mu, name, a):
    log("quality: fp32 reference fit (outside the timed region)")
    q = {name: partition_stats(km, X, a, mu), "f32": f32_reference(km, X, k, T, idx, mu)}
    q[f"objective_ratio_{name}_vs_f32"] = q[name]["cost"] / q["f32"]["cost"]
    return q


# ------------------------------------------------------------------------- workloads

def workload_c2(cfg, torch, km, args):
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T = cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        codes, params = km.quantize_sq8(X)
        P8 = km.points_sq8(codes)
        s32, s8 = km.KmFitStats(), km.KmFitStats()
        C32, a32, J32 = km.kmeans_fit(P32, k, T, idx, stats=s32)
        C8, a8, J8 = km.kmeans_fit(P8, k, T, idx, stats=s8)
        out = {"a_f32": a32, "a_sq8": a8}
        for name, a in (("f32", a32), ("sq8", a8)):  # full-precision cost of the final partition
            km.kmeans_update(P32, a, mu, km.KM_EMPTY_KEEP, counts=False)
            out[name] = km.kmeans_cost(X, mu, a)
        if timer is not None:
            timer.add("f32", s32)
            timer.add("sq8", s8)
        return out, (J32, J8)

    def quality(out):
        return {name: partition_stats(km, X, out["a_" + name], mu) for name in ("f32", "sq8")}

    def finish(out, timer, elapsed, K):
        c32 = float(out["f32"].item())
        c8 = float(out["sq8"].item())
        f = timer.stats["f32"]
        q = timer.stats["sq8"]
        a_ms = f["assign_ms"] / f["assign_passes"]
        flop = 2.0 * spec.n * k * spec.d
        achieved = flop / (a_ms * 1e-3) / 1e12
        q_ms = q["assign_ms"] / q["assign_passes"]
        iters = 2 * T * K
        res = {
            "value": iters / elapsed,
            "unit": "Lloyd iters/s",
            "dtype": "f32+i8",
            "config": {"workload": cfg["name"], "N": spec.n, "d": spec.d, "k": k, "iters": T,
                       "formats": ["f32", "sq8"], "components": spec.components, "sigma": spec.sigma},
            "distances_per_s": 2 * (T + 1) * spec.n * k * K / elapsed,
            "objective_ratio_sq8_vs_f32": c8 / c32,
            "partition_cost": {"f32": c32, "sq8": c8},
            "roofline": {"bound": "mfma", "kernel": "assign_f32_kernel", "achieved": achieved,
                         "peak": PEAK["fp32_mfma_tflops"], "unit": "TFLOP/s",
                         "frac": achieved / PEAK["fp32_mfma_tflops"],
                         "traffic": counted_traffic(cfg["name"]) if args.n is None else None,
                         "avg_launch_ms": a_ms, "flop_per_launch": flop},
            "roofline_sq8_assign": {"bound": "mfma", "achieved": 2.0 * spec.n * k * spec.d / (q_ms * 1e-3) / 1e12,
                                    "peak": PEAK["int8_mfma_tops"], "unit": "TOP/s",
                                    "frac": 2.0 * spec.n * k * spec.d / (q_ms * 1e-3) / 1e12 / PEAK["int8_mfma_tops"],
                                    "avg_launch_ms": q_ms},
            "update_f32_hbm": {"bytes_per_update": spec.n * (4 * spec.d + 4),
                               "achieved_gbs": spec.n * (4 * spec.d + 4) / (f["update_ms"] / f["updates"] * 1e-3) / 1e9,
                               "peak_gbs": PEAK["hbm_gbs"]},
            "stages": {"f32": stage_summary(f), "sq8": stage_summary(q)},
        }
        res["update_f32_hbm"]["frac"] = res["update_f32_hbm"]["achieved_gbs"] / PEAK["hbm_gbs"]
        return res

    def cpu_baseline():
        import oracle as orc
        Xh = synth.make_points(spec.with_n(min(spec.n, 200_000)))
        C = np.ascontiguousarray(Xh[:k])
        lo, hi = orc.sq8_fit(Xh)

        def one_iter(ns):
            xs = Xh[:ns]
            codes = orc.sq8_encode(xs, lo, hi)
            t0 = time.perf_counter()
            a, _ = orc.assign_f32(xs, C)
            orc.update_f32(xs, a, k, C)
            t1 = time.perf_counter()
            a8, _ = orc.assign_sq8(codes, codes[:k])
            orc.update_sq8(codes, a8, k, codes[:k])
            t2 = time.perf_counter()
            return t1 - t0, t2 - t1

        c32, c8 = one_iter(1000)
        ns = int(min(len(Xh), max(1000, 1000 * args.cpu_seconds / max(c32 + c8, 1e-6))))
        t32, t8 = one_iter(ns)
        scale = spec.n / ns
        per_iter = (t32 + t8) * scale / 2  # one fp32 and one SQ8 iteration, extrapolated to N
        return {"value": 1.0 / per_iter, "unit": "Lloyd iters/s", "cores": orc.num_threads(), "kind": "oracle",
                "sample": f"one fp32 and one SQ8 Lloyd iteration (assign + update) on the first {ns} of the "
                          f"{spec.n} points, k={k}, d={spec.d}, timed {t32 + t8:.2f} s, extrapolated linearly to N"}

    return step, finish, cpu_baseline, quality


def workload_bf16(cfg, torch, km, args):
    """The 1M x 768, k=1000 mixture stored as bfloat16 (measurement only)."""
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T = cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        Xb = km.quantize_bf16(X)
        st = km.KmFitStats()
        C, a, J = km.kmeans_fit(km.points_bf16(Xb), k, T, idx, stats=st)
        km.kmeans_update(P32, a, mu, km.KM_EMPTY_KEEP, counts=False)
        cost = km.kmeans_cost(X, mu, a)
        if timer is not None:
            timer.add("bf16", st)
        return {"bf16": cost, "a": a}, J

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "bf16", out["a"])

    def finish(out, timer, elapsed, K):
        s = timer.stats["bf16"]
        a_ms = s["assign_ms"] / s["assign_passes"]
        flop = 2.0 * spec.n * k * spec.d
        ach = flop / (a_ms * 1e-3) / 1e12
        return {"value": T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "bf16",
                "config": {"workload": "gmm1m_d768_k1000_bf16", "N": spec.n, "d": spec.d, "k": k, "iters": T,
                           "formats": ["bf16"]},
                "distances_per_s": (T + 1) * spec.n * k * K / elapsed,
                "partition_cost": {"bf16": float(out["bf16"].item())},
                "roofline": {"bound": "mfma", "kernel": "assign_q8_kernel<bf16>", "achieved": ach,
                             "peak": PEAK["bf16_mfma_tflops"], "unit": "TFLOP/s",
                             "frac": ach / PEAK["bf16_mfma_tflops"], "traffic": None, "avg_launch_ms": a_ms},
                "stages": {"bf16": stage_summary(s)}}

    return step, finish, None, quality


def workload_lvq4(cfg, torch, km, args):
    """The 1M x 768, k=1000 mixture as LVQ4 codes (measurement only).  One step: encode
    (per-vector bias, scale, packed 4-bit codes, cached A and N), kmeans_fit on the codes
    (centroids LVQ4-coded per pass, decode-averaging update), partition cost."""
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T = cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        codes, par = km.quantize_lvq4(X)
        st = km.KmFitStats()
        C, a, J = km.kmeans_fit(km.points_lvq4(codes, par, spec.d), k, T, idx, stats=st)
        km.kmeans_update(P32, a, mu, km.KM_EMPTY_KEEP, counts=False)
        cost = km.kmeans_cost(X, mu, a)
        if timer is not None:
            timer.add("lvq4", st)
        return {"lvq4": cost, "a": a}, J

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "lvq4", out["a"])

    def finish(out, timer, elapsed, K):
        s = timer.stats["lvq4"]
        a_ms = s["assign_ms"] / s["assign_passes"]
        ops = 2.0 * spec.n * k * spec.d
        ach = ops / (a_ms * 1e-3) / 1e12
        return {"value": T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "u4+i8",
                "config": {"workload": "gmm1m_d768_k1000_lvq4", "N": spec.n, "d": spec.d, "k": k, "iters": T,
                           "formats": ["lvq4"]},
                "distances_per_s": (T + 1) * spec.n * k * K / elapsed,
                "partition_cost": {"lvq4": float(out["lvq4"].item())},
                "roofline": {"bound": "mfma", "kernel": "assign_i8_kernel<lvq4>", "achieved": ach,
                             "peak": PEAK["int8_mfma_tops"], "unit": "TOP/s",
                             "frac": ach / PEAK["int8_mfma_tops"], "traffic": None, "avg_launch_ms": a_ms},
                "stages": {"lvq4": stage_summary(s)}}

    return step, finish, None, quality


def workload_hier(cfg, torch, km, args):
    """Hierarchical k-means (measurement only) on the 10M x 1024 mixture with the
    paper's k = 4 sqrt(N) = 12649 (Table 7): MESO (round(sqrt(k)) = 112 centroids)
    and FINE phases of 10 Lloyd iterations each, no refinement, once on the fp32
    vectors and once on their SQ8 codes (quantisation inside the step)."""
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    import math
    import synth
    k = int(round(4 * math.sqrt(spec.n)))
    Tm = Tf = 10
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    P32 = km.points_f32(X)
    kmeso = int(np.floor(np.sqrt(k) + 0.5))
    init = synth.init_indices(spec.n, kmeso)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    res = {}

    def step(timer):
        st32, st8 = km.KmFitStats(), km.KmFitStats()
        C, a, kf, J, ph, am = km.kmeans_fit_hier(P32, k, init, Tm, Tf, 0, stats=st32, phases=True, meso=True)
        codes, _ = km.quantize_sq8(X)
        C8, a8, kf8, J8, ph8 = km.kmeans_fit_hier(km.points_sq8(codes), k, init, Tm, Tf, 0, stats=st8, phases=True)
        if timer is not None:
            timer.add("f32", st32)
            timer.add("sq8", st8)
            res.update(ph32=ph, ph8=ph8, kf=kf, am=am)
        return {"f32": a, "sq8": a8}, J

    def finish(out, timer, elapsed, K):
        s = timer.stats["f32"]
        n_i = torch.bincount(res["am"].long(), minlength=kmeso).cpu().numpy().astype(np.float64)
        flop_pass_meso = 2.0 * spec.n * kmeso * spec.d
        flop_pass_fine = 2.0 * spec.d * float((n_i * res["kf"]).sum())
        flop = K * ((Tm + 1) * flop_pass_meso + (Tf + 1) * flop_pass_fine)
        ach = flop / (s["assign_ms"] * 1e-3) / 1e12
        return {"metric": "hierarchical k-means fits/s (build time of Table 7)", "value": 2 * K / elapsed,
                "unit": "fits/s", "dtype": "f32+i8",
                "config": {"workload": f"gmm{spec.n // 1000000}m_d{spec.d}_k{k}_hier_f32_sq8", "N": spec.n,
                           "d": spec.d, "k": k, "k_meso": kmeso, "iters_meso": Tm, "iters_fine": Tf,
                           "iters_refine": 0, "formats": ["f32", "sq8"]},
                "ms_per_fit": {"f32": float(res["ph32"].sum()), "sq8": float(res["ph8"].sum())},
                "phase_ms": {"f32": {"meso": res["ph32"][0], "fine": res["ph32"][1]},
                             "sq8": {"meso": res["ph8"][0], "fine": res["ph8"][1]}},
                "roofline": {"bound": "mfma", "kernel": "assign_f32_kernel (meso launches and segmented fine launches)",
                             "achieved": ach, "peak": PEAK["fp32_mfma_tflops"], "unit": "TFLOP/s",
                             "frac": ach / PEAK["fp32_mfma_tflops"], "traffic": None,
                             "algorithmic_flop_per_fit": flop / K},
                "stages": {"f32": stage_summary(s), "sq8": stage_summary(timer.stats["sq8"])}}

    def quality(out):
        q = {f: partition_stats(km, X, out[f], mu) for f in ("f32", "sq8")}
        q["objective_ratio_sq8_vs_f32"] = q["sq8"]["cost"] / q["f32"]["cost"]
        # vanilla Lloyd at the same k: one timed pass and update, scaled to 10 iterations
        log("quality: one vanilla fp32 pass at full k (outside the timed region)")
        C = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
        C.copy_(mu)
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
        q["speedup_vs_vanilla_f32"] = vanilla_ms / float(res["ph32"].sum())
        return q

    return step, finish, None, quality


def workload_pruned(cfg, torch, km, args):
    """The 1M x 768, k=1000 mixture under a random rotation, clustered with dimension
    pruning in every assignment pass after the first (SuperKMeans with the ADSampling
    test, eps0 = 2.1, d' = 96), as fp32 vectors and as SQ8 codes of the rotated
    vectors.  One step: rotation (projection with an orthogonal matrix), pruned fp32
    fit, SQ8 encode, pruned SQ8 fit, full-precision partition costs."""
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T = cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    R = torch.from_numpy(synth.random_rotation(spec.d, 11)).cuda()
    zero = torch.zeros(spec.d, dtype=torch.float32, device="cuda")
    Y = torch.empty_like(X)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")
    res = {}

    def step(timer):
        km.pca_project(X, zero, R, out=Y)
        st32, st8 = km.KmFitStats(), km.KmFitStats()
        C, a, J, c32 = km.kmeans_fit_pruned(km.points_f32(Y), k, T, idx, stats=st32, counters=True)
        codes, _ = km.quantize_sq8(Y)
        C8, a8, J8, c8 = km.kmeans_fit_pruned(km.points_sq8(codes), k, T, idx, stats=st8, counters=True)
        costs = {}
        for name, aa in (("f32", a), ("sq8", a8)):  # rotation keeps distances: cost on the raw rows
            km.kmeans_update(P32, aa, mu, km.KM_EMPTY_KEEP, counts=False)
            costs[name] = km.kmeans_cost(X, mu, aa)
        if timer is not None:
            timer.add("f32", st32)
            timer.add("sq8", st8)
            res.update(c32=c32, c8=c8, codes=codes)
        return {"a": a, "a8": a8, "costs": costs}, J

    def finish(out, timer, elapsed, K):
        s32, s8 = timer.stats["f32"], timer.stats["sq8"]
        pruned_passes = T  # per fit, after the full first pass

        def frac(c):
            c = c.astype(np.float64)
            return {"front_pass": c[1] / max(1.0, c[0]), "full_distance": c[2] / max(1.0, c[0]),
                    "candidates_tested_per_pass": c[0] / pruned_passes}
        return {"value": 2 * T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "f32+i8",
                "config": {"workload": f"gmm{spec.n // 1000000}m_d{spec.d}_k{k}_pruned_f32_sq8", "N": spec.n,
                           "d": spec.d, "k": k, "iters": T, "formats": ["f32", "sq8"], "eps0": 2.1,
                           "d_front": 32 * ((spec.d + 255) // 256), "rotation": "random orthogonal"},
                "partition_cost": {f: float(v.item()) for f, v in out["costs"].items()},
                "survivors": {"f32": frac(res["c32"]), "sq8": frac(res["c8"])},
                "stages": {"f32": stage_summary(s32), "sq8": stage_summary(s8)}}

    def quality(out):
        log("quality: exact fp32 and SQ8 fits on the rotated rows (outside the timed region)")
        st, st8 = km.KmFitStats(), km.KmFitStats()
        _, a_ex, _ = km.kmeans_fit(km.points_f32(Y), k, T, idx, objective=False, stats=st)
        _, a8_ex, _ = km.kmeans_fit(km.points_sq8(res["codes"]), k, T, idx, objective=False, stats=st8)
        q = {"f32_exact": partition_stats(km, X, a_ex, mu), "sq8_exact": partition_stats(km, X, a8_ex, mu),
             "f32_pruned": partition_stats(km, X, out["a"], mu), "sq8_pruned": partition_stats(km, X, out["a8"], mu)}
        q["objective_ratio_f32_pruned_vs_exact"] = q["f32_pruned"]["cost"] / q["f32_exact"]["cost"]
        q["objective_ratio_sq8_pruned_vs_f32_exact"] = q["sq8_pruned"]["cost"] / q["f32_exact"]["cost"]
        q["exact_assign_ms_per_pass"] = {"f32": st.assign_ms / st.assign_passes,
                                         "sq8": st8.assign_ms / st8.assign_passes}
        return q

    return step, finish, None, quality


def workload_sign1(cfg, torch, km, args):
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T = cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        bits, m, alpha, _ = km.quantize_sign1(X)
        P = km.points_sign1(bits, alpha, m, spec.d)
        st = km.KmFitStats()
        C, a, J = km.kmeans_fit(P, k, T, idx, stats=st)
        km.kmeans_update(P32, a, mu, km.KM_EMPTY_KEEP, counts=False)
        cost = km.kmeans_cost(X, mu, a)
        if timer is not None:
            timer.add("sign1", st)
        return {"sign1": cost, "a": a}, J

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "sign1", out["a"])

    def finish(out, timer, elapsed, K):
        s = timer.stats["sign1"]
        a_ms = s["assign_ms"] / s["assign_passes"]
        ops = 2.0 * spec.n * k * spec.d
        ach = ops / (a_ms * 1e-3) / 1e12
        return {"value": T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "i8",
                "config": {"workload": cfg["name"], "N": spec.n, "d": spec.d, "k": k, "iters": T,
                           "formats": ["sign1"]},
                "distances_per_s": (T + 1) * spec.n * k * K / elapsed,
                "partition_cost": {"sign1": float(out["sign1"].item())},
                "roofline": {"bound": "mfma", "kernel": "assign_bits_kernel<sign1>", "achieved": ach,
                             "peak": PEAK["int8_mfma_tops"], "unit": "TOP/s", "frac": ach / PEAK["int8_mfma_tops"],
                             "traffic": None, "avg_launch_ms": a_ms},
                "stages": {"sign1": stage_summary(s)}}

    return step, finish, None, quality


def workload_rabitq(cfg, torch, km, args):
    """The 1M x 1024, k=1024 mixture through the paper's RabitQ pipeline: centre, random
    rotation, 1-bit codes; SQ4 centroid codes; last update from the rotated raw rows."""
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T = cfg["k"], cfg["iters"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    rot = torch.from_numpy(synth.random_rotation(spec.d)).cuda()
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        bits, m, alpha, Y = km.rabitq_encode(X, rot, want_rotated=True)
        st = km.KmFitStats()
        C, a, J = km.kmeans_fit(km.points_rabitq(bits, alpha, spec.d, raw=Y), k, T, idx, stats=st)
        km.kmeans_update(km.points_f32(X), a, mu, km.KM_EMPTY_KEEP, counts=False)
        cost = km.kmeans_cost(X, mu, a)
        if timer is not None:
            timer.add("rabitq", st)
        return {"rabitq": cost, "a": a, "bits": bits, "alpha": alpha}, J

    def finish(out, timer, elapsed, K):
        s = timer.stats["rabitq"]
        a_ms = s["assign_ms"] / s["assign_passes"]
        ops = 2.0 * spec.n * k * spec.d
        ach = ops / (a_ms * 1e-3) / 1e12
        return {"value": T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "i8",
                "config": {"workload": "gmm1m_d1024_k1024_rabitq", "N": spec.n, "d": spec.d, "k": k, "iters": T,
                           "formats": ["rabitq"], "raw_last_update": True},
                "distances_per_s": (T + 1) * spec.n * k * K / elapsed,
                "partition_cost": {"rabitq": float(out["rabitq"].item())},
                "roofline": {"bound": "mfma", "kernel": "assign_bits_kernel<rabitq>", "achieved": ach,
                             "peak": PEAK["int8_mfma_tops"], "unit": "TOP/s", "frac": ach / PEAK["int8_mfma_tops"],
                             "traffic": None, "avg_launch_ms": a_ms},
                "stages": {"rabitq": stage_summary(s)}}

    def quality(out):
        q = quality_vs_f32(km, X, k, T, idx, mu, "rabitq", out["a"])
        _, a2, _ = km.kmeans_fit(km.points_rabitq(out["bits"], out["alpha"], spec.d), k, T, idx, objective=False)
        q["rabitq_codes_only"] = partition_stats(km, X, a2, mu)
        q["objective_ratio_rabitq_codes_only_vs_f32"] = q["rabitq_codes_only"]["cost"] / q["f32"]["cost"]
        return q

    return step, finish, None, quality


def workload_pca(cfg, torch, km, args):
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T, dout = cfg["k"], cfg["iters"], cfg["d_out"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    Y = torch.empty((spec.n, dout), dtype=torch.float32, device="cuda")
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        mean, cov = km.pca_fit_cov(X)
        # host eigensolve of the d x d covariance (harness step)
        w, V = np.linalg.eigh(cov.double().cpu().numpy())
        order = np.argsort(w)[::-1][:dout]
        W = torch.from_numpy(np.ascontiguousarray(V[:, order], dtype=np.float32)).cuda()
        km.pca_project(X, mean, W, out=Y)
        st = km.KmFitStats()
        C, a, J = km.kmeans_fit(km.points_f32(Y), k, T, idx, stats=st)
        if timer is not None:
            timer.add("pca", st)
        return {"a": a}, J

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "pca", out["a"])

    def finish(out, timer, elapsed, K):
        s = timer.stats["pca"]
        a_ms = s["assign_ms"] / s["assign_passes"]
        flop = 2.0 * spec.n * k * dout
        ach = flop / (a_ms * 1e-3) / 1e12
        return {"value": T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "f32",
                "config": {"workload": cfg["name"], "N": spec.n, "d": spec.d, "d_out": dout, "k": k, "iters": T},
                "distances_per_s": (T + 1) * spec.n * k * K / elapsed,
                "roofline": {"bound": "mfma", "kernel": "assign_f32_kernel", "achieved": ach,
                             "peak": PEAK["fp32_mfma_tflops"], "unit": "TFLOP/s",
                             "frac": ach / PEAK["fp32_mfma_tflops"], "traffic": None, "avg_launch_ms": a_ms},
                "stages": {"pca": stage_summary(s)}}

    return step, finish, None, quality


def workload_hybrid(cfg, torch, km, args):
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T, d0 = cfg["k"], cfg["iters"], cfg["d_front"]
    import synth
    log(f"generating {spec.n} x {spec.d} mixture")
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P32 = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        bits, m, alpha, front = km.quantize_sign1(X, d_front=d0, want_front=True)
        P = km.points_hybrid(front, bits, alpha, m, spec.d)
        st = km.KmFitStats()
        C, a, J = km.kmeans_fit(P, k, T, idx, stats=st)
        del front
        km.kmeans_update(P32, a, mu, km.KM_EMPTY_KEEP, counts=False)
        cost = km.kmeans_cost(X, mu, a)
        if timer is not None:
            timer.add("hybrid", st)
        return {"hybrid": cost, "a": a}, J

    def quality(out):
        return quality_vs_f32(km, X, k, T, idx, mu, "hybrid", out["a"])

    def finish(out, timer, elapsed, K):
        s = timer.stats["hybrid"]
        a_ms = s["assign_ms"] / s["assign_passes"]
        flop = 2.0 * spec.n * k * d0
        ach = flop / (a_ms * 1e-3) / 1e12
        return {"value": T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "f32+i8",
                "config": {"workload": cfg["name"], "N": spec.n, "d": spec.d, "d_front": d0, "k": k, "iters": T},
                "distances_per_s": (T + 1) * spec.n * k * K / elapsed,
                "partition_cost": {"hybrid": float(out["hybrid"].item())},
                "roofline": {"bound": "mfma", "kernel": "assign_kernel<hybrid>", "achieved_front": ach,
                             "peak": PEAK["fp32_mfma_tflops"], "unit": "TFLOP/s",
                             "frac": ach / PEAK["fp32_mfma_tflops"], "traffic": None, "avg_launch_ms": a_ms},
                "stages": {"hybrid": stage_summary(s)}}

    return step, finish, None, quality


def workload_c1(cfg, torch, km, args):
    spec = cfg["spec"] if args.n is None else cfg["spec"].with_n(args.n)
    k, T = cfg["k"], cfg["iters"]
    import synth
    X = upload(spec, torch)
    idx = synth.init_indices(spec.n, k)
    P = km.points_f32(X)
    mu = torch.empty((k, spec.d), dtype=torch.float32, device="cuda")

    def step(timer):
        st = km.KmFitStats()
        C, a, J = km.kmeans_fit(P, k, T, idx, stats=st)
        if timer is not None:
            timer.add("f32", st)
        return {"a": a}, J

    def quality(out):
        return {"f32": partition_stats(km, X, out["a"], mu)}

    def finish(out, timer, elapsed, K):
        s = timer.stats["f32"]
        return {"value": T * K / elapsed, "unit": "Lloyd iters/s", "dtype": "f32",
                "config": {"workload": cfg["name"], "N": spec.n, "d": spec.d, "k": k, "iters": T},
                "distances_per_s": (T + 1) * spec.n * k * K / elapsed, "stages": {"f32": stage_summary(s)}}

    return step, finish, None, quality


WORKLOADS = {1: workload_c1, 2: workload_c2, 3: workload_sign1, 4: workload_pca, 5: workload_hybrid,
             6: workload_bf16, 7: workload_rabitq, 8: workload_lvq4, 9: workload_hier,
             10: workload_pruned}
CONFIG_OF = {6: 2, 7: 3, 8: 2, 9: 4, 10: 2}  # measurement-only workloads and the configuration whose data they use


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=2, choices=sorted(WORKLOADS))
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

    if args.copy_probe:
        copy_probe(torch)
    cfg = synth.config(CONFIG_OF.get(args.workload, args.workload))
    step, finish, cpu_baseline, quality = WORKLOADS[args.workload](cfg, torch, km, args)
    for i in range(args.warmup):
        step(None)
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")
    timer = Timer()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    out = None
    for i in range(args.steps):
        out, _ = step(timer)
        log(f"timed step {i + 1}/{args.steps} issued")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    res = finish(out, timer, elapsed, args.steps)
    line = {"metric": res.pop("metric", METRIC), "value": res.pop("value"), "unit": res.pop("unit"), "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": res.pop("dtype"),
            "data": "synthetic (seeded Gaussian mixture shaped like the paper's embedding workloads)",
            "config": res.pop("config")}
    line.update(res)
    if quality is not None and not args.no_quality:
        line["quality"] = quality(out)
    if cpu_baseline is not None and not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        line["cpu_baseline"] = cpu_baseline()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
