#!/usr/bin/env python3
"""Benchmark of the kernel-SVM hot path on one MI355X.

One step = one complete pass of the method on the C3 workload (binary
C-SVC, RBF, dense n = 100000, d = 128, x = y*0.2*1 + N(0, I), C = 1,
gamma = 1/128, tol = 1e-3, working set q = 16): feature store and norms,
the working-set iterations to the KKT tolerance, the final recompute of the
responses, bias and model extraction, then the decision function on the
20000 test points.  Inputs are resident in HBM (torch tensors) before the
timed region starts.  `cpu_baseline` trains the same workload with the CPU
oracle to the same tolerance on the host's cores (all threads), and times a
bounded single-thread sample of its pair steps.

Prints one JSON line.  `value` is kernel rows per second: rows K(x_s, X)
(length n) evaluated by the working-set iterations, over the wall time of
the timed steps.  `roofline` is for the row/update kernel (k_rows), timed
with HIP events on the stream it runs on.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("train time to KKT tol 1e-3; kernel rows/s and % of HBM/MFMA peak")
HBM_PEAK_GBS = 8000.0
MFMA_FP32_PEAK_TFS = 157.3  # dense fp32 matrix-core peak of the MI355X


def log(msg: str) -> None:
    print("[bench] " + msg, file=sys.stderr, flush=True)


def row_bytes_per_launch(n: int, d: int, svr: bool) -> int:
    """Algorithmic HBM bytes of one k_rows launch (dense layout): per row the
    features (4d), the squared norm (4), F read and written (16), one state
    byte per variable and, for eps-SVR, the fp32 target (4)."""
    per = 4 * d + 4 + 16 + (2 + 4 if svr else 1)
    return n * per


KERNEL_SOURCES = ("paper_1706_05544_amd/csrc/rows.hip",
                  "paper_1706_05544_amd/csrc/rowtile.hpp",
                  "paper_1706_05544_amd/csrc/device.hpp",
                  "paper_1706_05544_amd/csrc/common.hpp")


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per k_rows launch from the committed counter runs
    (FETCH_SIZE and WRITE_SIZE, scaled by a copy of known size), or None
    when the kernel sources changed since they were taken."""
    path = os.path.join(ROOT, "profiles", "k_rows_%s_hbm_counters.md"
                        % workload)
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(("#", "|", " ", "`")):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("source_sha256") != kernel_source_hash():
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, kernel: int, gamma: float, degree: int, coef0: float,
                 gpu_train_ms: float, full: bool, sample_s: float) -> dict:
    """The oracle (untuned: fp64 maximal-violating-pair SMO, 2 kernel rows
    per pair step) on the GPU host's cores.

    full: the whole training to tol from alpha = 0 with all threads (the
    metric's train time), then its decision values on the test set;
    otherwise a bounded number of pair steps from alpha = 0 (the rate only).
    Either way also a bounded single-thread sample of pair steps."""
    import numpy as np

    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    if threads <= 0:
        threads = len(os.sched_getaffinity(0))
    X = oracle.Matrix(w.X)
    N = oracle.num_vars(w.type, w.n)

    def params(t):
        return oracle.Params(w.type, C=w.C, eps=w.eps, gamma=gamma, tol=w.tol,
                             threads=t, kernel=kernel, degree=degree,
                             coef0=coef0)

    def steps_for(t, seconds):  # pair steps that take about `seconds`
        t0 = time.perf_counter()
        oracle.solve(X, w.y, params(t), np.zeros(N), np.zeros(w.n),
                     max_steps=10)
        dt = time.perf_counter() - t0
        return max(10, int(10 * seconds / max(dt, 1e-6)))

    out = {"unit": "kernel rows/s", "cores": threads, "threads": threads,
           "kind": "oracle", "cpu_model": cpu_model(),
           "nproc": os.cpu_count()}
    if full:
        t0 = time.perf_counter()
        r = oracle.train(X, w.y, params(threads))
        train_s = time.perf_counter() - t0
        t0 = time.perf_counter()
        oracle.model_decision(X, w.y, params(threads), r, w.Xt, threads)
        pred_s = time.perf_counter() - t0
        log("cpu baseline: oracle training %d pair steps in %.1f s, "
            "prediction %.1f s" % (r.iters, train_s, pred_s))
        out.update({
            "value": 2 * r.iters / train_s,
            "train_s_to_tol": train_s,
            "iters": r.iters,
            "dual_obj": r.obj,
            "gap": r.gap,
            "predict_s": pred_s,
            "gpu_train_ms_device": gpu_train_ms,
            "train_speedup_gpu": 1e3 * train_s / gpu_train_ms,
            "sample": "the whole training of the %s workload (%d x %d) to "
                      "tol %g from alpha=0 (%d pair steps, 2 kernel rows "
                      "each, fp64, %d threads, %.1f s), then the decision "
                      "values of its %d test points (%.1f s); value = "
                      "kernel rows per second of that training"
                      % (w.name, w.n, w.d, w.tol, r.iters, threads, train_s,
                         w.Xt.shape[0], pred_s)})
    else:
        k = steps_for(threads, sample_s)
        t0 = time.perf_counter()
        r = oracle.solve(X, w.y, params(threads), np.zeros(N), np.zeros(w.n),
                         max_steps=k)
        dt = time.perf_counter() - t0
        log("cpu baseline: %d oracle steps in %.1f s" % (r.iters, dt))
        out.update({
            "value": 2 * r.iters / dt,
            "s_per_step": dt / r.iters,
            "gap_reached": r.gap,
            "sample": "%d maximal-violating-pair SMO steps from alpha=0 on "
                      "the full %s training set (%d x %d), 2 kernel rows of "
                      "length n per step, fp64, %d threads, %.1f s (the "
                      "whole training does not fit a bounded run)"
                      % (r.iters, w.name, w.n, w.d, threads, dt)})
    # one thread: a bounded sample of pair steps (a rate; the train time at
    # one thread is extrapolated from it and labelled so)
    k1 = steps_for(1, sample_s)
    t0 = time.perf_counter()
    r1 = oracle.solve(X, w.y, params(1), np.zeros(N), np.zeros(w.n),
                      max_steps=k1)
    dt1 = time.perf_counter() - t0
    single = {"threads": 1, "steps": r1.iters, "seconds": dt1,
              "s_per_step": dt1 / r1.iters,
              "kernel_rows_per_s": 2 * r1.iters / dt1}
    if full:
        single["train_s_to_tol_extrapolated"] = out["iters"] * dt1 / r1.iters
    out["single_thread"] = single
    log("cpu baseline: 1 thread, %d steps in %.1f s" % (r1.iters, dt1))
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="C3")
    ap.add_argument("--n", type=int, default=None,
                    help="override the workload's training-set size")
    ap.add_argument("--layout", default=None,
                    help="feature layout of workloads that offer both "
                         "(C4: dense or csr)")
    ap.add_argument("--working-set", type=int, default=16)
    ap.add_argument("--kernel", default="rbf",
                    choices=["linear", "poly", "rbf", "sigmoid"],
                    help="kernel function (e1071 parameterisation)")
    ap.add_argument("--gamma", type=float, default=None,
                    help="kernel gamma (default: the workload's)")
    ap.add_argument("--degree", type=int, default=3)
    ap.add_argument("--coef0", type=float, default=0.0)
    ap.add_argument("--cv", type=int, default=0,
                    help="K > 1: one step is a K-fold cross-validation of "
                         "the training set instead of a training + "
                         "prediction")
    ap.add_argument("--lockstep", type=int, default=0,
                    help="P > 1: one-vs-rest classes and cross-validation "
                         "folds train P at a time in lockstep (one pass "
                         "over X serves P working sets; no row cache)")
    ap.add_argument("--fused", type=int, default=0, choices=[0, 1],
                    help="1: every outer iteration as one launch (dense, "
                         "q <= 16, no row cache); 0: selection and row "
                         "update as two launches")
    ap.add_argument("--scale", action="store_true",
                    help="standardise the features (and eps-SVR targets)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="length of each bounded oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--time-select", action="store_true",
                    help="also time the select/solve kernel with events in "
                         "the sampled iterations (costs the loop ~5 us per "
                         "timed launch; reported under 'iteration')")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain device copy of 256 MiB (the "
                         "reference kernel for the HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: the library runs on one GPU; --gpus %d is not "
              "supported (the training rows would be sharded over GPUs, "
              "with one exchange of selection candidates per iteration)"
              % args.gpus, file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_1706_05544_amd import native as nv
    from paper_1706_05544_amd import workloads

    nv.load()
    w = workloads.make(args.workload, n=args.n,
                       **({"layout": args.layout} if args.layout else {}))
    if w.type != workloads.C_SVC and w.type != workloads.EPS_SVR:
        raise SystemExit("unsupported workload")
    log("workload %s: n=%d d=%d n_test=%d" % (w.name, w.n, w.d,
                                             w.Xt.shape[0]))
    dev = torch.device("cuda:0")

    def to_device(A):
        if hasattr(A, "indptr"):  # scipy CSR -> torch sparse CSR in HBM
            return torch.sparse_csr_tensor(
                torch.from_numpy(A.indptr.astype(np.int64)),
                torch.from_numpy(A.indices.astype(np.int64)),
                torch.from_numpy(A.data.astype(np.float32)), size=A.shape,
                device=dev)
        return torch.from_numpy(A).to(dev)

    X = to_device(w.X)
    y = torch.from_numpy(w.y).to(dev)
    Xt = to_device(w.Xt)
    torch.cuda.synchronize()
    kernel = {"linear": nv.SVM_KERNEL_LINEAR, "poly": nv.SVM_KERNEL_POLY,
              "rbf": nv.SVM_KERNEL_RBF,
              "sigmoid": nv.SVM_KERNEL_SIGMOID}[args.kernel]
    gamma = args.gamma if args.gamma is not None else w.gamma
    kw = dict(type=w.type, C=w.C, epsilon=w.eps, gamma=gamma, tol=w.tol,
              working_set=args.working_set, kernel=kernel,
              degree=args.degree, coef0=args.coef0,
              scale=1 if args.scale else 0, fused=args.fused)
    multi = w.n_classes > 2
    # lockstep applies to one-vs-rest classes and cross-validation folds
    lock = args.lockstep if (args.lockstep > 1 and (multi or args.cv > 1)) \
        else 0
    if lock:
        kw["lockstep"] = lock
    if multi:
        kw.pop("type")
        kw.pop("epsilon")

    class CvRun:
        """One cross-validation in the shape of a model's statistics."""
        n_outputs = 1

        def __init__(self, st, ms):
            self.st, self.ms = st, ms

        def info(self, c=0):
            st = self.st
            return {"train_ms": self.ms, "iters": st["iters"],
                    "kernel_rows": st["kernel_rows"],
                    "row_kernel_ms": st["row_kernel_ms"],
                    "row_kernel_launches": st["row_kernel_launches"],
                    "row_kernel_bytes": st["row_kernel_bytes"],
                    "cached_kernel_ms": 0.0, "cached_kernel_launches": 0,
                    "cached_kernel_bytes": 0.0, "cache_hits": 0,
                    "cache_fills": 0, "n_sv_output": 0, "dual_obj": 0.0,
                    "gap": 0.0, "select_kernel_ms": 0.0,
                    "select_kernel_launches": 0}

    y_host = w.y
    cv_stats = {}

    def step(profile: int):
        if args.cv > 1:
            t = time.perf_counter()
            if multi:
                D, st = nv.svm_cross_validate(X, labels=y_host,
                                              n_classes=w.n_classes, k=args.cv,
                                              profile=profile, **kw)
            else:
                D, st = nv.svm_cross_validate(X, y_host, k=args.cv,
                                              profile=profile, **kw)
            t1 = time.perf_counter()
            cv_stats.update(st)
            return CvRun(st, 1e3 * (t1 - t)), torch.from_numpy(D), t1
        if multi:
            m = nv.svm_train_ovr(X, y, w.n_classes, profile=profile, **kw)
        else:
            m = nv.svm_train(X, y, profile=profile, **kw)
        t1 = time.perf_counter()
        D = nv.svm_predict(m, Xt)
        return m, D, t1

    def infos_of(m):
        return [m.info(c) for c in range(m.n_outputs)]

    if args.copy_calibration:
        src = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device=dev)
        src.fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("copy calibration: 3 copies of 256 MiB")

    for i in range(args.warmup):
        m, _, _ = step(0)
        log("warmup %d: iters=%d" % (i, m.info()["iters"]))

    infos = []
    pred_s = 0.0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ts = time.perf_counter()
        m, D, t1 = step(2 if args.time_select else 1)
        torch.cuda.synchronize()
        te = time.perf_counter()
        per = infos_of(m)
        info = dict(per[0])
        for k in ("train_ms", "iters", "kernel_rows", "row_kernel_ms",
                  "row_kernel_launches", "row_kernel_bytes",
                  "cached_kernel_ms", "cached_kernel_launches",
                  "cached_kernel_bytes", "cache_hits", "cache_fills",
                  "n_sv_output", "select_kernel_ms",
                  "select_kernel_launches"):
            info[k] = sum(x[k] for x in per)
        info["dual_obj"] = sum(x["dual_obj"] for x in per)
        info["gap"] = max(x["gap"] for x in per)
        infos.append(info)
        pred_s += te - t1
        log("step %d: %.1f ms (train %.1f ms device, iters %d, rows %d)"
            % (i, 1e3 * (te - ts), info["train_ms"], info["iters"],
               info["kernel_rows"]))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    rows = sum(i["kernel_rows"] for i in infos)
    # roofline of the row/update kernel over its launches that compute the
    # rows from X (launches served from the row cache are reported apart):
    # algorithmic bytes (features, norm, F, state; plus the rows written to
    # the cache) over the kernel's own time
    launches = sum(i["row_kernel_launches"] for i in infos)
    row_ms = sum(i["row_kernel_ms"] for i in infos)
    row_bytes = sum(i["row_kernel_bytes"] for i in infos)
    avg_ms = row_ms / max(launches, 1)
    bytes_launch = row_bytes / max(launches, 1)
    achieved = row_bytes / (row_ms * 1e-3) / 1e9 if row_ms > 0 else 0.0
    lock_tflops = (launches * 2.0 * w.n * w.d * 16 / (row_ms * 1e-3) / 1e12
                   if row_ms > 0 else 0.0)
    s_launches = sum(i["select_kernel_launches"] for i in infos)
    s_ms = sum(i["select_kernel_ms"] for i in infos)
    c_launches = sum(i["cached_kernel_launches"] for i in infos)
    c_ms = sum(i["cached_kernel_ms"] for i in infos)
    c_bytes = sum(i["cached_kernel_bytes"] for i in infos)

    last = infos[-1]
    Dn = D.cpu().numpy()
    if args.cv > 1:
        quality = ({"cv_accuracy": cv_stats["accuracy"]}
                   if w.type == workloads.C_SVC else
                   {"cv_mse": cv_stats["mse"], "cv_scc": cv_stats["scc"]})
    elif multi:
        acc = float(np.mean(np.argmax(Dn, axis=1) == w.yt))
        quality = {"test_accuracy": acc}
    elif w.type == workloads.C_SVC:
        acc = float(np.mean(np.where(Dn >= 0, 1.0, -1.0) == w.yt))
        quality = {"test_accuracy": acc}
    else:
        quality = {"test_mse": float(np.mean((Dn - w.yt) ** 2))}

    kernel_desc = {"rbf": "RBF", "linear": "linear",
                   "poly": "polynomial (degree %d, coef0 %g)"
                           % (args.degree, args.coef0),
                   "sigmoid": "sigmoid (coef0 %g)" % args.coef0}[args.kernel]
    out = {
        "metric": METRIC,
        "value": rows / wall,
        "unit": "kernel rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * wall / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s: %s %s, %s n=%d d=%d, C=%g, gamma=%g, "
                        "tol=%g, q=%d; %s"
                        % (w.name, ("one-vs-rest %d-class C-SVC" % w.n_classes)
                           if multi else
                           ("C-SVC" if w.type == 0 else "eps-SVR"),
                           kernel_desc,
                           ("CSR (%d nonzeros)" % w.X.nnz)
                           if hasattr(w.X, "indptr") else "dense",
                           w.n, w.d, w.C, gamma, w.tol, args.working_set,
                           ("%d-fold cross-validation" % args.cv)
                           if args.cv > 1 else
                           "predict %d points" % w.Xt.shape[0])
                        + ("; features standardised" if args.scale else "")
                        + ("; %d problems in lockstep" % lock
                           if lock else ""),
            "kernel": args.kernel,
            "n": w.n, "d": w.d, "n_test": int(w.Xt.shape[0]),
            "working_set": args.working_set,
        },
        "train_ms_device": sum(i["train_ms"] for i in infos) / len(infos),
        "predict_ms_wall": 1e3 * pred_s / len(infos),
        "iters": last["iters"],
        "n_sv": last["n_sv_output"],
        "dual_obj": last["dual_obj"],
        "gap": last["gap"],
        **quality,
        "roofline": {
            "kernel": "k_rows (kernel rows + gradient update + candidates)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": measured_traffic(w.name),
            "avg_launch_us": 1e3 * avg_ms,
            "bytes_per_launch": bytes_launch,
            "bytes_per_launch_no_cache_fill": (
                row_bytes_per_launch(w.n, w.d, w.type == workloads.EPS_SVR)
                if not hasattr(w.X, "indptr") else None),
            "launches_timed": launches,
        } if not lock else {
            # k_lock: each pass computes the dot products of every row with
            # the P working sets on the matrix cores; the statistics split
            # each pass's time over its problems, so the sum over problems
            # of 2 n d 16 flops over the summed time is the pass's rate
            "kernel": "k_lock (P working sets over one pass of X)",
            "bound": "mfma",
            "achieved": lock_tflops,
            "peak": MFMA_FP32_PEAK_TFS,
            "unit": "TFLOP/s",
            "frac": lock_tflops / MFMA_FP32_PEAK_TFS,
            "traffic": None,
            "hbm_GBps": achieved,
            "problem_launches_timed": launches,
            "us_per_problem_launch": 1e3 * avg_ms,
        },
        # the per-iteration chain: device time per outer iteration; with
        # --time-select the single-block select/solve kernel (latency-bound:
        # merge of the block records, K_BB, subproblem) and the row kernel
        # of the same timed iterations, computed or cached
        "iteration": {
            "us_per_iteration": 1e3 * sum(i["train_ms"] for i in infos)
                                / max(sum(i["iters"] for i in infos), 1),
            "k_select_avg_us": 1e3 * s_ms / s_launches if s_launches else None,
            "k_rows_avg_us": (1e3 * (row_ms + c_ms) / (launches + c_launches)
                              if s_launches and launches + c_launches
                              else None),
            "launches_timed": s_launches,
        },
        "row_cache": {
            "rows_served": last["cache_hits"],
            "rows_filled": last["cache_fills"],
            "rows_used": last["kernel_rows"],
            "cached_launches": c_launches,
            "cached_avg_launch_us": 1e3 * c_ms / max(c_launches, 1),
            "cached_GBps": c_bytes / (c_ms * 1e-3) / 1e9 if c_ms > 0 else 0.0,
        },
    }
    if not args.no_cpu_baseline:
        # the whole training where the oracle finishes it in about a
        # minute of the host's cores (the dense C-SVC workloads of up to
        # 100000 x 128; not the one-vs-rest, eps-SVR or 2M-row workloads)
        full = (not multi and args.cv <= 1 and args.kernel == "rbf"
                and w.type == workloads.C_SVC and w.n * w.d <= 1.3e7
                and not hasattr(w.X, "indptr") and not args.scale)
        out["cpu_baseline"] = cpu_baseline(
            w, kernel, gamma, args.degree, args.coef0,
            out["train_ms_device"], full, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
