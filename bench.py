"""Benchmark of the LS-SVM training hot path on one MI355X.

One step = one full training (layout, q-vector, right-hand side, CG with one
implicit Q~ product per iteration, bias) plus the prediction of 1024 held-out
points, on synthetic data already resident in HBM. Default workload: cubic
polynomial kernel, fp32, n = 32768 points x d = 4096 features, C = 1,
eps = 1e-5.

Prints one JSON line. `value` is the whole-step throughput in GFLOP/s with
the symmetric count N(N+1)d per implicit product (N = n - 1) plus
2 n_test n d for the prediction. `roofline` is the tile kernel's own rate:
N(N+1)d divided by its average duration, measured with HIP events recorded
on the launch stream over the even steps (`matvec_median_ms`, `matvec_cov`
over every timed product). `time_to_eps_ms` is the median over the odd
steps, which record no events (5 steps by default: 3 with product events, 2
without; `time_to_eps_timed_ms` is the median over the others); one more
training reports the true relative residual. `a5_cg_vector_step` times the CG
vector step alone (lssvm_cg_step, 11 passes of N doubles) on N = 2^26 against
the HBM peak. `cpu_baseline` times the CPU oracle's explicit row-panel product
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "implicit kernel matvec GFLOP/s (% MFMA peak); CG time-to-eps per training"
PEAK_TFLOPS = {"f32": 157.3, "f64": 78.6}      # MI355X dense matrix-core peaks
HBM_GBS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def code_only(text: str) -> str:
    """C++ source without comments, whitespace collapsed: what the compiler sees
    of it (the kernel sources hold no string literal that contains a comment
    marker)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash() -> str:
    """Hash of the tile kernel's code (tiles.h and its interface tile_args.h,
    comments left out), so a measurement stays tied to the code it measured."""
    h = hashlib.sha256()
    for f in ("tiles.h", "tile_args.h"):
        with open(os.path.join(ROOT, "paper_2202_12674_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def traffic_record(workload: str):
    """HBM bytes per implicit product (its tile launches together) from
    committed rocprofv3 counter runs, or None when missing or taken on a
    different kernel source."""
    path = os.path.join(ROOT, "profiles", f"k_tiles_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_product")


def host_facts():
    """The host CPU's model name, its logical CPUs available to this process
    and numpy's BLAS (name and version), as the oracle's timings depend on them."""
    import numpy as np
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        b = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{b.get('name')} {b.get('version')}"
    except Exception:  # noqa: BLE001
        pass
    return {"cpu_model": model, "cpus_available": len(os.sched_getaffinity(0)), "blas": blas}


def cpu_baseline(cfg, X, budget_s: float):
    """The oracle's explicit row-panel product Q~[rows] @ p on the host cores."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([t.get("num_threads", 1) for t in threadpool_info()
                       if t.get("user_api") == "blas"] or [1])
    except Exception:  # noqa: BLE001
        threads = len(os.sched_getaffinity(0))
    spec = O.KernelSpec(cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)
    N = cfg.n - 1
    p = np.random.default_rng(12345).standard_normal(N)
    X64 = X.astype(np.float64)
    panel = 256
    rows_done = 0
    t0 = time.perf_counter()
    start = 0
    while True:
        rows = np.arange(start, min(N, start + panel))
        _ = O.reduced_rows(X64, spec, cfg.C, rows) @ p
        rows_done += len(rows)
        start = (start + panel) % N
        if time.perf_counter() - t0 >= budget_s or rows_done >= N:
            break
    dt = time.perf_counter() - t0
    flops = rows_done * (N + 1) * cfg.d          # share of the symmetric count N(N+1)d
    return {"value": flops / dt / 1e9, "unit": "GFLOP/s", "cores": int(threads),
            "kind": "oracle", "host": host_facts(),
            "sample": f"{rows_done} of {N} rows of the explicit reduced matrix (fp64, "
                      f"panels of {panel}) times a vector, {dt:.1f} s"}


def a5_standalone(torch, dev, N: int, reps: int = 20):
    """The CG vector step (lssvm_cg_step: d^T q, update, direction; 8 reads and
    3 writes of N doubles) on vectors of length N, timed per step with HIP
    events on the launch stream; the state is restored between steps."""
    import paper_2202_12674_amd as P
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    x0 = torch.randn(N, dtype=torch.float64, device=dev, generator=g)
    r0 = torch.randn(N, dtype=torch.float64, device=dev, generator=g)
    d0 = torch.randn(N, dtype=torch.float64, device=dev, generator=g)
    q = d0 * torch.rand(N, dtype=torch.float64, device=dev, generator=g).add_(0.5)
    x, r, d = x0.clone(), r0.clone(), d0.clone()
    rr0 = float(r0.dot(r0))
    sc = torch.zeros(4, dtype=torch.float64, device=dev)
    ws = P.alloc_workspace(P.lib().lssvm_cg_step_workspace_bytes(N), dev)
    times = []
    for k in range(reps + 3):
        x.copy_(x0)
        r.copy_(r0)
        d.copy_(d0)
        sc[0] = rr0
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        P.cg_step(x, r, d, q, sc, workspace=ws)
        e1.record()
        e1.synchronize()
        if k >= 3:
            times.append(e0.elapsed_time(e1))
    if float(sc[1]) <= 0.0:
        raise RuntimeError("a5 measurement broke down (d^T q <= 0)")
    ms = statistics.median(times)
    nbytes = 11 * 8 * N
    return {"N": N, "ms_per_step": round(ms, 4), "bytes_per_step": nbytes,
            "achieved_GBs": round(nbytes / (ms * 1e-3) / 1e9, 1), "peak_GBs": HBM_GBS,
            "frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_GBS, 4),
            "cov": round(statistics.pstdev(times) / statistics.mean(times), 4), "reps": reps}


def cpu_phases(cfg, X, y, X_test, n_sub: int):
    """The oracle's phases (Q~ assembly, Cholesky factor + solve, CG with the
    explicit Q~, prediction) on the first n_sub points of the workload, timed
    with time.perf_counter."""
    import numpy as np
    import oracle as O
    spec = O.KernelSpec(cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)
    Xs, ys = X[:n_sub].astype(np.float64), y[:n_sub].astype(np.float64)
    out = {"sample": f"first {n_sub} points of the workload ({n_sub} x {cfg.d}, fp64), "
                     f"{len(X_test)} test points"}
    t = time.perf_counter()
    Qt, q, Qmm = O.reduced_matrix(Xs, spec, cfg.C)
    out["assembly_s"] = round(time.perf_counter() - t, 4)
    rhs = O.reduced_rhs(ys)
    t = time.perf_counter()
    O.solve_cholesky(Qt, rhs)
    out["cholesky_s"] = round(time.perf_counter() - t, 4)
    t = time.perf_counter()
    res = O.solve_cg(lambda v: O.matvec_dense(Qt, v), rhs, cfg.eps)
    out["cg_s"] = round(time.perf_counter() - t, 4)
    out["cg_iterations"] = res.iterations
    alpha, b = O.recover(res.x, ys, q, Qmm)
    t = time.perf_counter()
    O.predict(Xs, alpha, b, X_test, spec)
    out["predict_s"] = round(time.perf_counter() - t, 4)
    return out


def cpu_full(cfg, X, y, X_test):
    """The oracle's time to eps on the whole workload, every phase on the host
    cores: dense Q~ assembly (BLAS), CG with the explicit Q~ at the workload's
    eps (the same stop rule as the GPU), the recovery of alpha and b, the
    Cholesky factor and solve of the same system, and the prediction of the
    test points. Dense fp64 Q~ of the 32768-point workload is 8 GiB; run it
    where the host has room (not part of the default run)."""
    import numpy as np
    import oracle as O
    spec = O.KernelSpec(cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)
    X64, y64 = X.astype(np.float64), y.astype(np.float64)
    out = {"workload": cfg.name, "host": host_facts()}
    t0 = time.perf_counter()
    Qt, q, Qmm = O.reduced_matrix(X64, spec, cfg.C)
    out["assembly_s"] = round(time.perf_counter() - t0, 3)
    rhs = O.reduced_rhs(y64)
    t = time.perf_counter()
    res = O.solve_cg(lambda v: O.matvec_dense(Qt, v), rhs, cfg.eps, cfg.max_iter)
    alpha, b = O.recover(res.x, y64, q, Qmm)
    out["cg_s"] = round(time.perf_counter() - t, 3)
    out["cg_iterations"] = res.iterations
    out["cg_s_per_iteration"] = round(out["cg_s"] / max(1, res.n_matvec), 4)
    out["time_to_eps_s"] = round(out["assembly_s"] + out["cg_s"], 3)
    t = time.perf_counter()
    O.solve_cholesky(Qt, rhs)
    out["cholesky_s"] = round(time.perf_counter() - t, 3)
    del Qt
    t = time.perf_counter()
    O.predict(X64, alpha, b, X_test.astype(np.float64), spec)
    out["predict_s"] = round(time.perf_counter() - t, 3)
    # the oracle's CG multiplies by the assembled Q~ (2 N^2 flop, memory-bound);
    # the assembly is where it forms the kernel values the GPU forms per product
    N = cfg.n - 1
    out["dense_product_gflops"] = round(2.0 * N * N / 1e9 / out["cg_s_per_iteration"], 2)
    return out


def device_facts(torch, dev):
    p = torch.cuda.get_device_properties(dev)
    return {"name": p.name, "compute_units": p.multi_processor_count,
            "hbm_gib": round(p.total_memory / 2**30, 1),
            "arch": getattr(p, "gcnArchName", "")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="poly_f32_32768x4096")
    ap.add_argument("--n-test", type=int, default=1024)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--a5-n", type=int, default=1 << 26,
                    help="vector length of the standalone CG vector-step measurement (0: skip)")
    ap.add_argument("--cpu-phase-points", type=int, default=4096,
                    help="points of the workload for the oracle's per-phase timing (0: skip)")
    ap.add_argument("--cpu-full", action="store_true",
                    help="only the oracle's time to eps on the whole workload (host cores; "
                         "dense Q~ of 8 GiB at the default workload), then exit")
    ap.add_argument("--only-peak", choices=["f32", "f64"],
                    help="only the matrix-core loop peak probe for one dtype (for profiling)")
    ap.add_argument("--only-a5", action="store_true",
                    help="only the standalone CG vector-step measurement (for profiling)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (3 times) and exit: the "
                         "reference kernel for scaling HBM byte counters")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        src = torch.empty(args.calibrate_copy << 20, dtype=torch.uint8, device="cuda:0")
        src.fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": args.calibrate_copy << 20, "reps": 3}))
        return
    if args.cpu_full:
        import synthdata as S
        cfg = S.CONFIGS[args.config]
        X, y, scale = S.make_train(cfg)
        Xte, _ = S.make_test(cfg, scale, n_test=args.n_test)
        print(json.dumps({"cpu_full": cpu_full(cfg, X, y, Xte)}), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2202_12674_amd as P
    import synthdata as S

    if args.only_peak:
        dt = torch.float32 if args.only_peak == "f32" else torch.float64
        print(json.dumps({"measured_loop_peak_tflops": P.mfma_peak(dt, torch.device("cuda:0")),
                          "dtype": args.only_peak}), flush=True)
        return
    if args.only_a5:
        print(json.dumps({"a5_cg_vector_step": a5_standalone(torch, torch.device("cuda:0"),
                                                             args.a5_n)}), flush=True)
        return

    cfg = S.CONFIGS[args.config]
    dev = torch.device("cuda:0")
    log(f"[bench] generating {cfg.name}")
    X, y, scale = S.make_train(cfg)
    Xte, _ = S.make_test(cfg, scale, n_test=args.n_test)
    Xd = torch.from_numpy(X).to(dev)
    yd = torch.from_numpy(y).to(dev)
    Xted = torch.from_numpy(Xte).to(dev)
    kw = dict(kernel=cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)
    ws = P.alloc_workspace(P.workspace_bytes(cfg.n, cfg.d, Xd.dtype), dev)
    wsp = P.alloc_workspace(P.predict_workspace_bytes(cfg.n, args.n_test, cfg.d, Xd.dtype), dev)
    torch.cuda.synchronize()

    pred_ms = []

    # Even steps time every product with HIP events on the launch stream (the
    # roofline's launch durations); odd steps run without them, and give the
    # time to eps: an event pair costs the stream several microseconds, which
    # is most of an iteration on the smallest workload.
    def step(timed=True):
        r = P.train(Xd, yd, C=cfg.C, eps=cfg.eps, max_iter=cfg.max_iter, workspace=ws,
                    time_matvec=timed, matvec_times=4096 if timed else 0, **kw)
        t0 = time.perf_counter()
        P.predict(Xd, r.alpha, r.b, Xted, workspace=wsp, **kw)   # returns after the GPU work
        pred_ms.append((time.perf_counter() - t0) * 1e3)
        return r

    for i in range(args.warmup):
        r = step()
        log(f"[bench] warmup {i}: {r.iterations} it, train {r.t_total_ms:.1f} ms")
    torch.cuda.synchronize()
    results, walls = [], []
    t_all = time.perf_counter()
    for i in range(args.steps):
        t0 = time.perf_counter()
        r = step(timed=(i % 2 == 0))
        torch.cuda.synchronize()
        walls.append((time.perf_counter() - t0) * 1e3)
        results.append(r)
        log(f"[bench] step {i}: {r.iterations} it, train {r.t_total_ms:.1f} ms, "
            f"matvec avg {r.t_matvec_ms / max(1, r.n_matvec_timed):.3f} ms, "
            f"wall {walls[-1]:.1f} ms")
    torch.cuda.synchronize()
    total_ms = (time.perf_counter() - t_all) * 1e3
    # one more training, untimed, with the true residual ||rhs - Q~ x|| / ||rhs||
    # (one extra product after the solve)
    r_true = P.train(Xd, yd, C=cfg.C, eps=cfg.eps, max_iter=cfg.max_iter, workspace=ws,
                     true_residual=True, **kw)

    N = cfg.n - 1
    mv_flops = N * (N + 1) * cfg.d
    pred_flops = 2 * args.n_test * cfg.n * cfg.d
    n_mv = sum(r.n_matvec for r in results)
    step_flops = (n_mv * mv_flops + len(results) * pred_flops)
    ms_per_step = total_ms / args.steps
    value = step_flops / (total_ms * 1e-3) / 1e9
    mv_ms = sum(r.t_matvec_ms for r in results) / max(1, sum(r.n_matvec_timed for r in results))
    mv_each = [t for r in results for t in r.matvec_times]   # every timed product, in order
    achieved = mv_flops / (mv_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[cfg.dtype]
    measured_peak = P.mfma_peak(Xd.dtype, dev)
    log(f"[bench] measured matrix-core loop peak {measured_peak:.1f} TFLOP/s")
    traffic = traffic_record(cfg.name)
    untimed = [r for i, r in enumerate(results) if i % 2 == 1] or results
    train_ms = [r.t_total_ms for r in untimed]
    train_ms_timed = [r.t_total_ms for i, r in enumerate(results) if i % 2 == 0]
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "n": cfg.n, "d": cfg.d, "kernel": cfg.kernel,
                   "gamma": cfg.gamma, "coef0": cfg.coef0, "degree": cfg.degree, "C": cfg.C,
                   "eps": cfg.eps, "n_test": args.n_test},
        "time_to_eps_ms": round(statistics.median(train_ms), 3),
        "time_to_eps_cov": round(statistics.pstdev(train_ms) / statistics.mean(train_ms), 4),
        "time_to_eps_timed_ms": round(statistics.median(train_ms_timed), 3),
        "predict_ms": round(statistics.median(pred_ms[args.warmup:] or pred_ms), 3),
        "cg_iterations": results[-1].iterations,
        "cg_ms_per_iteration": round(statistics.median(train_ms) / max(1, results[-1].iterations),
                                     3),
        "rel_residual": r_true.rel_residual,
        "true_rel_residual": r_true.true_rel_residual,
        "n_matvec_per_step": results[-1].n_matvec,
        "matvec_ms": round(mv_ms, 4),
        "matvec_median_ms": round(statistics.median(mv_each), 4) if mv_each else None,
        "matvec_cov": (round(statistics.pstdev(mv_each) / statistics.mean(mv_each), 4)
                       if len(mv_each) > 1 else None),
        "matvec_reps": len(mv_each),
        "matvec_gflops": round(mv_flops / (mv_ms * 1e-3) / 1e9, 2),
        "matvec_dense_equiv_gflops": round(2 * N * N * cfg.d / (mv_ms * 1e-3) / 1e9, 2),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": traffic, "measured_loop_peak": round(measured_peak, 2),
                     "frac_of_measured_loop_peak": round(achieved / measured_peak, 4)},
        "device": device_facts(torch, dev),
        "kernel_source_hash": kernel_source_hash(),
    }
    del ws, wsp
    if args.a5_n > 0:
        log(f"[bench] CG vector step on N = {args.a5_n}")
        line["a5_cg_vector_step"] = a5_standalone(torch, dev, args.a5_n)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle sample")
        line["cpu_baseline"] = cpu_baseline(cfg, X, args.cpu_seconds)
        if args.cpu_phase_points > 0:
            log("[bench] timing the CPU oracle phases")
            line["cpu_baseline"]["phases"] = cpu_phases(cfg, X, y, Xte,
                                                        min(args.cpu_phase_points, cfg.n))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
