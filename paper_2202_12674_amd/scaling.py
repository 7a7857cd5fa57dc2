"""GPU training runtime against the number of points and the number of features.

The paper measures how its GPU training time grows with the data: in points
(2^8 .. 2^15 at 2^12 features) and in features (2^6 .. 2^14 at 2^15 points)
(Sec. IV-D). This harness runs the same two sweeps on one MI355X, with
synthetic data of the workloads' recipe, and prints one JSON line per size:
the implicit product's time (HIP events around each product inside the
training), its rate in the symmetric count N(N+1)d against the matrix-core
peak, the CG iterations and the time to eps (data resident in HBM). Each
size is trained twice and the second run is reported.

    python -m paper_2202_12674_amd.scaling [--dtype f64 --kernel linear --eps 1e-3]
    python -m paper_2202_12674_amd.scaling --only 16384 4096
"""
from __future__ import annotations

import argparse
import json
import os
import sys

PEAK_TFLOPS = {"f64": 78.6, "f32": 157.3}   # MI355X dense matrix-core peaks


def sizes(points_exp=(8, 15), features_exp=(6, 14), d_fixed=4096, n_fixed=32768):
    """(sweep, n, d) of the two sweeps, in the order they run."""
    out = [("points", 2 ** e, d_fixed) for e in range(points_exp[0], points_exp[1] + 1)]
    out += [("features", n_fixed, 2 ** e) for e in range(features_exp[0], features_exp[1] + 1)]
    return out


def measure(cfg, device, reps: int = 2):
    """Train cfg `reps` times on the device and report the last run."""
    import torch

    from . import _binding as B
    import synthdata as S
    X, y, _ = S.make_train(cfg)
    Xd, yd = torch.from_numpy(X).to(device), torch.from_numpy(y).to(device)
    del X, y
    kw = dict(kernel=cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)
    ws = B.alloc_workspace(B.workspace_bytes(cfg.n, cfg.d, Xd.dtype), device)
    r = None
    for _ in range(reps):
        torch.cuda.synchronize()
        r = B.train(Xd, yd, C=cfg.C, eps=cfg.eps, workspace=ws, time_matvec=True, **kw)
    N = cfg.n - 1
    mv_ms = r.t_matvec_ms / max(1, r.n_matvec_timed)
    tflops = N * (N + 1) * cfg.d / (mv_ms * 1e-3) / 1e12 if mv_ms > 0 else 0.0
    return {"n": cfg.n, "d": cfg.d, "iterations": r.iterations, "converged": r.converged,
            "time_to_eps_ms": round(r.t_total_ms, 3), "product_ms": round(mv_ms, 4),
            "product_tflops": round(tflops, 2),
            "frac_of_peak": round(tflops / PEAK_TFLOPS[cfg.dtype], 4)}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--kernel", default="linear", choices=["linear", "poly", "rbf"])
    ap.add_argument("--dtype", default="f64", choices=["f64", "f32"])
    ap.add_argument("--C", type=float, default=1.0)
    ap.add_argument("--eps", type=float, default=1e-3)
    ap.add_argument("--max-points-exp", type=int, default=15)
    ap.add_argument("--max-features-exp", type=int, default=14)
    ap.add_argument("--only", type=int, nargs=2, metavar=("N", "D"),
                    help="one size only (for instance under a profiler)")
    args = ap.parse_args(argv)

    import torch

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import synthdata as S

    dev = torch.device("cuda:0")
    todo = ([("one", args.only[0], args.only[1])] if args.only
            else sizes((8, args.max_points_exp), (6, args.max_features_exp)))
    for sweep, n, d in todo:
        kparams = {"linear": {}, "poly": dict(gamma=1.0 / d, coef0=1.0, degree=3),
                   "rbf": dict(gamma=1.0 / d)}[args.kernel]
        cfg = S.Config(f"{args.kernel}_{args.dtype}_{n}x{d}", args.dtype, args.kernel, n, d,
                       mu=1.0, inf_frac=0.3, flip_frac=0.05, C=args.C, eps=args.eps, **kparams)
        print(f"[scaling] {sweep}: {cfg.name}", file=sys.stderr, flush=True)
        row = measure(cfg, dev)
        print(json.dumps({"sweep": sweep, "workload": cfg.name, "dtype": args.dtype,
                          "kernel": args.kernel, "eps": args.eps, **row}), flush=True)
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
