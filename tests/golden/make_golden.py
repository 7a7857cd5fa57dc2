"""Write the oracle's expected values for the five workloads.

Calls only the CPU oracle and the seeded generator; nothing here touches the
HIP path. Output: one ``<config>.npz`` per workload (no pickles) holding the
input hashes, the oracle's CG solution (alpha, b, iterations, residuals), the
reduced-matrix product with the seeded probe vector, and decision values and
labels on 1024 held-out points.

Usage: python tests/golden/make_golden.py [config names...]
       python tests/golden/make_golden.py --tight [config names...]
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle as O  # noqa: E402
import synthdata as S  # noqa: E402


def spec_of(cfg):
    return O.KernelSpec(cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)


def make(name):
    cfg = S.CONFIGS[name]
    t0 = time.time()
    X, y, scale = S.make_train(cfg)
    Xte, yte = S.make_test(cfg, scale)
    N = cfg.n - 1
    p = S.probe_vector(N, cfg.np_dtype)
    spec = spec_of(cfg)
    print(f"[{name}] data {time.time() - t0:.1f}s", flush=True)
    Qt, q, Qmm = O.reduced_matrix(X, spec, cfg.C)
    print(f"[{name}] reduced matrix {time.time() - t0:.1f}s", flush=True)
    mv = Qt @ p.astype(np.float64)
    # cross-check the dense route against the entry-by-entry rows of Eq. (16)
    rows = [0, 1, N // 3, N - 1]
    mr = O.matvec_rows(X, spec, cfg.C, p, rows)
    dev = float(np.abs(mv[rows] - mr).max() / np.abs(mv).max())
    print(f"[{name}] dense vs row route: {dev:.2e}", flush=True)
    if dev > 1e-12:
        raise SystemExit(f"[{name}] dense reduced matrix disagrees with the row route")
    rhs = O.reduced_rhs(y)
    res = O.solve_cg(lambda v: Qt @ v, rhs, cfg.eps, cfg.max_iter)
    print(f"[{name}] cg {res.iterations} it, conv={res.converged}, "
          f"true rel res {res.true_rel_residual:.3e}, {time.time() - t0:.1f}s", flush=True)
    alpha, b = O.recover(res.x, y, q, Qmm)
    # the same CG with only the summation order of the product changed: the
    # spread of the aggregates alpha_m = -sum(alpha~) and b that rounding alone causes
    h = N // 3
    res2 = O.solve_cg(lambda v: Qt[:, :h] @ v[:h] + Qt[:, h:] @ v[h:], rhs, cfg.eps, cfg.max_iter)
    alpha2, b2 = O.recover(res2.x, y, q, Qmm)
    print(f"[{name}] order spread: alpha {np.abs(alpha2 - alpha).max() / np.abs(alpha).max():.2e}"
          f" b {abs(b2 - b):.2e} ({res2.iterations} it)", flush=True)
    del Qt
    f_te, lab_te = O.predict(X, alpha, b, Xte, spec)
    f_tr, lab_tr = O.predict(X, alpha, b, X[:1024], spec)
    np.savez_compressed(
        os.path.join(HERE, f"{name}.npz"),
        hash_train=np.array(S.sha256_arrays(X, y)),
        hash_test=np.array(S.sha256_arrays(Xte)),
        hash_probe=np.array(S.sha256_arrays(p)),
        alpha=alpha, b=np.float64(b), q=q, Qmm=np.float64(Qmm),
        alpha_alt_order=alpha2, b_alt_order=np.float64(b2),
        iterations=np.int64(res.iterations), converged=np.bool_(res.converged),
        rel_residual=np.float64(res.rel_residual),
        true_rel_residual=np.float64(res.true_rel_residual),
        history=np.array(res.history), mv_probe=mv,
        f_test=f_te, labels_test=lab_te, f_train1024=f_tr, labels_train1024=lab_tr,
        acc_test=np.float64(np.mean(lab_te == yte)),
    )
    print(f"[{name}] done {time.time() - t0:.1f}s test acc {np.mean(lab_te == yte):.4f}", flush=True)


# Tighter eps for every workload: there two oracle CG runs that differ only in
# the summation order of their products agree far below the bar in every
# output (alpha~, alpha_m and b, each relative to its own size; 1e-10 for the
# fp64 workloads, 1e-6 for fp32), while the point CG stalls (its floor) is
# still further down. At the workloads' own eps they do not: the cubic fp32
# workload's b spreads by 7.1e-4 at eps = 1e-5 (25 against 26 iterations).
# Measured spreads: 256 x 64 at 1e-12 1.3e-13 (b); 4096 x 1024 at 1e-11
# 5.6e-11 (b; 1e-12 reaches the floor and stalls); 16384 x 2048 RBF at 1e-11
# 3.9e-12 (alpha_m; at 1e-10 b still spreads by 1.8e-10); 32768 x 4096 cubic
# at 1e-8 1.7e-9 (b).
TIGHT_EPS = {"linear_f64_256x64": 1e-12, "linear_f64_4096x1024": 1e-11,
             "rbf_f64_16384x2048": 1e-11, "poly_f32_32768x4096": 1e-8,
             "rbf_f32_65536x1024": 1e-8}
TIGHT_SPREAD = {"f64": 1e-10, "f32": 1e-6}


def make_tight(name):
    """<config>_tight.npz: the oracle's CG at the tight eps and its spread under
    a change of summation order; for the fp64 workloads also the Cholesky
    solution of the reduced system (Sec. III-B) with its alpha_m and b
    (Eqs. (11), (15)). (A dense factor of the fp32 workloads' 8 and 32 GiB
    reduced matrices is left out.)"""
    cfg = S.CONFIGS[name]
    eps = TIGHT_EPS[name]
    t0 = time.time()
    X, y, _ = S.make_train(cfg)
    spec = spec_of(cfg)
    Qt, q, Qmm = O.reduced_matrix(X, spec, cfg.C)
    rhs = O.reduced_rhs(y)
    N = Qt.shape[0]
    print(f"[{name}] reduced matrix {time.time() - t0:.1f}s", flush=True)
    res = O.solve_cg(lambda v: Qt @ v, rhs, eps, cfg.max_iter)
    if not res.converged:
        raise SystemExit(f"[{name}] CG at eps {eps:g} did not converge")
    alpha, b = O.recover(res.x, y, q, Qmm)
    h = N // 3
    res2 = O.solve_cg(lambda v: Qt[:, :h] @ v[:h] + Qt[:, h:] @ v[h:], rhs, eps, cfg.max_iter)
    alpha2, b2 = O.recover(res2.x, y, q, Qmm)
    spread = (float(np.abs(alpha2[:-1] - alpha[:-1]).max() / np.abs(alpha).max()),
              abs(alpha2[-1] - alpha[-1]) / abs(alpha[-1]), abs(b2 - b) / abs(b))
    print(f"[{name}] eps {eps:g}: cg {res.iterations} it, order spread alpha~ {spread[0]:.1e} "
          f"alpha_m {spread[1]:.1e} b {spread[2]:.1e} (relative), {time.time() - t0:.1f}s",
          flush=True)
    if max(spread) > TIGHT_SPREAD[cfg.dtype]:
        raise SystemExit(f"[{name}] eps {eps:g} is not tight enough")
    extra = {}
    if cfg.dtype == "f64":
        xs = O.solve_cholesky(Qt, rhs)
        alpha_c, b_c = O.recover(xs, y, q, Qmm)
        print(f"[{name}] cholesky: |alpha - alpha_chol| {np.abs(alpha - alpha_c).max():.1e}, "
              f"b {b:.12g} vs {b_c:.12g}, {time.time() - t0:.1f}s", flush=True)
        extra = dict(alpha_chol=alpha_c, b_chol=np.float64(b_c))
    np.savez_compressed(
        os.path.join(HERE, f"{name}_tight.npz"),
        hash_train=np.array(S.sha256_arrays(X, y)),
        eps_tight=np.float64(eps), alpha_tight=alpha, b_tight=np.float64(b),
        iterations_tight=np.int64(res.iterations), spread_tight=np.array(spread),
        q=q, Qmm=np.float64(Qmm), **extra)


if __name__ == "__main__":
    args = sys.argv[1:]
    if args and args[0] == "--tight":
        for nm in args[1:] or list(TIGHT_EPS):
            make_tight(nm)
    else:
        for nm in args or list(S.CONFIGS):
            make(nm)
