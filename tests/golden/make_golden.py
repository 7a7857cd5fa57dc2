"""Write the oracle's expected values for the five workloads.

Calls only the CPU oracle and the seeded generator; nothing here touches the
HIP path. Output: one ``<config>.npz`` per workload (no pickles) holding the
input hashes, the oracle's CG solution (alpha, b, iterations, residuals), the
reduced-matrix product with the seeded probe vector, and decision values and
labels on 1024 held-out points.

Usage: python tests/golden/make_golden.py [config names...]
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


if __name__ == "__main__":
    names = sys.argv[1:] or list(S.CONFIGS)
    for nm in names:
        make(nm)
