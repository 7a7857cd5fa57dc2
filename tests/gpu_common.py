"""Helpers of the GPU parity tests: seeded workloads, the oracle's reference
solution of a training, and the training check that applies the named rules
of parity_rules.py. Test infrastructure only."""
from __future__ import annotations

import dataclasses
import os
import sys

import numpy as np
import pytest

import oracle as O
import synthdata as S
from parity_rules import (BAR_MV, BAR_SOL, U32, alpha_tilde_error, bias_step_errors,
                          end_to_end_errors, label_check, p9_check, rel_err)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL_MV = BAR_MV
TOL_ALPHA = BAR_SOL

__all__ = ["GOLDEN", "TOL_MV", "TOL_ALPHA", "BAR_MV", "BAR_SOL", "rel_err", "log", "spec_of",
           "kw_of", "small_cfg", "data_of", "to_dev", "golden", "golden_tight", "SPLIT_SHAPES",
           "TAIL_SHAPES", "random_cases", "random_large_cases", "random_param_cases", "random_param_train_cases",
           "fp32_sensitivity", "OracleRef", "oracle_ref", "check_train", "labels_match"]


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def spec_of(cfg):
    return O.KernelSpec(cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)


def kw_of(cfg):
    return dict(kernel=cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)


def small_cfg(kernel, dtype, n, d, C=1.0, eps=None, flip=0.05):
    eps = eps if eps is not None else (1e-10 if dtype == "f64" else 1e-5)
    kw = dict(linear={}, poly=dict(gamma=1.0 / d, coef0=1.0, degree=3),
              rbf=dict(gamma=1.0 / d))[kernel]
    return S.Config(f"{kernel}_{dtype}_{n}x{d}", dtype, kernel, n, d, mu=1.0, inf_frac=0.5,
                    flip_frac=flip, C=C, eps=eps, **kw)


_DATA = {}


def data_of(cfg):
    key = (cfg.name, cfg.n, cfg.d, cfg.dtype)
    if key not in _DATA:
        X, y, scale = S.make_train(cfg)
        Xte, yte = S.make_test(cfg, scale)
        _DATA.clear()
        _DATA[key] = (X, y, Xte, yte)
    return _DATA[key]


def to_dev(torch, dev, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def golden(name):
    path = os.path.join(GOLDEN, f"{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"golden values for {name} not generated")
    return np.load(path, allow_pickle=False)


# Linear products of few tiles split each tile's features over several
# workgroups; these shapes give every split the library uses.
# (dtype, n, d, plan) of the linear kernel's feature splits; plan is the
# library's (workgroups per tile, tiles of the finer-split last round,
# workgroups per such tile): splits without a tail, a tail over the split
# full rounds, and a tail after unsplit ones (the 4096 x 1024 fp64 workload).
SPLIT_SHAPES = [("f64", 600, 256, (16, 0, 16)), ("f64", 2000, 512, (4, 8, 16)),
                ("f64", 1000, 2048, (16, 4, 64)), ("f64", 3000, 256, (2, 44, 8)),
                ("f64", 4096, 1024, (1, 16, 32)), ("f32", 1000, 256, (8, 0, 8)),
                ("f32", 600, 1024, (16, 0, 16)), ("f32", 2000, 1024, (4, 8, 16)),
                ("f32", 3000, 512, (2, 44, 8)), ("f32", 4096, 256, (1, 16, 4))]

# (dtype, kernel, n, d, plan): the tiles after the last full round of 512
# workgroups split 4..16 ways, parked and fixed up (linear: added up).
TAIL_SHAPES = [("f64", "rbf", 600, 256, (1, 15, 8)), ("f32", "poly", 600, 256, (1, 15, 4)),
               ("f64", "poly", 4096, 256, (1, 16, 8)), ("f32", "rbf", 4096, 512, (1, 16, 8)),
               ("f64", "linear", 12288, 1024, (1, 48, 8))]


def random_cases(count=24, seed=2026):
    """Seeded shapes across kernels and precisions: ragged n and d that land on
    every way a product is laid out (padding, feature splits, split tails)."""
    rng = np.random.default_rng(seed)
    cases = []
    for k in range(count):
        n, d = int(rng.integers(2, 3000)), int(rng.integers(1, 700))
        C = float(rng.choice([0.1, 1.0, 10.0]))
        cases.append((["linear", "poly", "rbf"][k % 3], ["f64", "f32"][(k // 3) % 2], n, d, C))
    return cases


def random_large_cases(count=16, seed=11):
    """Seeded large shapes (2000..40000 points, 100..5000 features, log-uniform),
    random kernel parameters and C from 0.01 to 100."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        n = int(np.exp(rng.uniform(np.log(2000), np.log(40000))))
        d = int(np.exp(rng.uniform(np.log(100), np.log(5000))))
        kernel = ["linear", "poly", "rbf"][rng.integers(3)]
        dtype = ["f64", "f32"][rng.integers(2)]
        C = float(10 ** rng.uniform(-2, 2))
        kp = dict(linear={}, poly=dict(gamma=1.0 / d, coef0=float(rng.choice([0.0, 1.0])),
                                       degree=int(rng.integers(1, 5))),
                  rbf=dict(gamma=float(10 ** rng.uniform(-1, 0.5)) / d))[kernel]
        out.append((kernel, dtype, n, d, C, kp))
    return out


def random_param_cases(count=48, seed=31337):
    """Seeded small shapes (2..2500 points log-uniform, 1..1500 features) with
    random kernel parameters and C from 0.01 to 100: every split of the
    linear kernel's small problems (down to one feature block per workgroup)
    and every kernel function's epilogue on ragged tiles."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(count):
        n = max(2, int(np.exp(rng.uniform(np.log(2), np.log(2500)))))
        d = int(np.exp(rng.uniform(0, np.log(1500))))
        kernel = ["linear", "poly", "rbf"][k % 3]
        dtype = ["f64", "f32"][(k // 3) % 2]
        C = float(10 ** rng.uniform(-2, 2))
        kp = dict(linear={}, poly=dict(gamma=1.0 / d, coef0=float(rng.choice([0.0, 1.0])),
                                       degree=int(rng.integers(1, 5))),
                  rbf=dict(gamma=float(10 ** rng.uniform(-1, 0.5)) / d))[kernel]
        out.append((kernel, dtype, n, d, C, kp))
    return out


def random_param_train_cases(count=12, seed=4711):
    """Seeded trainings of 50..1500 points and 2..600 features with random
    kernel parameters (polynomial degree 1..4, coef0 0 or 1, RBF gamma 0.1/d
    to 3/d) and C from 0.1 to 10."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(count):
        n = int(np.exp(rng.uniform(np.log(50), np.log(1500))))
        d = int(np.exp(rng.uniform(np.log(2), np.log(600))))
        kernel = ["linear", "poly", "rbf"][k % 3]
        dtype = ["f64", "f32"][(k // 3) % 2]
        C = float(10 ** rng.uniform(-1, 1))
        kp = dict(linear={}, poly=dict(gamma=1.0 / d, coef0=float(rng.choice([0.0, 1.0])),
                                       degree=int(rng.integers(1, 5))),
                  rbf=dict(gamma=float(10 ** rng.uniform(-1, 0.5)) / d))[kernel]
        out.append((kernel, dtype, n, d, C, kp))
    return out


def fp32_sensitivity(X, cfg):
    """kappa(Q~) u32, a first-order bound on how far rounding the kernel values
    to fp32 can move the solution relative to its size: lambda_min(Q~) >= 1/C
    (Q~ = P^T Q P with P^T P >= I) and lambda_max(Q~) from power iteration."""
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    v = np.random.default_rng(0).standard_normal(Qt.shape[0])
    for _ in range(30):
        v = Qt @ v
        v /= np.linalg.norm(v)
    return float(v @ (Qt @ v)) * cfg.C * 2.0 ** -24


def golden_tight(name):
    path = os.path.join(GOLDEN, f"{name}_tight.npz")
    if not os.path.exists(path):
        pytest.skip(f"tight-eps golden values for {name} not generated")
    return np.load(path, allow_pickle=False)


@dataclasses.dataclass
class OracleRef:
    """The oracle's solution of one training: CG at the training's eps (alpha,
    b, iterations), q and Q_mm (Eq. (12)), and, where the reduced matrix fits
    in host memory, Q~, rhs and the Cholesky solution for the rigorous bound."""
    alpha: np.ndarray
    b: float
    iterations: int
    q: np.ndarray
    Qmm: float
    Qt: np.ndarray | None = None
    rhs: np.ndarray | None = None
    x_chol: np.ndarray | None = None
    b_chol: float | None = None


def oracle_ref(cfg, X, y, eps=None, cholesky=True):
    spec = spec_of(cfg)
    Qt, q, Qmm = O.reduced_matrix(X, spec, cfg.C)
    rhs = O.reduced_rhs(y)
    res = O.solve_cg(lambda v: Qt @ v, rhs, cfg.eps if eps is None else eps, cfg.max_iter)
    alpha, b = O.recover(res.x, y, q, Qmm)
    ref = OracleRef(alpha, b, res.iterations, q, Qmm, Qt, rhs)
    if cholesky:
        xs = O.solve_cholesky(Qt, rhs)
        ref.x_chol = xs
        ref.b_chol = O.recover(xs, y, q, Qmm)[1]
    return ref


def labels_match(lab, f_ref, scale_tol):
    """Labels equal wherever the oracle's decision value is not within
    scale_tol x max(1, max|f|) of 0 (prediction checks on a given model)."""
    f_ref = np.asarray(f_ref)
    lab_ref = np.where(f_ref > 0, 1, -1)
    tie = np.abs(f_ref) <= scale_tol * max(1.0, np.abs(f_ref).max())
    bad = (np.asarray(lab) != lab_ref) & ~tie
    return int(bad.sum()), int(tie.sum())


def check_train(torch, dev, cfg, ref: OracleRef, X, y, Xte=None, f_te=None, max_ties=None,
                alpha_tol=None, eps=None):
    """Train on the GPU and apply the parity rules against the oracle's ref.

    * alpha~ against the oracle's CG at the same eps: the contract bar
      (alpha_tol only for fp32 systems too ill-conditioned for it, see
      test_train_random_shapes);
    * the bias step on the GPU's own alpha~: the contract bar, relative to
      |alpha_m| and |b|;
    * where ref holds Q~ and the Cholesky solution: the rigorous distance of
      alpha~, alpha_m and b to the exact solution (P9), and for fp64 the
      residual formed by the oracle's Q~ at eps;
    * labels: equal except near-ties the solution difference can flip, at most
      max_ties of them (default: 1% of the test points, at least 1).
    alpha_m and b against the oracle's CG (each relative to its own size) are
    logged: at the training's eps they are defined only to eps (see the
    tight-eps test of the fp64 workloads, which asserts them)."""
    import paper_2202_12674_amd as P
    eps = cfg.eps if eps is None else eps
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=eps,
                  max_iter=cfg.max_iter, true_residual=True, **kw_of(cfg))
    log(f"  {cfg.name}: status {res.status} it {res.iterations} (oracle {ref.iterations}) "
        f"rel {res.rel_residual:.2e} true {res.true_rel_residual:.2e} cg {res.t_cg_ms:.1f} ms")
    assert res.converged
    bar = BAR_SOL[cfg.dtype]
    alpha = res.alpha.cpu().numpy().astype(np.float64)
    e_t = alpha_tilde_error(alpha, ref.alpha)
    tol_t = bar if alpha_tol is None else alpha_tol
    e_am, e_b, e_bf = end_to_end_errors(alpha, res.b, ref.alpha, ref.b)
    s_am, st_am, s_b, st_b = bias_step_errors(alpha, res.b, y, ref.q, ref.Qmm, cfg.dtype)
    log(f"  alpha~ err {e_t:.2e} (tol {tol_t:.0e}); bias step on the GPU's alpha~: alpha_m "
        f"{s_am:.1e} (tol {st_am:.1e}), b {s_b:.1e} (tol {st_b:.1e}); vs the oracle's CG "
        f"(relative to each): alpha_m {e_am:.1e}, b {e_b:.1e} (b on the scale of f {e_bf:.1e})")
    assert e_t <= tol_t
    assert s_am <= st_am and s_b <= st_b
    if ref.Qt is not None and ref.x_chol is not None:
        p9 = p9_check(alpha, res.b, ref.Qt, ref.q, ref.Qmm, ref.rhs, cfg.C, ref.x_chol,
                      ref.b_chol)
        log(f"  P9 vs Cholesky: |alpha~ - x*| {p9['dist']:.1e} <= {p9['bound']:.1e}, alpha_m "
            f"{p9['d_am']:.1e} <= {p9['bound_am']:.1e}, b {p9['d_b']:.1e} <= {p9['bound_b']:.1e}"
            f", ||r||/||rhs|| (oracle's Q~) {p9['rel_res']:.1e}")
        assert p9["dist"] <= p9["bound"]
        assert p9["d_am"] <= p9["bound_am"] and p9["d_b"] <= p9["bound_b"]
        if cfg.dtype == "f64":
            assert p9["rel_res"] <= 2 * eps + 1e-10
    if cfg.dtype == "f64":
        assert abs(res.iterations - ref.iterations) <= max(2, ref.iterations // 10)
    else:   # fp32 products perturb the Krylov space: a few more iterations are normal
        assert res.iterations <= 2 * ref.iterations + 10
    # alpha_m is minus the sum of the others (last row of Eq. (11)), up to rounding
    tol_sum = (1e-12 if cfg.dtype == "f64" else 1e-5) * max(1.0, np.abs(alpha).sum())
    assert abs(alpha.sum()) <= tol_sum
    if Xte is not None:
        scores, labels = P.predict(to_dev(torch, dev, X), res.alpha, res.b,
                                   to_dev(torch, dev, Xte), **kw_of(cfg))
        f_mix = O.decision(X, alpha, res.b, Xte, spec_of(cfg))
        bad, ties, band = label_check(labels.cpu().numpy(), f_te, f_mix, cfg.dtype)
        limit = max(1, len(Xte) // 100) if max_ties is None else max_ties
        log(f"  test labels: {bad} mismatches, {ties} near-ties (limit {limit}, widest band "
            f"{band:.1e}, min |f| {np.abs(f_te).min():.1e})")
        assert bad == 0 and ties <= limit
    return res
