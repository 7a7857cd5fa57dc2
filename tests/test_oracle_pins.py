"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each compares it with an
independent route (a product with the explicit bordered matrix, an exact
rational or 50-digit solve, a textbook closed form, an invariant). A
plausible slip in the oracle (a dropped 1/C, a wrong sign of b, a transposed
partition, a wrong CG update) fails at least one of them.
"""
from __future__ import annotations

import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest

import oracle as O
import synthdata as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SPECS = [
    O.KernelSpec("linear"),
    O.KernelSpec("poly", gamma=0.25, coef0=1.0, degree=3),
    O.KernelSpec("rbf", gamma=0.5),
]


def small_problem(n=40, d=5, seed=3, flip=0.1):
    X, y = S.gen_raw(n, d, seed, mu=0.7, inf_frac=0.6, flip_frac=flip)
    lo, hi = S.minmax_fit(X)
    return S.minmax_apply(X, lo, hi), y


def P_matrix(n):
    """P = [I_N; -1^T], so that P^T Q P is the reduced matrix."""
    N = n - 1
    return np.vstack([np.eye(N), -np.ones((1, N))])


# ---------------------------------------------------------------- kernels ---

def brute_kernel(x, z, spec):
    """Pure-Python kernel value, straight from the kernel table of Sec. II-E."""
    dot = sum(float(a) * float(b) for a, b in zip(x, z))
    if spec.kind == "linear":
        return dot
    if spec.kind == "poly":
        return (spec.gamma * dot + spec.coef0) ** spec.degree
    dist = sum((float(a) - float(b)) ** 2 for a, b in zip(x, z))
    return float(np.exp(-spec.gamma * dist))


@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_kernel_matrix_brute_force(spec):
    X, _ = small_problem(n=9, d=4)
    K = O.kernel_matrix(X, spec)
    for i in range(9):
        for j in range(9):
            assert K[i, j] == pytest.approx(brute_kernel(X[i], X[j], spec), rel=1e-13, abs=1e-14)
    Z = X[:3] * 0.5
    R = O.kernel_rows(Z, X, spec)
    for i in range(3):
        for j in range(9):
            assert R[i, j] == pytest.approx(brute_kernel(Z[i], X[j], spec), rel=1e-13, abs=1e-14)


def test_kernel_matrix_exactly_symmetric_large():
    X, _ = small_problem(n=1500, d=9)
    for spec in SPECS:
        K = O.kernel_matrix(X, spec)
        assert np.array_equal(K, K.T)


# --------------------------------------------------- reduced matrix (P1) ---

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
@pytest.mark.parametrize("C", [1.0, 10.0, 0.1])
def test_reduced_matrix_is_PtQP(spec, C):
    """Eq. (13) elementwise equals P^T Q P with Q the block of Eq. (11)."""
    X, _ = small_problem(n=33, d=6)
    n = X.shape[0]
    M = O.bordered_matrix(X, spec, C)
    Q = M[:n, :n]
    Pm = P_matrix(n)
    ref = Pm.T @ Q @ Pm
    Qt, q, Qmm = O.reduced_matrix(X, spec, C)
    assert np.abs(Qt - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())
    # the Eq. (16) entry-by-entry rows, multiplied by a vector
    p = np.random.default_rng(1).standard_normal(n - 1)
    rows = [0, 5, n - 2]
    mv = O.matvec_rows(X, spec, C, p, rows)
    assert np.allclose(mv, (ref @ p)[rows], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_reduced_rows_match_PtQP(spec):
    """Row panels of Q~ (used where the full matrix does not fit) equal P^T Q P."""
    X, _ = small_problem(n=41, d=5)
    n = X.shape[0]
    M = O.bordered_matrix(X, spec, 0.3)
    ref = P_matrix(n).T @ M[:n, :n] @ P_matrix(n)
    rows = [0, 3, 17, 39]
    R = O.reduced_rows(X, spec, 0.3, rows)
    assert np.abs(R - ref[rows]).max() <= 1e-12 * max(1.0, np.abs(ref).max())


def test_reduced_parts_partition():
    """Eq. (12): q is the last column of Q (without the last entry), Q_mm its corner."""
    X, _ = small_problem(n=12, d=3)
    spec = SPECS[1]
    C = 2.0
    M = O.bordered_matrix(X, spec, C)
    Qbar, q, Qmm = O.reduced_parts(X, spec, C)
    assert np.allclose(Qbar, M[:11, :11], rtol=0, atol=1e-14)
    assert np.allclose(q, M[:11, 11], rtol=0, atol=1e-14)
    assert Qmm == pytest.approx(M[11, 11], abs=1e-14)
    assert Qmm == pytest.approx(brute_kernel(X[11], X[11], spec) + 1.0 / C, abs=1e-13)


# ------------------------------------------------------ SPD (P2) ------------

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
@pytest.mark.parametrize("C", [1.0, 10.0])
def test_reduced_matrix_spd_bounds(spec, C):
    """Q~ symmetric, Cholesky succeeds, lambda_min >= 1/C, lambda_max <= n lambda_max(Q)."""
    X, _ = small_problem(n=60, d=4)
    Qt, _, _ = O.reduced_matrix(X, spec, C)
    assert np.array_equal(Qt, Qt.T)
    np.linalg.cholesky(Qt)
    ev = np.linalg.eigvalsh(Qt)
    assert ev[0] >= 1.0 / C * (1 - 1e-10)
    Q = O.bordered_matrix(X, spec, C)[:60, :60]
    assert ev[-1] <= 60 * np.linalg.eigvalsh(Q)[-1] * (1 + 1e-12)


# ------------------------------------------- bordered system routes (P3) ----

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_reduced_route_equals_bordered_and_schur(spec):
    X, y = small_problem(n=50, d=5)
    C = 1.5
    alpha, b, _ = O.train(X, y, spec, C, eps=1e-12, method="cholesky")
    n = X.shape[0]
    M = O.bordered_matrix(X, spec, C)
    sol = np.linalg.solve(M, np.concatenate([y, [0.0]]))        # LU of Eq. (11)
    assert np.abs(alpha - sol[:n]).max() <= 1e-11 * np.abs(sol[:n]).max()
    assert b == pytest.approx(sol[n], abs=1e-11)
    # Schur complement closed form: b = 1^T Q^-1 y / 1^T Q^-1 1, alpha = Q^-1 (y - b 1)
    Q = M[:n, :n]
    Qi_y = np.linalg.solve(Q, y)
    Qi_1 = np.linalg.solve(Q, np.ones(n))
    b_s = Qi_y.sum() / Qi_1.sum()
    a_s = Qi_y - b_s * Qi_1
    assert b == pytest.approx(b_s, abs=1e-11)
    assert np.abs(alpha - a_s).max() <= 1e-11 * np.abs(a_s).max()


# ----------------------------------------- KKT residual identity (P4, P6) ---

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_full_system_residual_equals_reduced(spec):
    X, y = small_problem(n=70, d=6)
    C, eps = 1.0, 1e-6
    alpha, b, info = O.train(X, y, spec, C, eps=eps, method="cg")
    assert info["converged"]
    Qt, q, Qmm = O.reduced_matrix(X, spec, C)
    rhs = O.reduced_rhs(y)
    red = Qt @ alpha[:-1] - rhs
    full = O.full_system_residual(X, y, spec, C, alpha, b)
    n = X.shape[0]
    assert np.abs(full[:n - 1] - red).max() <= 1e-12 * max(1.0, np.abs(rhs).max())
    assert abs(full[n - 1]) <= 1e-12          # the pivot's row of Eq. (11)
    assert abs(full[n]) <= 1e-12              # sum(alpha) = 0
    assert abs(alpha.sum()) <= 1e-12
    assert np.linalg.norm(red) <= 1.5 * eps * np.linalg.norm(rhs)


# --------------------------------------------------- pivot invariance (P5) --

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_pivot_invariance(spec):
    X, y = small_problem(n=30, d=4)
    C = 3.0
    a1, b1, _ = O.train(X, y, spec, C, 1e-12, method="cholesky")
    perm = np.roll(np.arange(30), 7)          # another point becomes the last one
    a2, b2, _ = O.train(X[perm], y[perm], spec, C, 1e-12, method="cholesky")
    back = np.empty(30)
    back[perm] = a2
    assert np.abs(a1 - back).max() <= 1e-11 * np.abs(a1).max()
    assert b1 == pytest.approx(b2, abs=1e-11)


# ---------------------------------------------- training identity (P7) -----

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_training_identity(spec):
    """Row i of Eq. (11): f(x_i) = sum_j alpha_j k(x_i, x_j) + b = y_i - alpha_i / C."""
    X, y = small_problem(n=45, d=5)
    C = 2.0
    alpha, b, _ = O.train(X, y, spec, C, 1e-12, method="cholesky")
    f, lab = O.predict(X, alpha, b, X, spec)
    assert np.abs(f - (y - alpha / C)).max() <= 1e-11
    assert np.array_equal(lab, np.where(f > 0, 1, -1))


# ------------------------------------------------- ridge regression (P8) ----

def test_linear_kernel_is_ridge_with_free_intercept():
    X, y = small_problem(n=80, d=6)
    C = 0.7
    alpha, b, _ = O.train(X, y, O.KernelSpec("linear"), C, 1e-12, method="cholesky")
    xbar = X.mean(axis=0)
    ybar = y.mean()
    Xc = X - xbar
    w = np.linalg.solve(Xc.T @ Xc + np.eye(6) / C, Xc.T @ (y - ybar))
    assert np.abs(X.T @ alpha - w).max() <= 1e-12 * max(1.0, np.abs(w).max())
    assert b == pytest.approx(ybar - w @ xbar, abs=1e-12)


# ------------------------------------------------ CG error bound (P9) -------

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
@pytest.mark.parametrize("C", [1.0, 10.0])
def test_cg_error_bound_against_cholesky(spec, C):
    """||x_cg - x*||_2 <= ||Q~^-1||_2 ||r||_2 <= C ||rhs - Q~ x_cg||_2."""
    X, y = small_problem(n=200, d=8, seed=5)
    Qt, _, _ = O.reduced_matrix(X, spec, C)
    rhs = O.reduced_rhs(y)
    xs = O.solve_cholesky(Qt, rhs)
    for eps in (1e-2, 1e-4, 1e-8):
        res = O.solve_cg(lambda v: Qt @ v, rhs, eps)
        assert res.converged
        r = np.linalg.norm(rhs - Qt @ res.x)
        assert np.linalg.norm(res.x - xs) <= C * r * (1 + 1e-8) + 1e-13
        assert res.true_rel_residual == pytest.approx(r / np.linalg.norm(rhs), rel=1e-12)


# ------------------------------------------- exact tiny solves (P10) --------

def _exact_solve(M, rhs):
    """Gauss-Jordan elimination over exact rationals (or mpmath numbers)."""
    n = len(M)
    A = [list(row) + [rhs[i]] for i, row in enumerate(M)]
    for c in range(n):
        piv = next(r for r in range(c, n) if A[r][c] != 0)
        A[c], A[piv] = A[piv], A[c]
        pv = A[c][c]
        A[c] = [v / pv for v in A[c]]
        for r in range(n):
            if r != c and A[r][c] != 0:
                f = A[r][c]
                A[r] = [a - f * b for a, b in zip(A[r], A[c])]
    return [A[i][n] for i in range(n)]


def _tiny_points():
    # small dyadic rationals: exact in binary floating point
    X = np.array([[0.5, -1.0, 0.25], [1.0, 0.75, -0.5], [-0.25, 0.5, 1.0],
                  [-1.0, -0.5, 0.0], [0.0, 1.0, -0.75], [0.75, -0.25, 0.5]])
    y = np.array([1.0, 1.0, -1.0, -1.0, 1.0, -1.0])
    return X, y


@pytest.mark.parametrize("spec", [O.KernelSpec("linear"),
                                  O.KernelSpec("poly", gamma=0.5, coef0=1.0, degree=3),
                                  O.KernelSpec("poly", gamma=2.0, coef0=0.0, degree=2)],
                         ids=["linear", "poly3", "poly2"])
@pytest.mark.parametrize("C", [Fraction(1), Fraction(1, 4)])
def test_exact_rational_solve(spec, C):
    X, y = _tiny_points()
    n = len(y)
    Xf = [[Fraction(v) for v in row] for row in X]
    g, r = Fraction(spec.gamma), Fraction(spec.coef0)

    def k(a, b):
        dot = sum(p * q for p, q in zip(a, b))
        return dot if spec.kind == "linear" else (g * dot + r) ** spec.degree

    M = [[k(Xf[i], Xf[j]) + (1 / C if i == j else 0) for j in range(n)] + [Fraction(1)]
         for i in range(n)] + [[Fraction(1)] * n + [Fraction(0)]]
    sol = _exact_solve(M, [Fraction(v) for v in y] + [Fraction(0)])
    alpha, b, _ = O.train(X, y, spec, float(C), 1e-14, method="cholesky")
    ex_a = np.array([float(v) for v in sol[:n]])
    assert np.abs(alpha - ex_a).max() <= 1e-13 * max(1.0, np.abs(ex_a).max())
    assert b == pytest.approx(float(sol[n]), abs=1e-13)
    # the CG route converges to the same exact answer
    alpha2, b2, info = O.train(X, y, spec, float(C), 1e-14, method="cg")
    assert np.abs(alpha2 - ex_a).max() <= 1e-11 * max(1.0, np.abs(ex_a).max())
    assert b2 == pytest.approx(float(sol[n]), abs=1e-11)


@pytest.mark.parametrize("gamma", [0.5, 2.0])
def test_rbf_50_digit_solve(gamma):
    mpmath.mp.dps = 50
    X, y = _tiny_points()
    n = len(y)
    Xm = [[mpmath.mpf(v) for v in row] for row in X]
    C = mpmath.mpf(1)

    def k(a, b):
        return mpmath.exp(-mpmath.mpf(gamma) * sum((p - q) ** 2 for p, q in zip(a, b)))

    M = [[k(Xm[i], Xm[j]) + (1 / C if i == j else 0) for j in range(n)] + [mpmath.mpf(1)]
         for i in range(n)] + [[mpmath.mpf(1)] * n + [mpmath.mpf(0)]]
    sol = _exact_solve(M, [mpmath.mpf(v) for v in y] + [mpmath.mpf(0)])
    alpha, b, _ = O.train(X, y, O.KernelSpec("rbf", gamma=gamma), 1.0, 1e-14, method="cholesky")
    ex_a = np.array([float(v) for v in sol[:n]])
    assert np.abs(alpha - ex_a).max() <= 1e-12 * max(1.0, np.abs(ex_a).max())
    assert b == pytest.approx(float(sol[n]), abs=1e-12)


# ------------------------------------------------- worked example (P11) -----

def _read_fixture(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *rest = line.split()
            vals[key] = [float(Fraction(v)) for v in rest]
    return vals


def test_two_point_worked_example():
    fx = _read_fixture("n2_worked_example.txt")
    X = np.array(fx["x"])[:, None]
    y = np.array(fx["y"])
    C = fx["C"][0]
    for method in ("cholesky", "cg"):
        alpha, b, _ = O.train(X, y, O.KernelSpec("linear"), C, 1e-14, method=method)
        assert np.allclose(alpha, fx["alpha"], rtol=0, atol=1e-15)
        assert b == pytest.approx(fx["b"][0], abs=1e-15)
        f = O.decision(X, alpha, b, X, O.KernelSpec("linear"))
        assert np.allclose(f, fx["f"], rtol=0, atol=1e-15)


# --------------------------------------------------- special cases (P12) ----

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_equal_labels_and_single_point(spec):
    X, _ = small_problem(n=20, d=3)
    for lab in (1.0, -1.0):
        y = np.full(20, lab)
        alpha, b, info = O.train(X, y, spec, 1.0, 1e-8)
        assert np.all(alpha == 0.0) and b == lab and info["iterations"] == 0
    alpha, b, _ = O.train(X[:1], np.array([-1.0]), spec, 1.0, 1e-8)
    assert alpha.tolist() == [0.0] and b == -1.0


# ------------------------------------------- linear O(nd) matvec (P13) ------

@pytest.mark.parametrize("C", [1.0, 5.0])
def test_linear_matvec_factored(C):
    """Q~ p = P^T (X (X^T (P p)) + P p / C) for the linear kernel."""
    X, _ = small_problem(n=300, d=7)
    n = X.shape[0]
    p = np.random.default_rng(2).standard_normal(n - 1)
    Pp = np.concatenate([p, [-p.sum()]])
    v = X @ (X.T @ Pp) + Pp / C
    ref = v[:-1] - v[-1]
    Qt, _, _ = O.reduced_matrix(X, O.KernelSpec("linear"), C)
    assert np.abs(Qt @ p - ref).max() <= 1e-12 * np.abs(ref).max()
    rows = [0, 17, n - 2]
    assert np.allclose(O.matvec_rows(X, O.KernelSpec("linear"), C, p, rows), ref[rows],
                       rtol=1e-12, atol=1e-12)


# ------------------------------------------------ CG finite termination (P14)

@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.kind)
def test_cg_full_iterations_matches_cholesky(spec):
    X, y = small_problem(n=48, d=4)
    Qt, _, _ = O.reduced_matrix(X, spec, 1.0)
    rhs = O.reduced_rhs(y)
    xs = O.solve_cholesky(Qt, rhs)
    res = O.solve_cg(lambda v: Qt @ v, rhs, eps=1e-15, max_iter=47)
    assert np.abs(res.x - xs).max() <= 1e-9 * np.abs(xs).max()


def test_cg_residual_replacement_and_max_iter():
    """Ill-conditioned case (C = 100) that needs more than 50 iterations."""
    X, y = small_problem(n=300, d=10, seed=9)
    spec = O.KernelSpec("rbf", gamma=1.0)
    C = 100.0
    Qt, _, _ = O.reduced_matrix(X, spec, C)
    rhs = O.reduced_rhs(y)
    xs = O.solve_cholesky(Qt, rhs)
    res = O.solve_cg(lambda v: Qt @ v, rhs, eps=1e-10)
    assert res.converged and res.iterations > 50
    # a replaced residual counts an extra product each 50 iterations (+1 for the final check)
    assert res.n_matvec == res.iterations + res.iterations // 50
    assert res.true_rel_residual <= 1e-9
    assert np.linalg.norm(res.x - xs) <= C * np.linalg.norm(rhs - Qt @ res.x) * 1.01 + 1e-12
    short = O.solve_cg(lambda v: Qt @ v, rhs, eps=1e-10, max_iter=3)
    assert not short.converged and short.iterations == 3


def test_cg_runs_to_max_iter_without_progress():
    """An affine (not linear) operator keeps CG from converging. With the
    residual never recomputed, nothing but max_iter ends it; with the default
    recomputation every 50 iterations, the missing progress of the true
    residual ends it, unconverged, long before."""
    rng = np.random.default_rng(0)
    A = np.diag(np.linspace(1, 10, 30))
    z = rng.standard_normal(30)
    mv = lambda v: A @ v + 0.5 * z  # noqa: E731
    res = O.solve_cg(mv, np.ones(30), eps=1e-14, max_iter=500, replace_every=10**9)
    assert not res.converged and not res.stalled and res.iterations == 500
    assert len(res.history) == 500
    res = O.solve_cg(mv, np.ones(30), eps=1e-14, max_iter=500)
    assert not res.converged and res.stalled and res.iterations < 500
    assert res.iterations % 50 == 0


def _fp32_operator(n=200, kappa=1000.0, seed=1):
    """SPD A with eigenvalues spread evenly over [1, kappa] and a product
    rounded to float32: the computed true residual b - fl32(A x) cannot fall
    much below 2^-24 ||A x||, a floor far above eps = 1e-12."""
    rng = np.random.default_rng(seed)
    Qm, _ = np.linalg.qr(rng.standard_normal((n, n)))
    A = (Qm * np.linspace(1.0, kappa, n)) @ Qm.T
    A = 0.5 * (A + A.T)
    b = rng.standard_normal(n)
    return A, b, (lambda v: (A @ v).astype(np.float32).astype(np.float64))


def test_cg_stagnation_stops_at_the_attainable_floor():
    """eps = 1e-12 is out of reach of a float32 product. CG must stop
    unconverged within a few recomputations of the residual after reaching the
    floor (here: 50-150 iterations of progress, then at most two recomputations
    without a new minimum), not run to max_iter, and return the iterate whose
    recomputed residual was the smallest. kappa = 1000 keeps the recurrence
    residual from dropping below eps between two recomputations (a faster
    operator lets the recurrence reach eps first, a false convergence that the
    stop test on the recurrence cannot see)."""
    A, b, mv = _fp32_operator()
    res = O.solve_cg(mv, b, eps=1e-12, max_iter=5000)
    assert res.stalled and not res.converged and not res.breakdown
    assert res.iterations % 50 == 0 and 100 <= res.iterations <= 300
    # the returned iterate sits at the floor: its exact residual is a few 2^-24
    exact = np.linalg.norm(b - A @ res.x) / np.linalg.norm(b)
    assert exact <= 1e-6
    # and it is the best of the recomputed (true) residuals, each of which is
    # ||b - fl32(A x_k)||^2 at an iterate x_k
    refreshed = [res.history[k - 1] for k in range(50, res.iterations + 1, 50)]
    assert res.rel_residual ** 2 * float(b @ b) == pytest.approx(min(refreshed), rel=1e-12)
    assert res.true_rel_residual == pytest.approx(res.rel_residual, rel=1e-9)
    assert refreshed[-1] >= min(refreshed[:-1])      # the last one set no new minimum


def test_cg_stagnation_rule_leaves_slow_progress_alone():
    """kappa = 1e4 (eigenvalues spread geometrically), exact arithmetic: ~1000
    iterations. The true residual after 50 of them is above the initial one
    (CG's residual norm is not monotone), but the energy has fallen, and every
    later recomputation sets a new residual minimum: CG must converge as
    without the stagnation rule."""
    rng = np.random.default_rng(2)
    n = 400
    Qm, _ = np.linalg.qr(rng.standard_normal((n, n)))
    A = (Qm * np.geomspace(1.0, 1e4, n)) @ Qm.T
    A = 0.5 * (A + A.T)
    b = rng.standard_normal(n)
    res = O.solve_cg(lambda v: A @ v, b, eps=1e-10, max_iter=5000)
    assert res.converged and not res.stalled and res.iterations > 100
    assert np.linalg.norm(b - A @ res.x) <= 2e-10 * np.linalg.norm(b)
    assert res.history[49] > float(b @ b)        # the swing the energy vouches for
    plain = O.solve_cg(lambda v: A @ v, b, eps=1e-10, max_iter=5000, replace_every=10**9)
    assert abs(plain.iterations - res.iterations) <= 100


def test_cg_breakdown_on_an_indefinite_matrix_worked_example():
    """A = diag(3, 1, -1), b = (1, 1, 1), worked by hand. Iteration 1:
    d = b, d^T A d = 3, a = 1, x = (1, 1, 1), r = (-2, 0, 2), r^T r = 8,
    beta = 8/3, d = (2/3, 8/3, 14/3). Iteration 2: d^T A d = (12 + 64 - 196)/9
    = -120/9 <= 0, so CG stops there with x = (1, 1, 1)."""
    A = np.diag([3.0, 1.0, -1.0])
    b = np.ones(3)
    res = O.solve_cg(lambda v: A @ v, b, eps=1e-12)
    assert res.breakdown and not res.converged and not res.stalled
    assert res.iterations == 2
    np.testing.assert_array_equal(res.x, [1.0, 1.0, 1.0])
    res = O.solve_cg(lambda v: np.diag([1.0, -1.0]) @ v, np.ones(2), eps=1e-12)
    assert res.breakdown and res.iterations == 1     # d^T A d = 1 - 1 = 0
    np.testing.assert_array_equal(res.x, [0.0, 0.0])


def test_cg_matches_textbook_on_diagonal():
    """On a diagonal SPD matrix with k distinct eigenvalues CG ends in k steps."""
    A = np.diag([1.0] * 5 + [3.0] * 5 + [7.0] * 5)
    b = np.arange(1.0, 16.0)
    res = O.solve_cg(lambda v: A @ v, b, eps=1e-14)
    assert res.converged and res.iterations == 3
    assert np.allclose(res.x, b / np.diag(A), rtol=1e-13)


# ---------------------------------------------------------- predict ---------

def test_predict_tie_and_sign():
    X = np.array([[1.0], [-1.0]])
    f, lab = O.predict(X, np.array([0.5, 0.5]), 0.0, np.array([[0.0], [2.0], [-2.0]]),
                       O.KernelSpec("linear"))
    assert f.tolist() == [0.0, 0.0, 0.0] and lab.tolist() == [-1, -1, -1]
    f, lab = O.predict(X, np.array([1.0, -1.0]), 0.0, np.array([[0.5], [-0.5]]),
                       O.KernelSpec("linear"))
    assert lab.tolist() == [1, -1]


# ---------------------------------------------------- generator ------------

def test_generator_recipe():
    cfg = S.CONFIGS["linear_f64_4096x1024"]
    X, y, scale = S.make_train(cfg)
    assert X.shape == (4096, 1024) and X.dtype == np.float64 and X.flags.c_contiguous
    assert np.all(np.abs(y) == 1)
    assert X.min() == -1.0 and X.max() == 1.0
    assert np.allclose(X.min(axis=0), -1.0) and np.allclose(X.max(axis=0), 1.0)
    # 5% flips after a balanced draw
    X2, y2, _ = S.make_train(cfg)
    assert np.array_equal(X, X2) and np.array_equal(y, y2)
    assert abs(int((y > 0).sum()) - 2048) <= round(0.05 * 4096)
    Xt, yt = S.make_test(cfg, scale)
    assert Xt.shape == (1024, 1024)


# ---------------------------------------------------------------- cg_step ---

def test_cg_step_worked_example():
    """A = diag(2, 1), b = (1, 1), x0 = 0, worked by hand: gamma = 3, a = 2/3,
    x = (2/3, 2/3), r = (-1/3, 1/3), r^T r = 2/9, beta = 1/9, d = (-2/9, 4/9)."""
    A = np.diag([2.0, 1.0])
    b = np.array([1.0, 1.0])
    d = b.copy()
    x, r, d, rr, gamma, step, beta = O.cg_step(np.zeros(2), b, d, A @ d, float(b @ b))
    assert gamma == 3.0 and abs(step - 2 / 3) < 1e-16
    np.testing.assert_allclose(x, [2 / 3, 2 / 3], rtol=0, atol=1e-16)
    np.testing.assert_allclose(r, [-1 / 3, 1 / 3], rtol=0, atol=1e-16)
    assert abs(rr - 2 / 9) < 1e-16 and abs(beta - 1 / 9) < 1e-16
    np.testing.assert_allclose(d, [-2 / 9, 4 / 9], rtol=0, atol=1e-16)


def test_cg_step_textbook_properties():
    """Iterated steps: residuals mutually orthogonal, directions A-conjugate,
    r_k = b - A x_k, and the exact solution after n steps (finite termination)."""
    rng = np.random.default_rng(21)
    n = 12
    M = rng.standard_normal((n, n))
    A = M @ M.T + n * np.eye(n)
    b = rng.standard_normal(n)
    x, r, d = np.zeros(n), b.copy(), b.copy()
    rr = float(b @ b)
    rs, ds = [r.copy()], [d.copy()]
    for _ in range(n):
        x, r, d, rr, gamma, step, beta = O.cg_step(x, r, d, A @ d, rr)
        assert gamma > 0
        np.testing.assert_allclose(r, b - A @ x, rtol=0, atol=1e-10 * np.abs(b).max())
        rs.append(r.copy())
        ds.append(d.copy())
    R = np.array(rs[:n])
    D = np.array(ds[:n])
    G = R @ R.T
    off = G - np.diag(np.diag(G))
    assert np.abs(off).max() <= 1e-9 * np.abs(np.diag(G)).max()
    H = D @ A @ D.T
    off = H - np.diag(np.diag(H))
    assert np.abs(off).max() <= 1e-9 * np.abs(np.diag(H)).max()
    np.testing.assert_allclose(x, np.linalg.solve(A, b), rtol=1e-9, atol=1e-12)


def test_cg_step_breakdown_leaves_vectors():
    x, r = np.ones(3), np.full(3, 2.0)
    d = np.zeros(3)
    out = O.cg_step(x, r, d, np.zeros(3), 12.0)
    np.testing.assert_array_equal(out[0], x)
    np.testing.assert_array_equal(out[1], r)
    np.testing.assert_array_equal(out[2], d)
    assert out[3] == 12.0 and out[4] == 0.0 and out[6] == 0.0
    out = O.cg_step(x, r, np.ones(3), -np.ones(3), 12.0)       # negative curvature
    np.testing.assert_array_equal(out[0], x)
    assert out[4] == -3.0 and out[6] == 0.0


def test_cg_step_at_an_exact_solution_stays_finite():
    """r = 0 on entry (rr = 0): the step is 0 / d^T q = 0, nothing moves, and
    beta (0 / 0) is taken as 0, so d becomes r = 0 and no NaN appears."""
    x, d = np.array([1.0, -2.0, 3.0]), np.array([0.5, 0.25, -1.0])
    out = O.cg_step(x, np.zeros(3), d, 2.0 * d, 0.0)
    np.testing.assert_array_equal(out[0], x)
    np.testing.assert_array_equal(out[1], 0.0)
    np.testing.assert_array_equal(out[2], 0.0)
    assert out[3] == 0.0 and out[4] == 2.0 * float(d @ d) and out[5] == 0.0 and out[6] == 0.0


# ------------------------------------------------------------- warm start ---

def _spd_case(seed=31, n=40, d=6, C=1.0):
    rng = np.random.default_rng(seed)
    X = rng.uniform(-1, 1, (n, d))
    y = np.where(rng.random(n) < 0.5, 1.0, -1.0)
    spec = O.KernelSpec("rbf", gamma=0.5)
    Qt, q, Qmm = O.reduced_matrix(X, spec, C)
    return X, y, spec, Qt, O.reduced_rhs(y)


def test_warm_start_from_the_solution_takes_no_iteration():
    _, _, _, Qt, rhs = _spd_case()
    xs = np.linalg.solve(Qt, rhs)
    res = O.solve_cg(lambda v: Qt @ v, rhs, 1e-8, x0=xs)
    assert res.iterations == 0 and res.converged
    np.testing.assert_array_equal(res.x, xs)
    assert res.n_matvec == 1


def test_warm_start_from_zero_is_the_cold_start():
    _, _, _, Qt, rhs = _spd_case()
    cold = O.solve_cg(lambda v: Qt @ v, rhs, 1e-10)
    warm = O.solve_cg(lambda v: Qt @ v, rhs, 1e-10, x0=np.zeros_like(rhs))
    assert warm.iterations == cold.iterations
    np.testing.assert_array_equal(warm.x, cold.x)


def test_warm_start_meets_the_rigorous_bound():
    """From a random start CG still stops at ||r|| <= eps ||rhs|| (the stop test
    stays relative to the right-hand side), and ||x - x*|| <= C ||r|| (P9)."""
    C = 2.0
    _, _, _, Qt, rhs = _spd_case(C=C)
    xs = np.linalg.solve(Qt, rhs)
    x0 = np.random.default_rng(5).standard_normal(rhs.shape[0]) * 10
    res = O.solve_cg(lambda v: Qt @ v, rhs, 1e-9, x0=x0)
    assert res.converged and res.rel_residual <= 1e-9
    r = rhs - Qt @ res.x
    assert np.linalg.norm(res.x - xs) <= C * np.linalg.norm(r) * (1 + 1e-6)
    assert res.true_rel_residual <= 1e-8


def test_warm_start_with_zero_rhs_returns_zero():
    X, _, spec, Qt, _ = _spd_case()
    y = np.ones(X.shape[0])
    alpha, b, info = O.train(X, y, spec, 1.0, 1e-8, alpha0=np.ones(X.shape[0]))
    assert info["iterations"] == 0
    np.testing.assert_array_equal(alpha, 0.0)
    assert b == 1.0
