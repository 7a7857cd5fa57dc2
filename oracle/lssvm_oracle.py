"""CPU oracle for LS-SVM training by the reduced system (test infrastructure).

THIS IS TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT. Only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it. It shares
no code with the HIP path and never calls it.

Everything is plain NumPy/SciPy in float64. Inputs given in float32 are
upcast exactly before any arithmetic. Each function follows one passage of
the paper (arXiv 2202.12674); section and equation numbers refer to it:

* Sec. II-E, kernel table: linear <x,y>, polynomial (gamma<x,y> + r)^deg,
  radial exp(-gamma ||x - y||^2).
* Sec. II-F, Eq. (11): the bordered system [Q 1; 1^T 0][alpha; b] = [y; 0]
  with Q_ij = k(x_i, x_j) + delta_ij / C.
* Sec. II-F, Eqs. (12)-(13): partition of Q around the last point m and the
  reduced matrix Q~ = Qbar - 1 q^T - q 1^T + Q_mm 1 1^T.
* Sec. II-F, Eq. (14): the reduced system Q~ alpha~ = ybar - y_m 1.
* Sec. II-F, Eq. (15): b = y_m + Q_mm <1, alpha~> - <q, alpha~>.
* Sec. III-B: Q~ is symmetric positive definite, solved by conjugate
  gradients (a variant of Shewchuk's method); Eq. (16) writes one entry of
  Q~ out in terms of kernel values.
* Sec. II-E, Eq. (10): the decision function, here without the y_i factor
  because the LS-SVM alpha already carries the sign (w = sum alpha_i Phi(x_i),
  Eq. (15)).

Readings where the paper leaves a choice (each is also listed with the
design notes of the repository):
* the pivot m is the last point (Eq. (12) puts q in the last row/column);
* CG starts at x = 0 and stops when r^T r <= eps^2 r0^T r0 (relative
  residual eps, Sec. IV-B and IV-F) or, unconverged, after max_iter
  iterations (default N); the residual is recomputed as rhs - Q~ x every
  50th iteration (Shewchuk's recommendation);
* an eps below what the arithmetic can reach ends CG early: at each of those
  recomputations either the true residual or the CG energy
  phi(x) = x^T Q~ x / 2 - rhs^T x (which CG lowers at every step in exact
  arithmetic) must set a new minimum, else CG stops, unconverged, with the
  iterate of the smallest recomputed residual (Sec. III-B names only "a
  variant of Shewchuk"; Sec. IV-F shows such a floor);
* CG stops on curvature breakdown, d^T Q~ d <= 0 or a non-finite step (Q~ is
  SPD for every kernel of Sec. II-E with coef0 >= 0; a negative coef0 can make
  it indefinite), with the iterate before that step;
* the decision label is +1 iff f(x) > 0.

Pins (see tests/test_oracle_pins.py): every function here is checked against
identities, closed forms, exact rational solves or textbook routines that do
not reuse its own formulas. No function is "parity unpinned".
"""
from __future__ import annotations

import dataclasses

import numpy as np
import scipy.linalg as sla

__all__ = [
    "KernelSpec", "kernel_matrix", "kernel_rows", "bordered_matrix",
    "reduced_parts", "reduced_matrix", "reduced_rows", "reduced_rhs", "matvec_dense",
    "matvec_rows", "solve_cholesky", "CGResult", "solve_cg", "cg_step", "recover",
    "train", "decision", "predict", "full_system_residual",
]


@dataclasses.dataclass(frozen=True)
class KernelSpec:
    """Kernel function of Sec. II-E with its parameters."""
    kind: str               # "linear", "poly" or "rbf"
    gamma: float = 1.0
    coef0: float = 0.0      # the polynomial's r
    degree: int = 1         # the polynomial's exponent


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def _kernel_from_gram_(G, na, nb, spec: KernelSpec):
    """Kernel values from inner products G = A B^T, overwriting G.

    na, nb are the squared norms of the rows of A and B (radial kernel only).
    Sec. II-E: the radial kernel's ||x - y||^2 is expanded as
    ||x||^2 + ||y||^2 - 2<x, y> and clipped at 0 against rounding.
    """
    if spec.kind == "linear":
        return G
    if spec.kind == "poly":
        G *= spec.gamma
        G += spec.coef0
        np.power(G, spec.degree, out=G)
        return G
    if spec.kind == "rbf":
        G *= -2.0
        G += na[:, None]
        G += nb[None, :]
        np.maximum(G, 0.0, out=G)
        G *= -spec.gamma
        np.exp(G, out=G)
        return G
    raise ValueError(f"unknown kernel {spec.kind!r}")


def _sqnorms(A):
    return np.einsum("ij,ij->i", A, A)


def _gemm_nt(A, B):
    """A @ B^T as a general matrix product.

    numpy routes ``a @ a.T`` on one buffer to a symmetric rank-k update;
    OpenBLAS 0.3.29's dsyrk returns wrong entries at n = 32768, d = 4096, so
    aliasing operands are separated first.
    """
    if np.shares_memory(A, B):
        B = B.copy()
    return A @ B.T


def kernel_rows(XA, XB, spec: KernelSpec):
    """k(a_i, b_j) for every row a_i of XA and b_j of XB (Sec. II-E)."""
    A, B = _f64(XA), _f64(XB)
    G = _gemm_nt(A, B)
    if spec.kind == "rbf":
        return _kernel_from_gram_(G, _sqnorms(A), _sqnorms(B), spec)
    return _kernel_from_gram_(G, None, None, spec)


def _mirror_upper_(G, bs: int = 1024):
    """Copy the upper triangle of square G onto its lower triangle, in place."""
    n = G.shape[0]
    for j0 in range(0, n, bs):
        j1 = min(n, j0 + bs)
        # rows below the diagonal block receive the transpose of the strip above
        G[j1:, j0:j1] = G[j0:j1, j1:].T
        blk = G[j0:j1, j0:j1]
        il = np.tril_indices(j1 - j0, -1)
        blk[il] = blk.T[il]
    return G


def kernel_matrix(X, spec: KernelSpec, panel: int = 2048):
    """Symmetric n x n kernel matrix K_ij = k(x_i, x_j) (Sec. II-E).

    Row panels of the upper triangle come from general matrix products, get
    the kernel map, and are mirrored, so K is exactly symmetric. One n x n
    buffer plus one panel.
    """
    A = _f64(X)
    B = A.copy()                 # a separate operand: always a general product
    n = A.shape[0]
    nrm = _sqnorms(A) if spec.kind == "rbf" else None
    K = np.empty((n, n))
    for i0 in range(0, n, panel):
        i1 = min(n, i0 + panel)
        blk = A[i0:i1] @ B[i0:].T
        if spec.kind == "rbf":
            _kernel_from_gram_(blk, nrm[i0:i1], nrm[i0:], spec)
        else:
            _kernel_from_gram_(blk, None, None, spec)
        K[i0:i1, i0:] = blk
    del B
    _mirror_upper_(K)
    return K


def bordered_matrix(X, spec: KernelSpec, C: float):
    """The (n+1) x (n+1) matrix of Eq. (11): [Q 1; 1^T 0], Q = K + I/C."""
    K = kernel_matrix(X, spec)
    n = K.shape[0]
    M = np.zeros((n + 1, n + 1))
    M[:n, :n] = K + np.eye(n) / C
    M[:n, n] = 1.0
    M[n, :n] = 1.0
    return M


def reduced_parts(X, spec: KernelSpec, C: float):
    """Eq. (12): Q = K + I/C split around the last point m = n-1.

    Returns (Qbar, q, Q_mm) with Qbar = Q[:N, :N], q = Q[:N, m] and
    Q_mm = Q[m, m] = k(x_m, x_m) + 1/C, where N = n - 1.
    """
    K = kernel_matrix(X, spec)
    n = K.shape[0]
    Q = K
    Q[np.diag_indices(n)] += 1.0 / C
    N = n - 1
    return Q[:N, :N], Q[:N, N].copy(), float(Q[N, N])


def reduced_matrix(X, spec: KernelSpec, C: float):
    """Eq. (13): Q~ = Qbar - 1 q^T - q 1^T + Q_mm 1 1^T, returned with q and Q_mm.

    Built in place on the kernel matrix to keep one n x n buffer.
    """
    Qbar, q, Qmm = reduced_parts(X, spec, C)
    Qt = Qbar                      # view into the n x n buffer (row stride n)
    N = Qt.shape[0]
    bs = 1024
    for i0 in range(0, N, bs):     # row blocks keep the temporaries small
        i1 = min(N, i0 + bs)
        # subtract (q_i + q_j) as one symmetric term so that Q~ stays exactly symmetric
        Qt[i0:i1] -= q[i0:i1, None] + q[None, :]
        Qt[i0:i1] += Qmm
    return Qt, q, Qmm


def reduced_rows(X, spec: KernelSpec, C: float, rows):
    """Selected rows of Q~ (Eq. (13)) without forming the whole matrix.

    Q~[r, j] = K[r, j] + delta_rj / C - (q_r + q_j) + Q_mm for j < N, with
    q_j = k(x_j, x_m) and Q_mm = k(x_m, x_m) + 1/C as in Eq. (12).
    """
    X = _f64(X)
    rows = np.asarray(rows, dtype=np.int64)
    n = X.shape[0]
    N = n - 1
    xm = X[N:N + 1]
    q = kernel_rows(X[:N], xm, spec)[:, 0]
    Qmm = float(kernel_rows(xm, xm, spec)[0, 0]) + 1.0 / C
    R = kernel_rows(X[rows], X[:N], spec)
    R[np.arange(len(rows)), rows] += 1.0 / C
    R -= q[rows][:, None] + q[None, :]
    R += Qmm
    return R


def reduced_rhs(y):
    """Eq. (14): right-hand side ybar - y_m 1 (ybar = first N labels)."""
    y = _f64(y)
    return y[:-1] - y[-1]


def matvec_dense(Qt, p):
    """Q~ p with the explicit matrix."""
    return Qt @ _f64(p)


def matvec_rows(X, spec: KernelSpec, C: float, p, rows):
    """(Q~ p)_i for selected rows i, one explicit row of Q~ at a time.

    Row i of Q~ is written out entry by entry as Eq. (16) has it:
    k(x_i, x_j) + delta_ij / C - k(x_m, x_j) - k(x_i, x_m) + k(x_m, x_m) + 1/C,
    for j < N = n - 1.
    """
    X = _f64(X)
    p = _f64(p)
    n = X.shape[0]
    N = n - 1
    xm = X[N:N + 1]
    k_mj = kernel_rows(xm, X[:N], spec)[0]          # k(x_m, x_j), j < N
    k_mm = float(kernel_rows(xm, xm, spec)[0, 0])
    out = np.empty(len(rows))
    for t, i in enumerate(rows):
        k_ij = kernel_rows(X[i:i + 1], X[:N], spec)[0]
        k_im = float(kernel_rows(X[i:i + 1], xm, spec)[0, 0])
        row = k_ij - k_mj - k_im + k_mm + 1.0 / C
        row[i] += 1.0 / C
        out[t] = row @ p
    return out


def solve_cholesky(Qt, rhs):
    """Direct solve of Eq. (14) by Cholesky (valid because Q~ is SPD, Sec. III-B)."""
    c = sla.cho_factor(Qt, lower=True, check_finite=False)
    return sla.cho_solve(c, _f64(rhs), check_finite=False)


@dataclasses.dataclass
class CGResult:
    x: np.ndarray
    iterations: int
    converged: bool
    rel_residual: float          # sqrt(delta / delta0) (recurrence; a true one on a stall)
    true_rel_residual: float     # ||rhs - Q~ x|| / ||rhs||
    n_matvec: int
    history: list                # delta after every iteration
    stalled: bool = False        # stopped: no new minimum of the true residual
    breakdown: bool = False      # stopped: d^T Q~ d <= 0 or a non-finite step


def solve_cg(matvec, rhs, eps: float, max_iter: int = 0,
             replace_every: int = 50, x0=None) -> CGResult:
    """Conjugate gradients for the SPD reduced system (Sec. III-B).

    matvec(v) returns Q~ v. Steps per iteration, in Shewchuk's notation:
    q = A d; alpha = delta / d^T q; x += alpha d; r -= alpha q (or r = b - A x
    every ``replace_every`` iterations); delta_new = r^T r; stop once
    delta_new <= eps^2 delta_0; beta = delta_new / delta_old; d = r + beta d.

    Two more ways to stop, both unconverged:
    * stagnation: at every recomputed residual (a true residual) that has not
      met eps, progress is a new minimum of either delta_new = r^T r or the
      energy phi = x^T A x / 2 - b^T x = -(b + r)^T x / 2 over the start and
      the earlier recomputations. Without progress x returns to the iterate of
      the smallest recomputed delta. In exact arithmetic phi falls at every
      step (by (r^T r)^2 / (2 d^T A d)), so it vouches for progress while the
      residual norm still swings; once phi's changes are below its rounding
      (near eps ~ sqrt(u)) the residual has to fall. At a floor of the
      arithmetic neither does, and CG ends a few recomputations later.
    * breakdown: d^T q <= 0 or a non-finite alpha (an indefinite operator);
      x is the iterate before that step and ``iterations`` counts the step
      that found it.

    x0 (optional) is a starting iterate: r = b - A x0 (one product). delta_0
    stays b^T b, so the stop test is relative to the right-hand side wherever
    CG starts. A zero right-hand side returns x = 0 whatever x0 is.
    """
    b = _f64(rhs)
    N = b.shape[0]
    if max_iter <= 0:
        max_iter = N
    x = np.zeros(N)
    r = b.copy()
    delta0 = float(b @ b)
    hist = []
    nmv = 0
    if delta0 == 0.0:
        return CGResult(x, 0, True, 0.0, 0.0, 0, hist)
    if x0 is not None:
        x = _f64(x0).copy()
        r = b - matvec(x)
        nmv += 1
    d = r.copy()
    delta = float(r @ r)
    if delta <= eps * eps * delta0:
        true_res = float(np.linalg.norm(b - matvec(x)) / np.linalg.norm(b))
        return CGResult(x, 0, True, float(np.sqrt(delta / delta0)), true_res, nmv, hist)
    best_delta, best_x = delta, x.copy()    # the start's residual is a true one
    best_phi = -0.5 * float((b + r) @ x)
    converged = stalled = broke = False
    it = 0
    while it < max_iter:
        it += 1
        q = matvec(d)
        nmv += 1
        curv = float(d @ q)
        with np.errstate(divide="ignore", invalid="ignore"):
            alpha = float(np.float64(delta) / np.float64(curv))
        if not (curv > 0.0) or not np.isfinite(alpha):
            broke = True
            break
        x += alpha * d
        refresh = it % replace_every == 0
        if refresh:
            r = b - matvec(x)
            nmv += 1
        else:
            r -= alpha * q
        delta_old = delta
        delta = float(r @ r)
        hist.append(delta)
        if delta <= eps * eps * delta0:
            converged = True
            break
        if refresh:
            phi = -0.5 * float((b + r) @ x)
            progress = False
            if delta < best_delta:
                best_delta, best_x = delta, x.copy()
                progress = True
            if phi < best_phi:
                best_phi = phi
                progress = True
            if not progress:
                stalled = True
                x, delta = best_x, best_delta
                break
        d = r + (delta / delta_old) * d
    true_res = float(np.linalg.norm(b - matvec(x)) / np.linalg.norm(b))
    return CGResult(x, it, converged, float(np.sqrt(delta / delta0)), true_res, nmv, hist,
                    stalled, broke)


def cg_step(x, r, d, q, rr):
    """One CG iteration given q = A d (Sec. III-B, the steps of solve_cg without
    the product and the stop test): returns x, r, d, r^T r, d^T q, step, beta.
    On curvature breakdown (d^T q <= 0 or a non-finite step) the vectors are
    returned unchanged with r^T r kept and beta = 0. At an exact solution
    (rr = 0 on entry, so r = 0) the ratio defining beta is 0 / 0; beta is taken
    as 0, which restarts the direction at r."""
    x, r, d, q = (_f64(v).copy() for v in (x, r, d, q))
    gamma = float(d @ q)
    with np.errstate(divide="ignore", invalid="ignore"):
        step = float(np.float64(rr) / np.float64(gamma))
    if not (gamma > 0.0) or not np.isfinite(step):
        return x, r, d, float(rr), gamma, step, 0.0
    x += step * d
    r -= step * q
    rr_new = float(r @ r)
    beta = rr_new / rr if rr != 0.0 else 0.0
    d = r + beta * d
    return x, r, d, rr_new, gamma, step, beta


def recover(alpha_t, y, q, Qmm):
    """Full alpha and bias from the reduced solution.

    alpha_m = -sum(alpha~) is the last row of Eq. (11) (sum of alpha = 0);
    b follows Eq. (15).
    """
    a = _f64(alpha_t)
    y = _f64(y)
    s = float(a.sum())
    alpha = np.concatenate([a, [-s]])
    b = float(y[-1] + Qmm * s - q @ a)
    return alpha, b


def train(X, y, spec: KernelSpec, C: float, eps: float, max_iter: int = 0,
          method: str = "cg", alpha0=None):
    """Solve the LS-SVM for (alpha, b, info) by the reduced route of Sec. II-F.

    method "cg" follows Sec. III-B; "cholesky" is the direct dense solve.
    alpha0 (optional, "cg" only): CG starts from its first n - 1 entries.
    """
    X = _f64(X)
    y = _f64(y)
    n = X.shape[0]
    if n == 1:
        return np.zeros(1), float(y[0]), {"iterations": 0, "converged": True}
    Qt, q, Qmm = reduced_matrix(X, spec, C)
    rhs = reduced_rhs(y)
    if method == "cholesky":
        at = solve_cholesky(Qt, rhs)
        info = {"iterations": 0, "converged": True}
    elif method == "cg":
        x0 = None if alpha0 is None else _f64(alpha0)[:-1]
        res = solve_cg(lambda v: Qt @ v, rhs, eps, max_iter, x0=x0)
        at = res.x
        info = dataclasses.asdict(res)
        del info["x"]
    else:
        raise ValueError(method)
    alpha, b = recover(at, y, q, Qmm)
    return alpha, b, info


def decision(X_train, alpha, b, X_test, spec: KernelSpec):
    """f(x) = sum_i alpha_i k(x_i, x) + b (Eq. (10) with alpha carrying the sign)."""
    K = kernel_rows(X_test, X_train, spec)
    return K @ _f64(alpha) + float(b)


def predict(X_train, alpha, b, X_test, spec: KernelSpec):
    """Scores and labels: +1 iff f(x) > 0, else -1."""
    f = decision(X_train, alpha, b, X_test, spec)
    return f, np.where(f > 0.0, 1, -1).astype(np.int32)


def full_system_residual(X, y, spec: KernelSpec, C: float, alpha, b):
    """Residual of Eq. (11) for a given (alpha, b): M [alpha; b] - [y; 0]."""
    M = bordered_matrix(X, spec, C)
    v = np.concatenate([_f64(alpha), [float(b)]])
    rhs = np.concatenate([_f64(y), [0.0]])
    return M @ v - rhs
