"""CPU checks of the GPU tests' parity rules themselves (tests/parity_rules.py):
each accepts an exact or well-converged answer and rejects one with a planted
error just above what it allows."""
from __future__ import annotations

import numpy as np

import oracle as O
from parity_rules import bias_step_errors, p9_check


def _system(n=60, d=5, C=10.0, seed=3):
    rng = np.random.default_rng(seed)
    X = rng.uniform(-1, 1, (n, d))
    y = np.where(rng.uniform(size=n) < 0.5, 1.0, -1.0)
    Qt, q, Qmm = O.reduced_matrix(X, O.KernelSpec("linear"), C)
    rhs = O.reduced_rhs(y)
    return X, y, Qt, q, Qmm, rhs, C


def test_p9_accepts_cg_and_rejects_an_inconsistent_bias():
    """The distance bound holds for any iterate (lambda_min(Q~) >= 1/C); what
    the check can fail on is an alpha_m or b that does not follow from the
    iterate by Eqs. (11), (15), or a reference that is not the exact solution
    to within its own residual."""
    X, y, Qt, q, Qmm, rhs, C = _system()
    xs = O.solve_cholesky(Qt, rhs)
    _, b_s = O.recover(xs, y, q, Qmm)
    res = O.solve_cg(lambda v: Qt @ v, rhs, 1e-6)
    alpha, b = O.recover(res.x, y, q, Qmm)
    r = p9_check(alpha, b, Qt, q, Qmm, rhs, C, xs, b_s)
    assert r["dist"] <= r["bound"] and r["d_am"] <= r["bound_am"] and r["d_b"] <= r["bound_b"]
    rb = p9_check(alpha, b + 2 * r["bound_b"], Qt, q, Qmm, rhs, C, xs, b_s)
    assert rb["d_b"] > rb["bound_b"]
    a2 = alpha.copy()
    a2[-1] += 2 * r["bound_am"]
    ra = p9_check(a2, b, Qt, q, Qmm, rhs, C, xs, b_s)
    assert ra["d_am"] > ra["bound_am"]
    # a perturbed reference is still accepted only within its own residual
    rr = p9_check(alpha, b, Qt, q, Qmm, rhs, C, xs + 1e-3, b_s)
    assert rr["bound"] >= r["bound"]


def test_bias_step_accepts_its_own_recovery_and_rejects_a_shifted_b():
    X, y, Qt, q, Qmm, rhs, C = _system()
    xs = O.solve_cholesky(Qt, rhs)
    alpha, b = O.recover(xs, y, q, Qmm)
    e_am, t_am, e_b, t_b = bias_step_errors(alpha, b, y, q, Qmm, "f64")
    assert e_am <= t_am and e_b <= t_b
    assert t_b < 1e-8                  # well-conditioned sums: close to the bar
    shifted = b + 10 * t_b * abs(b)
    _, _, e_b2, t_b2 = bias_step_errors(alpha, shifted, y, q, Qmm, "f64")
    assert e_b2 > t_b2
    a2 = alpha.copy()
    a2[-1] += 10 * t_am * abs(alpha[-1])
    e_am2, t_am2, _, _ = bias_step_errors(a2, b, y, q, Qmm, "f64")
    assert e_am2 > t_am2
