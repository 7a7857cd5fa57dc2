"""The parity rules of the GPU tests, each named for what it checks.

Contract bars (the same for every test): the implicit product within 1e-11
(fp64) / 1e-5 (fp32) and the solution within 1e-9 / 1e-4, as max-norm
relative errors; predicted labels identical. Everything below is either that
bar applied to one output, or a bound derived from the arithmetic, and says
which.

* ``alpha_tilde_error``: alpha~ (the N CG unknowns) against the oracle's CG at
  the same eps, normwise: the contract bar.
* ``bias_step_errors``: the bias step alone (Eqs. (11), (15)) on the GPU's own
  alpha~: alpha_m = -sum alpha~ and b = y_m + Q_mm sum alpha~ - q^T alpha~,
  each relative to its own size, against the oracle's recovery from the same
  alpha~: the contract bar, plus the fp64 rounding bound of the two sums
  where the result is much smaller than its terms (plus, in fp32, the
  rounding of each alpha~_i to fp32 on output, which the library's fp64 b
  does not see).
* ``p9_check``: the CG iterate against the exact solution: for the SPD
  reduced matrix lambda_min >= 1/C, so ||x - x*||_2 <= C ||rhs - Q~ x||_2
  with the residual formed by the oracle's explicit fp64 Q~, for the
  iterate and for the Cholesky solution the check compares it with (a
  rigorous bound, no tolerance), and the alpha_m and b it implies.
* ``label_check``: labels equal to the oracle's except at points whose label
  the solution difference itself can flip: |f_ref| <= |f_mix - f_ref| + the
  prediction bar, where f_mix is the oracle's decision value for the GPU's
  alpha and b. Such near-ties are counted and bounded by the caller.
"""
from __future__ import annotations

import numpy as np

import oracle as O

BAR_MV = {"f64": 1e-11, "f32": 1e-5}      # implicit product, max-norm relative
BAR_SOL = {"f64": 1e-9, "f32": 1e-4}      # alpha and b
U32 = 2.0 ** -24
U64 = 2.0 ** -53


def rel_to(delta, ref, scale):
    """|delta| relative to |ref|: the literal relative error. A reference that
    is zero up to rounding (|ref| <= 1e-6 scale, as b and alpha_m are for
    symmetric data) has no relative error; there delta is taken relative to
    scale (1 for b, the scale of f; max |alpha| for alpha_m)."""
    delta, ref = abs(float(delta)), abs(float(ref))
    if delta == 0.0:
        return 0.0
    return delta / (ref if ref > 1e-6 * scale else scale)


def rel_err(a, ref):
    """max |a - ref| / max |ref| (normwise, max norm)."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-300))


def alpha_tilde_error(alpha, ref_alpha):
    """Normwise error of the CG unknowns alpha~ = alpha[:-1], relative to max |alpha_ref|."""
    alpha = np.asarray(alpha, dtype=np.float64)
    ref_alpha = np.asarray(ref_alpha, dtype=np.float64)
    return float(np.abs(alpha[:-1] - ref_alpha[:-1]).max() / np.abs(ref_alpha).max())


def end_to_end_errors(alpha, b, ref_alpha, ref_b):
    """alpha_m and b against a reference solution, each relative to its own size
    (the literal reading), and b relative to max(1, |b|) (the scale of f)."""
    alpha = np.asarray(alpha, dtype=np.float64)
    ref_alpha = np.asarray(ref_alpha, dtype=np.float64)
    e_am = rel_to(alpha[-1] - ref_alpha[-1], ref_alpha[-1], np.abs(ref_alpha).max())
    e_b = rel_to(b - ref_b, ref_b, 1.0)
    e_bf = abs(b - ref_b) / max(1.0, abs(ref_b))
    return float(e_am), float(e_b), float(e_bf)


def bias_step_errors(alpha, b, y, q, Qmm, dtype):
    """The bias step on the GPU's own alpha~: (error of alpha_m, its tolerance,
    error of b, its tolerance), errors relative to |alpha_m| and |b|.

    Tolerance: the contract bar, plus the rounding of the two sums themselves
    where alpha_m or b is much smaller than their terms (both sides sum in
    fp64: the library a strided sum of ceil(N / 1024) terms per thread and a
    tree, the oracle pairwise; together below (ceil(N / 1024) + 40) u64 times
    the sum of the terms' magnitudes), plus in fp32 the effect of rounding each
    alpha~_i to fp32 on output (|delta alpha~_i| <= 2^-24 |alpha~_i|; the
    library forms alpha_m and b from its fp64 iterate): sum |alpha~_i| u32 for
    alpha_m (and u32 |alpha_m| for its own rounding), sum |Q_mm - q_i|
    |alpha~_i| u32 for b."""
    alpha = np.asarray(alpha, dtype=np.float64)
    ref_alpha, ref_b = O.recover(alpha[:-1], y, q, Qmm)
    bar = BAR_SOL[dtype]
    at = np.abs(alpha[:-1])
    sa = max(float(np.abs(ref_alpha).max()), 1e-300)
    e_am = rel_to(alpha[-1] - ref_alpha[-1], ref_alpha[-1], sa)
    e_b = rel_to(b - ref_b, ref_b, 1.0)
    tol_am, tol_b = bar, bar
    n_sum = (-(-at.shape[0] // 1024) + 40) * U64
    den_am64 = abs(ref_alpha[-1]) if abs(ref_alpha[-1]) > 0 else sa
    den_b64 = abs(ref_b) if abs(ref_b) > 0 else 1.0
    tol_am += n_sum * float(at.sum()) / den_am64
    tol_b += n_sum * (abs(Qmm) * float(at.sum()) + float(np.abs(q) @ at)) / den_b64
    if dtype == "f32":
        den_am = abs(ref_alpha[-1]) if abs(ref_alpha[-1]) > 1e-6 * sa else sa
        den_b = abs(ref_b) if abs(ref_b) > 1e-6 else 1.0
        tol_am += U32 * (at.sum() + abs(ref_alpha[-1])) / den_am
        tol_b += U32 * float(np.abs(Qmm - q) @ at) / den_b
    return float(e_am), float(tol_am), float(e_b), float(tol_b)


def p9_check(alpha, b, Qt, q, Qmm, rhs, C, x_exact, b_exact):
    """Rigorous distance of the GPU's solution to the exact one.

    ||alpha~ - x*||_2 <= C ||rhs - Q~ alpha~||_2 because lambda_min(Q~) >= 1/C
    (Q~ = P^T Q P with Q >= I/C and P^T P = I + 1 1^T >= I). The reference
    x_exact is the Cholesky solution, itself within C ||rhs - Q~ x_exact||_2 of
    x* by the same bound (which matters where Q~ is ill-conditioned), so the
    distance between the two is below the sum D of both bounds. It implies
    |alpha_m - alpha_m*| <= sqrt(N) D and |b - b*| <= (|Q_mm| sqrt(N) + ||q||_2) D
    (Eqs. (11), (15) are linear in alpha~). Returns the distances, their
    bounds and the relative residual ||r|| / ||rhs||."""
    alpha = np.asarray(alpha, dtype=np.float64)
    at = alpha[:-1]
    N = at.shape[0]
    r = rhs - Qt @ at
    r_exact = rhs - Qt @ x_exact[:N]
    D = C * (float(np.linalg.norm(r)) + float(np.linalg.norm(r_exact)))
    slack = 1e-12 * (float(np.linalg.norm(x_exact)) + 1.0)   # rounding of the residuals
    dist = float(np.linalg.norm(at - x_exact[:N]))
    d_am = abs(alpha[-1] - (-float(x_exact[:N].sum())))
    d_b = abs(b - b_exact)
    bound_am = np.sqrt(N) * (D + slack)
    bound_b = (abs(Qmm) * np.sqrt(N) + float(np.linalg.norm(q))) * (D + slack)
    return {"dist": dist, "bound": D + slack, "d_am": d_am, "bound_am": float(bound_am),
            "d_b": d_b, "bound_b": float(bound_b),
            "rel_res": float(np.linalg.norm(r) / np.linalg.norm(rhs))}


def label_check(labels, f_ref, f_mix, dtype):
    """(mismatches outside the near-ties, near-ties, widest band): a point is a
    near-tie when |f_ref| <= |f_mix - f_ref| + tol, f_mix being the oracle's
    decision value for the GPU's alpha and b, tol the prediction bar (10 x the
    product bar, times max(1, max |f_ref|))."""
    labels = np.asarray(labels)
    f_ref = np.asarray(f_ref, dtype=np.float64)
    f_mix = np.asarray(f_mix, dtype=np.float64)
    tol = 10 * BAR_MV[dtype] * max(1.0, float(np.abs(f_ref).max()))
    band = np.abs(f_mix - f_ref) + tol
    tie = np.abs(f_ref) <= band
    lab_ref = np.where(f_ref > 0, 1, -1)
    bad = (labels != lab_ref) & ~tie
    return int(bad.sum()), int(tie.sum()), float(band.max())
