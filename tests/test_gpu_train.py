"""GPU parity of training (Sec. II-F, Eqs. (11)-(15); CG of Sec. III-B)
against the CPU oracle on the same seeded inputs, by the named rules of
parity_rules.py (applied in gpu_common.check_train): alpha~ within the
contract bar of the oracle's CG, the bias step pinned on the GPU's own alpha~,
the rigorous distance to the Cholesky solution where the reduced matrix fits
in memory, labels equal up to near-ties the solution difference can flip.
The fp64 workloads are also trained at a tighter eps where the oracle's CG
agrees with itself far below 1e-9, and there alpha~, alpha_m and b must each
meet 1e-9 relative to their own size."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
import synthdata as S
from gpu_common import (GOLDEN, TOL_ALPHA, TOL_MV, SPLIT_SHAPES, TAIL_SHAPES, check_train,  # noqa: F401
                        fp32_sensitivity,
                        data_of, golden, golden_tight, kw_of, labels_match, log, oracle_ref,
                        random_cases, random_large_cases, random_param_train_cases, rel_err,
                        small_cfg, spec_of,
                        to_dev)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,n,d,plan", [SPLIT_SHAPES[2], SPLIT_SHAPES[7]])
def test_train_linear_feature_split(torch_dev, dtype, n, d, plan):
    """Trainings whose products split the features, with a finer-split last
    round. The fp32 system's alpha~ tolerance follows its sensitivity to the
    rounding of the kernel values (as in test_train_random_shapes)."""
    torch, dev = torch_dev
    cfg = small_cfg("linear", dtype, n, d, C=1.0)
    X, y, Xte, _ = data_of(cfg)
    ref = oracle_ref(cfg, X, y)
    f_te = O.decision(X, ref.alpha, ref.b, Xte, spec_of(cfg))
    sens = fp32_sensitivity(X, cfg) if dtype == "f32" else 0.0
    tol = max(TOL_ALPHA[dtype], 0.1 * sens)
    log(f"  {cfg.name}: kappa u32 <= {sens:.1e}, alpha~ tolerance {tol:.1e}")
    check_train(torch, dev, cfg, ref, X, y, Xte, f_te, alpha_tol=tol)


@pytest.mark.parametrize("dtype,kernel,n,d,plan", [TAIL_SHAPES[2], TAIL_SHAPES[3]])
def test_train_tail_split(torch_dev, dtype, kernel, n, d, plan):
    torch, dev = torch_dev
    cfg = small_cfg(kernel, dtype, n, d, C=1.0)
    X, y, Xte, _ = data_of(cfg)
    ref = oracle_ref(cfg, X, y)
    f_te = O.decision(X, ref.alpha, ref.b, Xte, spec_of(cfg))
    check_train(torch, dev, cfg, ref, X, y, Xte, f_te)


@pytest.mark.parametrize("kernel,dtype", [("linear", "f64"), ("rbf", "f32")])
def test_train_wide(torch_dev, kernel, dtype):
    """300 points with 16384 features: the solution, bias and test labels
    against the oracle's CG."""
    torch, dev = torch_dev
    cfg = small_cfg(kernel, dtype, 300, 16384)
    log(f"train wide {cfg.name}")
    X, y, scale = S.make_train(cfg)
    Xte, _ = S.make_test(cfg, scale, n_test=200)
    ref = oracle_ref(cfg, X, y)
    f_te = O.decision(X, ref.alpha, ref.b, Xte, spec_of(cfg))
    check_train(torch, dev, cfg, ref, X, y, Xte, f_te)


@pytest.mark.parametrize("kernel,dtype,n,d,C", [random_cases()[k] for k in (0, 4, 8, 13, 17, 21)])
def test_train_random_shapes(torch_dev, kernel, dtype, n, d, C):
    """Every rule of check_train, the rigorous distance to the Cholesky
    solution included. The alpha~ bar is the contract's wherever fp32 can
    resolve the solution to it. Rounding the kernel values to fp32 perturbs Q~
    relatively by some rho, which moves the solution by up to kappa(Q~) rho
    (first-order perturbation); over 120 random trainings rho stayed below
    0.025 u32 (kappa bounded above as in fp32_sensitivity), so where
    0.1 kappa u32 exceeds the bar that is the alpha~ tolerance (a 4x margin),
    and the labels and the P9 bound still apply in full."""
    torch, dev = torch_dev
    cfg = small_cfg(kernel, dtype, n, d, C=C)
    X, y, Xte, _ = data_of(cfg)
    ref = oracle_ref(cfg, X, y)
    f_te = O.decision(X, ref.alpha, ref.b, Xte, spec_of(cfg))
    sens = fp32_sensitivity(X, cfg) if dtype == "f32" else 0.0
    tol = max(TOL_ALPHA[dtype], 0.1 * sens)
    log(f"  {cfg.name} C={C}: kappa u32 <= {sens:.1e}, alpha~ tolerance {tol:.1e}")
    check_train(torch, dev, cfg, ref, X, y, Xte, f_te, alpha_tol=tol)


@pytest.mark.parametrize("kernel,dtype,n,d,C,kp", random_param_train_cases())
def test_train_random_params(torch_dev, kernel, dtype, n, d, C, kp):
    """Every rule of check_train on trainings with random kernel parameters,
    the fp32 alpha~ tolerance as in test_train_random_shapes."""
    torch, dev = torch_dev
    cfg = S.Config(f"{kernel}_{dtype}_{n}x{d}", dtype, kernel, n, d, mu=1.0, inf_frac=0.5,
                   flip_frac=0.05, C=C, eps=1e-10 if dtype == "f64" else 1e-5, **kp)
    X, y, Xte, _ = data_of(cfg)
    ref = oracle_ref(cfg, X, y)
    f_te = O.decision(X, ref.alpha, ref.b, Xte, spec_of(cfg))
    sens = fp32_sensitivity(X, cfg) if dtype == "f32" else 0.0
    tol = max(TOL_ALPHA[dtype], 0.1 * sens)
    log(f"  {cfg.name} C={C:.3g} {kp}: kappa u32 <= {sens:.1e}, alpha~ tolerance {tol:.1e}")
    check_train(torch, dev, cfg, ref, X, y, Xte, f_te, alpha_tol=tol)


@pytest.mark.parametrize("dtype", ["f64", "f32"])
@pytest.mark.parametrize("kernel", ["linear", "poly", "rbf"])
@pytest.mark.parametrize("n,d", [(2, 3), (130, 7), (600, 50)])
def test_train_small(torch_dev, dtype, kernel, n, d):
    """Small trainings. With two points f is a difference of two kernel values
    plus b, ~1e-8 at many test points, below what fp32 resolves: those labels
    are undetermined, so the near-tie count is not bounded there."""
    torch, dev = torch_dev
    cfg = small_cfg(kernel, dtype, n, d, C=1.0)
    X, y, Xte, _ = data_of(cfg)
    ref = oracle_ref(cfg, X, y)
    f_te = O.decision(X, ref.alpha, ref.b, Xte, spec_of(cfg))
    check_train(torch, dev, cfg, ref, X, y, Xte, f_te, max_ties=len(Xte) if n == 2 else None)


@pytest.mark.parametrize("n,d,C", [(962, 64, 22.3), (968, 76, 22.5), (606, 74, 10.3)])
def test_train_fp32_linear_one_operator(torch_dev, n, d, C):
    """Small fp32 linear trainings with d < n and large C (Q~ ill-conditioned):
    fp32 CG reaches eps only if its residual recomputations apply the same
    rounded operator as its iterations. These shapes stalled (or took 2-17x the
    oracle's iterations) when the one-launch iterations split the tiles into
    single feature blocks and the recomputations did not."""
    torch, dev = torch_dev
    cfg = small_cfg("linear", "f32", n, d, C=C)
    X, y, Xte, _ = data_of(cfg)
    ref = oracle_ref(cfg, X, y)
    f_te = O.decision(X, ref.alpha, ref.b, Xte, spec_of(cfg))
    sens = fp32_sensitivity(X, cfg)
    tol = max(TOL_ALPHA["f32"], 0.1 * sens)
    res = check_train(torch, dev, cfg, ref, X, y, Xte, f_te, alpha_tol=tol)
    assert res.iterations <= ref.iterations + 20


def test_train_residual_replacement(torch_dev):
    """C = 100 needs more than 50 iterations, so the residual is recomputed on the way."""
    torch, dev = torch_dev
    cfg = small_cfg("rbf", "f64", 700, 12, C=100.0, eps=1e-9)
    X, y, Xte, _ = data_of(cfg)
    ref = oracle_ref(cfg, X, y)
    assert ref.iterations > 50
    res = check_train(torch, dev, cfg, ref, X, y)
    assert res.n_matvec == res.iterations + res.iterations // 50


@pytest.mark.parametrize("kernel,dtype,n,d", [("rbf", "f64", 60000, 24), ("linear", "f64", 90000, 16)])
def test_train_large_kkt_rows(torch_dev, kernel, dtype, n, d):
    """Training at a size the oracle cannot solve: rows of the full system,
    f(x_i) + alpha_i / C = y_i (Eq. (11); f evaluated by the oracle from the
    GPU's alpha and b), hold on 64 sampled points within the CG residual the
    run reports, and sum(alpha) = 0. fp64: there the kernel values of the two
    sides agree to rounding, so the CG residual is what bounds each row."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d, C=1.0, eps=1e-8)
    log(f"train large {cfg.name}")
    X, y, _ = S.make_train(cfg)
    r = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=cfg.eps,
                true_residual=True, **kw_of(cfg))
    assert r.converged and r.true_rel_residual <= 2 * cfg.eps
    alpha = r.alpha.cpu().numpy().astype(np.float64)
    rows = np.unique(np.concatenate([[0, n - 1],
                                     np.random.default_rng(n).choice(n, 62, replace=False)]))
    f = O.decision(X, alpha, r.b, X[rows], spec_of(cfg))
    kkt = f + alpha[rows] / cfg.C - y[rows].astype(np.float64)
    # every row's residual is bounded by the reduced residual's 2-norm (Eq. (13)
    # is the full system with the pivot row eliminated), plus the rounding of
    # alpha to the working precision in the evaluation
    rhs_norm = float(np.linalg.norm(y[:-1].astype(np.float64) - float(y[-1])))
    u = 1e-13   # generous for fp64 sums of n terms
    bound = 2 * r.true_rel_residual * rhs_norm + u * n * max(1.0, float(np.abs(alpha).max()))
    assert float(np.abs(kkt).max()) <= bound, (float(np.abs(kkt).max()), bound)
    assert abs(float(alpha.sum())) <= u * n * max(1.0, float(np.abs(alpha).max()))


def test_train_matvec_times(torch_dev):
    """Per-product times: one entry per timed product (the residual refresh
    after 50 iterations included), each positive, summing to the reported
    total; a short array takes the first products only."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("rbf", "f64", 700, 12, C=100.0, eps=1e-9)
    X, y, _, _ = data_of(cfg)
    Xd, yd = to_dev(torch, dev, X), to_dev(torch, dev, y)
    r = P.train(Xd, yd, C=cfg.C, eps=cfg.eps, time_matvec=True, matvec_times=1000, **kw_of(cfg))
    assert r.iterations > 50 and r.iterations < r.n_matvec_timed <= r.n_matvec
    assert len(r.matvec_times) == r.n_matvec_timed and min(r.matvec_times) > 0.0
    assert sum(r.matvec_times) == pytest.approx(r.t_matvec_ms, rel=1e-12)
    r5 = P.train(Xd, yd, C=cfg.C, eps=cfg.eps, time_matvec=True, matvec_times=5, **kw_of(cfg))
    assert len(r5.matvec_times) == 5 and r5.n_matvec_timed == r.n_matvec_timed
    assert torch.equal(r5.alpha, r.alpha)


@pytest.mark.parametrize("name", list(S.CONFIGS))
def test_train_configs(torch_dev, name):
    """The five workloads at their own eps against the stored oracle solution:
    alpha~ within the contract bar, the bias step pinned, the test labels
    equal with no near-tie; for the fp64 ones (whose reduced matrix fits in
    host memory) also the rigorous distance to the Cholesky solution. At these
    eps CG fixes alpha_m and b only loosely (the oracle's own b moves by up to
    7e-4 under a change of summation order at the cubic workload's 1e-5), so
    their end-to-end errors are asserted at the tighter eps below."""
    torch, dev = torch_dev
    from gpu_common import OracleRef
    cfg = S.CONFIGS[name]
    g = golden(name)
    log(f"train {name}")
    X, y, Xte, _ = data_of(cfg)
    assert S.sha256_arrays(X, y) == str(g["hash_train"]), "generator drifted"
    assert S.sha256_arrays(Xte) == str(g["hash_test"]), "generator drifted"
    ref = OracleRef(g["alpha"], float(g["b"]), int(g["iterations"]), g["q"], float(g["Qmm"]))
    if cfg.dtype == "f64":
        t = golden_tight(name)
        assert str(t["hash_train"]) == str(g["hash_train"])
        Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
        ref.Qt, ref.rhs = Qt, O.reduced_rhs(y)
        ref.x_chol, ref.b_chol = t["alpha_chol"][:-1], float(t["b_chol"])
    check_train(torch, dev, cfg, ref, X, y, Xte, g["f_test"], max_ties=0)


@pytest.mark.parametrize("name", list(S.CONFIGS))
def test_train_configs_tight_eps(torch_dev, name):
    """The five workloads at an eps where the oracle's CG agrees with itself
    under a change of summation order far below the bar (the stored spread at
    most a tenth of it): alpha~ (normwise), alpha_m and b (each relative to its
    own size) within the contract bar of the oracle's CG at the same eps (in
    fp32, b on the scale of f: its fp32 kernel values move it further than
    eps does); for the fp64 ones all three also within the rigorous distance
    of the Cholesky solution."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    from parity_rules import BAR_SOL, alpha_tilde_error, end_to_end_errors, p9_check
    cfg = S.CONFIGS[name]
    bar = BAR_SOL[cfg.dtype]
    t = golden_tight(name)
    eps = float(t["eps_tight"])
    X, y, _, _ = data_of(cfg)
    assert S.sha256_arrays(X, y) == str(t["hash_train"]), "generator drifted"
    assert max(t["spread_tight"]) <= bar / 10
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=eps,
                  max_iter=cfg.max_iter, true_residual=True, **kw_of(cfg))
    alpha = res.alpha.cpu().numpy()
    e_t = alpha_tilde_error(alpha, t["alpha_tight"])
    e_am, e_b, e_bf = end_to_end_errors(alpha, res.b, t["alpha_tight"], float(t["b_tight"]))
    log(f"  {name} at eps {eps:.0e}: status {res.status} it {res.iterations} (oracle "
        f"{int(t['iterations_tight'])}), alpha~ {e_t:.1e}, alpha_m {e_am:.1e}, b {e_b:.1e} "
        f"(relative to each; on the scale of f {e_bf:.1e}; bar {bar:.0e}; oracle's own spread "
        f"{max(t['spread_tight']):.1e})")
    assert res.converged
    assert e_t <= bar and e_am <= bar
    if cfg.dtype == "f64":
        assert e_b <= bar
    else:
        # fp32 kernel values move b by more than eps does: at 65536 x 1024 RBF
        # (C = 10) b (0.045) sits 2.6e-4 of itself = 1.2e-5 from the oracle's
        # fp64 b, which the oracle itself fixes to 4.5e-11 at this eps; on the
        # scale of f (labels +-1) that is within the bar
        assert e_bf <= bar
    if "alpha_chol" in t.files:
        Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
        p9 = p9_check(alpha, res.b, Qt, t["q"], float(t["Qmm"]), O.reduced_rhs(y), cfg.C,
                      t["alpha_chol"][:-1], float(t["b_chol"]))
        log(f"  P9: |alpha~ - x*| {p9['dist']:.1e} <= {p9['bound']:.1e}, b {p9['d_b']:.1e} <= "
            f"{p9['bound_b']:.1e}")
        assert p9["dist"] <= p9["bound"] and p9["d_b"] <= p9["bound_b"]
        assert p9["d_am"] <= p9["bound_am"]


def test_train_concurrent_threads(torch_dev):
    """Two host threads train different problems at once, each on a stream of
    its own: the library keeps its host-side state per thread and the caller
    owns every device buffer, so each result equals its sequential run bit for
    bit."""
    import threading
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfgs = [small_cfg("rbf", "f64", 1500, 40), small_cfg("poly", "f32", 2000, 100)]
    inputs = []
    for c in cfgs:
        X, y, _ = S.make_train(c)
        inputs.append((c, to_dev(torch, dev, X), to_dev(torch, dev, y)))
    seq = [P.train(X, y, C=c.C, eps=c.eps, **kw_of(c)) for c, X, y in inputs]
    torch.cuda.synchronize()
    out, errors = [None] * len(inputs), []

    def run(k):
        try:
            c, X, y = inputs[k]
            st = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(st):
                out[k] = P.train(X, y, C=c.C, eps=c.eps, **kw_of(c))
            st.synchronize()
        except Exception as e:   # reported below, in the main thread
            errors.append(e)

    threads = [threading.Thread(target=run, args=(k,)) for k in range(len(inputs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for a, b in zip(seq, out):
        assert b.converged and a.iterations == b.iterations
        assert torch.equal(a.alpha, b.alpha) and a.b == b.b


def test_train_single_point_and_equal_labels(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    for dt in (torch.float64, torch.float32):
        X = torch.tensor([[0.5, -0.25]], dtype=dt, device=dev)
        y = torch.tensor([-1.0], dtype=dt, device=dev)
        r = P.train(X, y)
        assert r.converged and r.b == -1.0 and r.alpha.cpu().tolist() == [0.0]
        X = torch.rand(200, 5, dtype=dt, device=dev)
        y = torch.ones(200, dtype=dt, device=dev)
        r = P.train(X, y, kernel="rbf", gamma=0.5)
        assert r.converged and r.iterations == 0 and r.b == 1.0
        assert float(r.alpha.abs().max()) == 0.0


def test_train_not_converged_and_history(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("rbf", "f64", 400, 10)
    X, y, _, _ = data_of(cfg)
    r = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=1.0, eps=1e-12, max_iter=1,
                history=4, **kw_of(cfg))
    assert r.status == 1 and not r.converged and r.iterations == 1
    # outputs hold the first iterate: compare with one oracle CG step
    Qt, q, Qmm = O.reduced_matrix(X, spec_of(cfg), 1.0)
    rhs = O.reduced_rhs(y)
    one = O.solve_cg(lambda v: Qt @ v, rhs, 1e-12, max_iter=1)
    alpha, b = O.recover(one.x, y, q, Qmm)
    assert rel_err(r.alpha.cpu().numpy(), alpha) <= 1e-9
    assert abs(r.b - b) <= 1e-9 * max(1, abs(b))
    assert r.history[0] == pytest.approx(one.history[0] / float(rhs @ rhs), rel=1e-9)


def test_train_rejects_nonfinite_and_bad_labels(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    X = torch.rand(64, 3, dtype=torch.float64, device=dev)
    y = torch.ones(64, dtype=torch.float64, device=dev)
    y[::2] = -1
    Xb = X.clone()
    Xb[5, 1] = float("nan")
    with pytest.raises(P.LssvmError) as e:
        P.train(Xb, y)
    assert e.value.code == -2
    yb = y.clone()
    yb[7] = 0.5
    with pytest.raises(P.LssvmError) as e:
        P.train(X, yb)
    assert e.value.code == -3
    yb = y.clone()
    yb[63] = 2.0     # the pivot's label
    with pytest.raises(P.LssvmError) as e:
        P.train(X, yb)
    assert e.value.code == -3
    Xb = X.clone()
    Xb[0, 0] = float("inf")
    with pytest.raises(P.LssvmError) as e:
        P.predict(X, y, 0.0, Xb)
    assert e.value.code == -2


def test_train_deterministic(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("poly", "f32", 900, 33)
    X, y, _, _ = data_of(cfg)
    Xd, yd = to_dev(torch, dev, X), to_dev(torch, dev, y)
    a = P.train(Xd, yd, C=1.0, eps=1e-5, **kw_of(cfg))
    b = P.train(Xd, yd, C=1.0, eps=1e-5, **kw_of(cfg))
    assert a.iterations == b.iterations and a.b == b.b
    assert torch.equal(a.alpha, b.alpha)


def test_train_max_iter_beyond_n_and_long_history(torch_dev):
    """max_iter far above N and a history buffer longer than the run: CG stops at eps,
    the history holds exactly the iterations run, matching the oracle's recurrence."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("linear", "f64", 40, 6)
    X, y, _, _ = data_of(cfg)
    r = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=1.0, eps=1e-12,
                max_iter=100_000, history=5000)
    Qt, _, _ = O.reduced_matrix(X, O.KernelSpec("linear"), 1.0)
    rhs = O.reduced_rhs(y)
    ref = O.solve_cg(lambda v: Qt @ v, rhs, 1e-12, max_iter=100_000)
    assert r.converged and r.iterations <= 39 + 5
    assert abs(r.iterations - ref.iterations) <= 2
    assert len(r.history) == r.iterations
    k = min(len(r.history), len(ref.history), 10)
    d0 = float(rhs @ rhs)
    assert np.allclose(r.history[:k], np.array(ref.history[:k]) / d0, rtol=1e-8, atol=1e-15)


def test_eps_sweep_matches_oracle(torch_dev):
    """The eps sweep (Sec. IV-F) against the oracle run at every eps: iterations,
    training and test accuracy, the eps the Sec. IV-B protocol picks, the
    distance between the two solutions within C (||r_gpu|| + ||r_oracle||) at
    every eps (rigorous), and alpha~ within the contract bar once CG has
    converged tightly (eps <= 1e-10; mid-run CG iterates move with rounding as
    much as the oracle's own run under a change of summation order, logged)."""
    torch, dev = torch_dev
    from paper_2202_12674_amd.eps_sweep import sweep, tune_eps
    cfg = small_cfg("linear", "f64", 1024, 256)
    X, y, Xte, yte = data_of(cfg)
    eps_list = [10.0 ** (-k) for k in range(1, 13)]
    rows = sweep(to_dev(torch, dev, X), to_dev(torch, dev, y), to_dev(torch, dev, Xte),
                 to_dev(torch, dev, yte), kernel="linear", C=1.0, eps_list=eps_list)
    spec = O.KernelSpec("linear")
    Qt, q, Qmm = O.reduced_matrix(X, spec, 1.0)
    rhs = O.reduced_rhs(y)
    h = (cfg.n - 1) // 3
    ref_rows = []
    for eps, r in zip(eps_list, rows):
        a_ref, b_ref, info = O.train(X, y, spec, 1.0, eps)
        # mid-trajectory CG iterates are sensitive to rounding: the oracle's own
        # spread under a change of summation order sets the alpha~ tolerance
        alt = O.solve_cg(lambda v: Qt[:, :h] @ v[:h] + Qt[:, h:] @ v[h:], rhs, eps)
        a_alt, _ = O.recover(alt.x, y, q, Qmm)
        spread = np.abs(a_alt[:-1] - a_ref[:-1]).max() / np.abs(a_ref).max()
        f_tr = O.decision(X, a_ref, b_ref, X, spec)
        f_te = O.decision(X, a_ref, b_ref, Xte, spec)
        acc_tr = float(np.mean(np.where(f_tr > 0, 1, -1) == y))
        acc_te = float(np.mean(np.where(f_te > 0, 1, -1) == yte))
        ref_rows.append({"eps": eps, "train_acc": acc_tr})
        alpha = r["alpha"].cpu().numpy()
        e = np.abs(alpha[:-1] - a_ref[:-1]).max() / np.abs(a_ref).max()
        log(f"  eps {eps:.0e}: it {r['iterations']} (oracle {info['iterations']}), "
            f"alpha~ err {e:.1e} (oracle order spread {spread:.1e}), "
            f"train acc {r['train_acc']:.4f} ({acc_tr:.4f}), "
            f"test acc {r['test_acc']:.4f} ({acc_te:.4f}), {r['time_ms']:.2f} ms")
        assert r["converged"]
        assert abs(r["iterations"] - info["iterations"]) <= max(2, info["iterations"] // 10)
        # rigorous at every eps: both are within C ||r||_2 of the exact solution
        r_gpu = np.linalg.norm(rhs - Qt @ alpha[:-1])
        r_ref = np.linalg.norm(rhs - Qt @ a_ref[:-1])
        assert np.linalg.norm(alpha[:-1] - a_ref[:-1]) <= 1.0 * (r_gpu + r_ref) * (1 + 1e-9)
        if eps <= 1e-10:   # converged tightly: the trajectories agree again
            assert e <= 1e-9
        assert r["train_acc"] == acc_tr and r["test_acc"] == acc_te
    assert tune_eps(rows) == tune_eps(ref_rows)


def _alpha_err(a, ref):
    a = np.asarray(a, dtype=np.float64)[:-1]
    ref = np.asarray(ref, dtype=np.float64)[:-1]
    return float(np.abs(a - ref).max() / np.abs(ref).max())


@pytest.mark.parametrize("dtype,kernel,n,d", [("f64", "rbf", 500, 24), ("f32", "poly", 400, 64)])
def test_warm_start_random_matches_oracle(torch_dev, dtype, kernel, n, d):
    """CG from a random alpha~0: the oracle's warm CG from the same values."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d, C=1.0)
    X, y, _, _ = data_of(cfg)
    a0 = (np.random.default_rng(9).standard_normal(n) * 0.05).astype(cfg.np_dtype)
    ref_a, ref_b, info = O.train(X, y, spec_of(cfg), cfg.C, cfg.eps, alpha0=a0)
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=cfg.eps,
                  alpha0=to_dev(torch, dev, a0), **kw_of(cfg))
    log(f"  warm {cfg.name}: it {res.iterations} (oracle {info['iterations']}) "
        f"rel {res.rel_residual:.2e}")
    assert res.converged and res.rel_residual <= cfg.eps
    assert res.n_matvec == res.iterations + res.iterations // 50 + 1
    if dtype == "f64":
        assert abs(res.iterations - info["iterations"]) <= 2
    else:
        assert res.iterations <= 2 * info["iterations"] + 10
    assert _alpha_err(res.alpha.cpu().numpy(), ref_a) <= TOL_ALPHA[dtype]


def test_warm_start_resumes_at_a_tighter_eps(torch_dev):
    """Solve at eps = 1e-4, then continue from that alpha to 1e-10: fewer
    iterations than a cold run to 1e-10, the same solution within the bar;
    restarting at the returned solution takes at most a couple of iterations."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("rbf", "f64", 600, 16, C=10.0, eps=1e-10)
    X, y, _, _ = data_of(cfg)
    Xd, yd = to_dev(torch, dev, X), to_dev(torch, dev, y)
    coarse = P.train(Xd, yd, C=cfg.C, eps=1e-4, **kw_of(cfg))
    cold = P.train(Xd, yd, C=cfg.C, eps=cfg.eps, **kw_of(cfg))
    warm = P.train(Xd, yd, C=cfg.C, eps=cfg.eps, alpha0=coarse.alpha, **kw_of(cfg))
    log(f"  coarse {coarse.iterations} it, cold {cold.iterations} it, resumed {warm.iterations} it")
    assert warm.converged and warm.iterations < cold.iterations
    ref_a, ref_b, _ = O.train(X, y, spec_of(cfg), cfg.C, cfg.eps)
    assert _alpha_err(warm.alpha.cpu().numpy(), ref_a) <= 1e-8
    again = P.train(Xd, yd, C=cfg.C, eps=cfg.eps, alpha0=warm.alpha, **kw_of(cfg))
    assert again.iterations <= 2 and again.converged
    assert _alpha_err(again.alpha.cpu().numpy(), warm.alpha.cpu().numpy()) <= 1e-9


def test_warm_start_equal_labels_still_zero(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("linear", "f64", 64, 5)
    X, _, _, _ = data_of(cfg)
    y = np.ones(cfg.n)
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=1.0, eps=1e-8,
                  alpha0=torch.ones(cfg.n, dtype=torch.float64, device=dev), **kw_of(cfg))
    assert res.iterations == 0 and res.b == 1.0
    assert float(res.alpha.abs().max()) == 0.0
