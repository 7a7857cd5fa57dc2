"""GPU: how CG ends, and what the outputs hold when it fails.

* Stagnation (Sec. III-B, Sec. IV-F): an eps below what the arithmetic attains
  ends CG, unconverged, a few residual recomputations after the floor, as the
  oracle's CG does under the same rule, instead of running N iterations.
* Curvature breakdown: an indefinite Q~ (polynomial kernel with coef0 < 0,
  Sec. II-E) returns LSSVM_EBREAKDOWN at the iteration where the oracle's CG
  finds d^T Q~ d <= 0, with the outputs untouched.
* Outputs untouched on every input error (NaN, bad label), for training,
  prediction and the single-point case, through the raw C ABI with sentinel
  buffers.
* Host contexts: threads that come and go reuse the library's pooled pinned
  buffers instead of each leaving one behind.
* lssvm_cg_step at an exact solution (r = 0): no NaN, beta = 0.
"""
from __future__ import annotations

import ctypes
import sys
import threading

import numpy as np
import pytest

import oracle as O
import synthdata as S

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2202_12674_amd as P
    P.lib()  # fail loudly if the HIP library is missing
    return torch, torch.device("cuda:0")


def to_dev(torch, dev, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def cfg_of(kernel, dtype, n, d, C=1.0, eps=1e-8, **kp):
    return S.Config(f"{kernel}_{dtype}_{n}x{d}", dtype, kernel, n, d, mu=1.0, inf_frac=0.3,
                    flip_frac=0.05, C=C, eps=eps, **kp)


def spec_of(cfg):
    return O.KernelSpec(cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)


def kw_of(cfg):
    return dict(kernel=cfg.kernel, gamma=cfg.gamma, coef0=cfg.coef0, degree=cfg.degree)


# ------------------------------------------------------------ stagnation ----

@pytest.mark.parametrize("eps", [1e-13, 1e-15])
def test_stall_below_the_fp64_floor_matches_oracle(torch_dev, eps):
    """Linear fp64 4096 x 1024 (the second workload's shape and generator):
    fp64 CG bottoms out near 1e-12. The GPU stops stalled, like the oracle,
    within a recomputation or two of it (the decision compares rounded values
    of two different summation orders), returning an iterate at the floor."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = S.CONFIGS["linear_f64_4096x1024"]
    X, y, _ = S.make_train(cfg)
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    rhs = O.reduced_rhs(y)
    ref = O.solve_cg(lambda v: Qt @ v, rhs, eps)
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=eps,
                  true_residual=True, history=5000, **kw_of(cfg))
    a = res.alpha.cpu().numpy()[:-1]
    gpu_true = float(np.linalg.norm(rhs - Qt @ a) / np.linalg.norm(rhs))
    log(f"  eps {eps:.0e}: gpu {res.iterations} it (stalled {res.stalled}, reported "
        f"{res.rel_residual:.2e}, true {res.true_rel_residual:.2e}, oracle-measured "
        f"{gpu_true:.2e}); oracle {ref.iterations} it (stalled {ref.stalled}, "
        f"true {ref.true_rel_residual:.2e})")
    assert ref.stalled and not ref.converged
    assert res.status == 1 and res.stalled and not res.converged
    assert res.iterations % 50 == 0 and res.iterations < cfg.n - 1
    assert abs(res.iterations - ref.iterations) <= 100
    # the returned iterate is the best recomputed one: its true residual is
    # what the report says, and it sits at the floor like the oracle's
    assert res.true_rel_residual == pytest.approx(res.rel_residual, rel=1e-6)
    assert gpu_true <= 10 * max(ref.true_rel_residual, 1e-13)
    hist = np.asarray(res.history)
    refreshed = hist[np.arange(49, res.iterations, 50)]
    assert res.rel_residual ** 2 == pytest.approx(min(1.0, refreshed.min()), rel=1e-9)


def test_fp32_products_end_near_the_fp64_floor(torch_dev):
    """fp32 kernel values with fp64 CG vectors (the fourth workload's precision
    and kernel at 4096 x 1024). The tile products are one fixed, exactly
    symmetric operator (row and column sums of the same fp32 kernel values,
    products and sums in fp64), so CG on it behaves like fp64 CG: asked for
    eps = 1e-15 it ends within a few hundred iterations, converged (on the
    recurrence) or stalled, with a true residual near the fp64 floor, as the
    oracle's fp64 CG does on the same points."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = cfg_of("poly", "f32", 4096, 1024, gamma=1.0 / 1024, coef0=1.0, degree=3)
    X, y, _ = S.make_train(cfg)
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    rhs = O.reduced_rhs(y)
    ref = O.solve_cg(lambda v: Qt @ v, rhs, 1e-15)
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=1.0, eps=1e-15,
                  true_residual=True, **kw_of(cfg))
    log(f"  fp32 cubic eps 1e-15: {res.iterations} it, status {res.status}, stalled "
        f"{res.stalled}, reported {res.rel_residual:.2e}, true {res.true_rel_residual:.2e}; "
        f"oracle {ref.iterations} it, converged {ref.converged}, stalled {ref.stalled}, "
        f"true {ref.true_rel_residual:.2e}")
    assert res.converged or res.stalled
    assert res.iterations <= max(300, ref.iterations + 100)
    assert res.true_rel_residual <= 1e-13
    if res.stalled:
        assert res.true_rel_residual == pytest.approx(res.rel_residual, rel=1e-6)


def test_benchmark_workload_at_eps_1e_8(torch_dev):
    """The fourth workload (cubic, fp32, 32768 x 4096) at eps = 1e-8 instead of
    1e-5: the fp32 kernel values form one fixed, exactly symmetric operator
    and CG runs in fp64 on it, so it either converges (true residual at eps)
    or ends stalled within a few hundred iterations, never running to N."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = S.CONFIGS["poly_f32_32768x4096"]
    X, y, _ = S.make_train(cfg)
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=1e-8,
                  true_residual=True, **kw_of(cfg))
    log(f"  32768 x 4096 cubic fp32, eps 1e-8: status {res.status}, {res.iterations} it, "
        f"stalled {res.stalled}, reported {res.rel_residual:.2e}, "
        f"true {res.true_rel_residual:.2e}, cg {res.t_cg_ms:.0f} ms")
    assert res.iterations <= 400
    if res.converged:
        assert res.true_rel_residual <= 2e-8
    else:
        assert res.stalled
        assert res.true_rel_residual == pytest.approx(res.rel_residual, rel=1e-6)


# ------------------------------------------------------------- breakdown ----

BREAKDOWN_CASES = [("f64", 300, 8, 2, -1.0, 10.0), ("f64", 500, 16, 3, -1.0, 10.0),
                   ("f32", 400, 32, 3, -0.5, 100.0), ("f32", 500, 16, 2, -0.5, 10.0)]


def oracle_breakdown(Qt, rhs):
    """The oracle's CG to its breakdown, and for every step the curvature
    d^T Q~ d (replayed with cg_step) over its rounding scale |d|^T |Q~| |d|, so
    the test can see that no decision is a rounding call."""
    res = O.solve_cg(lambda v: Qt @ v, rhs, 1e-12)
    x, r, d = np.zeros_like(rhs), rhs.copy(), rhs.copy()
    rr = float(rhs @ rhs)
    absQ = np.abs(Qt)
    rel = []
    for _ in range(res.iterations):
        scale = float(np.abs(d) @ (absQ @ np.abs(d)))
        x, r, d, rr, gamma, _, _ = O.cg_step(x, r, d, Qt @ d, rr)
        rel.append(gamma / scale)
    return res, rel


def raw_train(torch, dev, X, y, cfg, eps, alpha_buf, info):
    import paper_2202_12674_amd as P
    from paper_2202_12674_amd._binding import Params
    L = P.lib()
    n, d = X.shape
    dt = 0 if X.dtype == torch.float64 else 1
    kcode = {"linear": 0, "poly": 1, "rbf": 2}[cfg.kernel]
    kp = Params(cfg.gamma, cfg.coef0, cfg.degree)
    ws = P.alloc_workspace(L.lssvm_workspace_bytes(n, d, dt), dev)
    b = ctypes.c_double(12345.0)
    code = L.lssvm_train(ctypes.c_void_p(X.data_ptr()), ctypes.c_void_p(y.data_ptr()), n, d, dt,
                         kcode, ctypes.byref(kp), cfg.C, eps, 0, ctypes.c_void_p(ws.data_ptr()),
                         ws.numel(), ctypes.c_void_p(alpha_buf.data_ptr()), ctypes.byref(b),
                         ctypes.byref(info) if info is not None else None,
                         ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
    torch.cuda.synchronize()
    return code, b.value


@pytest.mark.parametrize("dtype,n,d,degree,coef0,C", BREAKDOWN_CASES)
def test_breakdown_on_indefinite_matrix(torch_dev, dtype, n, d, degree, coef0, C):
    torch, dev = torch_dev
    from paper_2202_12674_amd._binding import Info
    cfg = cfg_of("poly", dtype, n, d, C=C, gamma=1.0 / d, coef0=coef0, degree=degree)
    X, y, _ = S.make_train(cfg)
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), C)
    assert np.linalg.eigvalsh(Qt).min() < 0          # indefinite, by construction
    ref, curv = oracle_breakdown(Qt, O.reduced_rhs(y))
    assert ref.breakdown
    # clear decisions: every earlier curvature far above its rounding scale,
    # the last far below zero (fp32 kernel values move them by ~1e-6)
    assert all(c > 1e-5 for c in curv[:-1]) and curv[-1] < -1e-5
    Xd, yd = to_dev(torch, dev, X), to_dev(torch, dev, y)
    alpha = torch.full((n,), 7.5, dtype=Xd.dtype, device=dev)
    info = Info()
    code, b = raw_train(torch, dev, Xd, yd, cfg, 1e-12, alpha, info)
    log(f"  {cfg.name} deg {degree} coef0 {coef0} C {C}: code {code} at iteration "
        f"{info.iterations} (oracle {ref.iterations}), relative curvatures "
        f"{['%.2g' % c for c in curv]}")
    assert code == -4
    assert info.iterations == ref.iterations and info.stop_reason == 3
    assert bool((alpha == 7.5).all()) and b == 12345.0        # outputs untouched


# ------------------------------------------------------ untouched outputs ---

@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_train_errors_leave_outputs_untouched(torch_dev, dtype):
    torch, dev = torch_dev
    cfg = cfg_of("rbf", dtype, 300, 5, gamma=0.2)
    X, y, _ = S.make_train(cfg)
    for n in (1, 300):
        Xd = to_dev(torch, dev, X[:n].copy())
        yd = to_dev(torch, dev, y[:n].copy())
        for what in ("nan", "label"):
            Xb, yb = Xd.clone(), yd.clone()
            if what == "nan":
                Xb[n // 2, 3] = float("nan")
            else:
                yb[n - 1] = 0.5
            alpha = torch.full((n,), -3.25, dtype=Xd.dtype, device=dev)
            code, b = raw_train(torch, dev, Xb, yb, cfg, 1e-8, alpha, None)
            assert code == (-2 if what == "nan" else -3), (n, what, code)
            assert bool((alpha == -3.25).all()) and b == 12345.0, (n, what)


@pytest.mark.parametrize("kernel", ["linear", "rbf"])
def test_predict_errors_leave_outputs_untouched(torch_dev, kernel):
    """Scores and labels keep their contents when either point set holds a
    NaN, on the tile path (RBF) and the linear weight shortcut alike."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    from paper_2202_12674_amd._binding import Params
    L = P.lib()
    n, nt, d = 300, 70, 7
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    X = torch.rand(n, d, dtype=torch.float64, device=dev, generator=g)
    Xt = torch.rand(nt, d, dtype=torch.float64, device=dev, generator=g)
    alpha = torch.rand(n, dtype=torch.float64, device=dev, generator=g) - 0.5
    kcode = {"linear": 0, "rbf": 2}[kernel]
    kp = Params(0.5, 0.0, 1)
    ws = P.alloc_workspace(L.lssvm_predict_workspace_bytes(n, nt, d, 0), dev)
    for bad_train in (True, False):
        A, B = X.clone(), Xt.clone()
        (A if bad_train else B)[3, 2] = float("nan")
        scores = torch.full((nt,), 9.0, dtype=torch.float64, device=dev)
        labels = torch.full((nt,), 5, dtype=torch.int32, device=dev)
        code = L.lssvm_predict(ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(alpha.data_ptr()),
                               0.25, n, d, 0, kcode, ctypes.byref(kp),
                               ctypes.c_void_p(B.data_ptr()), nt, ctypes.c_void_p(ws.data_ptr()),
                               ws.numel(), ctypes.c_void_p(scores.data_ptr()),
                               ctypes.c_void_p(labels.data_ptr()),
                               ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
        torch.cuda.synchronize()
        assert code == -2
        assert bool((scores == 9.0).all()) and bool((labels == 5).all()), bad_train


# --------------------------------------------------------- host contexts ----

def test_host_contexts_are_pooled_across_threads(torch_dev):
    """32 short-lived threads, 4 at a time, each training once: the library
    keeps at most as many host contexts as calls that ran at once."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = cfg_of("linear", "f64", 200, 6)
    X, y, _ = S.make_train(cfg)
    Xd, yd = to_dev(torch, dev, X), to_dev(torch, dev, y)
    P.train(Xd, yd, C=1.0, eps=1e-8)
    before = P.host_contexts()
    errors = []

    def run():
        try:
            st = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(st):
                r = P.train(Xd, yd, C=1.0, eps=1e-8)
            st.synchronize()
            assert r.converged
        except Exception as e:   # reported in the main thread
            errors.append(e)

    for _ in range(8):
        ts = [threading.Thread(target=run) for _ in range(4)]
        for t in ts:
            t.start()
        for t in ts:
            t.join()
    assert not errors, errors
    after = P.host_contexts()
    log(f"  host contexts: {before} before, {after} after 32 threads")
    assert after <= before + 4


# --------------------------------------------------------------- cg_step ----

def test_cg_step_at_an_exact_solution(torch_dev):
    """r = 0 on entry (rr = 0): x stays, r and d become 0, beta = 0, no NaN,
    like the oracle's cg_step."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    n = 3000
    rng = np.random.default_rng(8)
    x0, d0 = rng.standard_normal(n), rng.standard_normal(n)
    q0 = 2.0 * d0
    xo, ro, do, rro, go, ao, bo = O.cg_step(x0, np.zeros(n), d0, q0, 0.0)
    x, r, d, q = (to_dev(torch, dev, a) for a in (x0, np.zeros(n), d0, q0))
    sc = torch.zeros(4, dtype=torch.float64, device=dev)
    P.cg_step(x, r, d, q, sc)
    torch.cuda.synchronize()
    got = sc.cpu().numpy()
    assert np.isfinite(got).all() and np.isfinite(d.cpu().numpy()).all()
    np.testing.assert_array_equal(x.cpu().numpy(), xo)
    np.testing.assert_array_equal(r.cpu().numpy(), ro)
    np.testing.assert_array_equal(d.cpu().numpy(), do)
    assert got[0] == rro == 0.0 and got[2] == ao == 0.0 and got[3] == bo == 0.0
    assert got[1] == pytest.approx(go, rel=1e-12)
