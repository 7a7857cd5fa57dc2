"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Same seeded inputs on both sides. Bars: fp64 matvec 1e-11 and alpha/b 1e-9,
fp32 matvec 1e-5 and alpha/b 1e-4 (max-norm relative error; b relative to
max(1, |b|)); predicted labels identical except exact near-ties of the
oracle's decision value, which are counted and bounded.
"""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest

import oracle as O
import synthdata as S

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL_MV = {"f64": 1e-11, "f32": 1e-5}
TOL_ALPHA = {"f64": 1e-9, "f32": 1e-4}


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


def rel_err(a, ref):
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-300))


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


def labels_match(lab, f_ref, scale_tol):
    """Labels equal wherever the oracle's decision value is not a near-tie."""
    f_ref = np.asarray(f_ref)
    lab_ref = np.where(f_ref > 0, 1, -1)
    tie = np.abs(f_ref) <= scale_tol * max(1.0, np.abs(f_ref).max())
    bad = (np.asarray(lab) != lab_ref) & ~tie
    return int(bad.sum()), int(tie.sum())


# ------------------------------------------------------------ matvec --------

SMALL_SHAPES = [(2, 1), (3, 3), (129, 65), (257, 3), (300, 100), (1000, 17)]


@pytest.mark.parametrize("dtype", ["f64", "f32"])
@pytest.mark.parametrize("kernel", ["linear", "poly", "rbf"])
@pytest.mark.parametrize("n,d", SMALL_SHAPES)
def test_matvec_small_shapes(torch_dev, dtype, kernel, n, d):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d, C=2.0)
    log(f"matvec {cfg.name}")
    X, y, _, _ = data_of(cfg)
    p = S.probe_vector(n - 1, cfg.np_dtype, seed=7)
    out = P.matvec(to_dev(torch, dev, X), to_dev(torch, dev, p), C=cfg.C, **kw_of(cfg))
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    ref = Qt @ p.astype(np.float64)
    assert rel_err(out.cpu().numpy(), ref) <= TOL_MV[dtype]


# Linear products of few tiles split each tile's features over several
# workgroups; these shapes give every split the library uses.
SPLIT_SHAPES = [("f64", 4096, 256, 2), ("f64", 4096, 1024, 4), ("f64", 1000, 256, 8),
                ("f64", 600, 1024, 16), ("f32", 2000, 1024, 2), ("f32", 1000, 256, 4),
                ("f32", 1000, 1024, 8), ("f32", 600, 1024, 16)]


@pytest.mark.parametrize("dtype,n,d,split", SPLIT_SHAPES)
def test_matvec_linear_feature_split(torch_dev, dtype, n, d, split):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    L = P.lib()
    assert L.lssvm_tile_split(n, d, 0 if dtype == "f64" else 1, 0) == split
    cfg = small_cfg("linear", dtype, n, d, C=2.0)
    log(f"matvec split {split} {cfg.name}")
    X, y, _, _ = data_of(cfg)
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    Xd = to_dev(torch, dev, X)
    for seed in (7, 8):
        p = S.probe_vector(n - 1, cfg.np_dtype, seed=seed)
        out = P.matvec(Xd, to_dev(torch, dev, p), C=cfg.C, **kw_of(cfg)).cpu().numpy()
        assert rel_err(out, Qt @ p.astype(np.float64)) <= TOL_MV[dtype]
    e = np.zeros(n - 1, dtype=cfg.np_dtype)
    e[n // 2] = 1   # one column: the diagonal entry and the 1/C term come from one split
    out = P.matvec(Xd, to_dev(torch, dev, e), C=cfg.C, **kw_of(cfg)).cpu().numpy()
    assert rel_err(out, Qt[:, n // 2]) <= TOL_MV[dtype]


@pytest.mark.parametrize("dtype,n,d,split", [SPLIT_SHAPES[2], SPLIT_SHAPES[5]])
def test_train_linear_feature_split(torch_dev, dtype, n, d, split):
    torch, dev = torch_dev
    cfg = small_cfg("linear", dtype, n, d, C=1.0)
    X, y, Xte, _ = data_of(cfg)
    alpha, b, iters, spread = oracle_cg_with_spread(cfg, X, y)
    f_te = O.decision(X, alpha, b, Xte, spec_of(cfg))
    check_train(torch, dev, cfg, alpha, b, iters, X, y, Xte, f_te, spread)


def tail_plan(n, d, dtype):
    """(tail tiles, splits) of a symmetric product as the library plans it: the
    tiles after the last full round of 512 workgroups, split 4..16 ways when
    they are at most a quarter round."""
    bk = 16 if dtype == "f64" else 32
    nkb = -(-d // (2 * bk)) * 2
    nT = -(-(n - 1) // 128)
    Q = nT * (nT + 1) // 2 % 512
    S = 1
    while S < 16 and Q * S * 2 <= 512 and nkb % (4 * S) == 0:
        S *= 2
    return (Q, S) if Q > 0 and S >= 4 else (0, 1)


# Tiles beyond the last full round are split over several workgroups whose
# inner products a fixup launch sums: every tile in the tail (600 points), one
# full round plus 16 tail tiles (4096 points), a linear product without the
# feature split (12288 points).
TAIL_SHAPES = [("f64", "rbf", 600, 256, (15, 8)), ("f32", "poly", 600, 256, (15, 4)),
               ("f64", "poly", 4096, 256, (16, 8)), ("f32", "rbf", 4096, 512, (16, 8)),
               ("f64", "linear", 12288, 1024, (48, 8))]


@pytest.mark.parametrize("dtype,kernel,n,d,plan", TAIL_SHAPES)
def test_matvec_tail_split(torch_dev, dtype, kernel, n, d, plan):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    assert tail_plan(n, d, dtype) == plan
    if kernel == "linear":
        assert P.lib().lssvm_tile_split(n, d, 0 if dtype == "f64" else 1, 0) == 1
    cfg = small_cfg(kernel, dtype, n, d, C=2.0)
    log(f"matvec tail {plan} {cfg.name}")
    X, y, _, _ = data_of(cfg)
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    Xd = to_dev(torch, dev, X)
    for seed in (7, 8):
        p = S.probe_vector(n - 1, cfg.np_dtype, seed=seed)
        out = P.matvec(Xd, to_dev(torch, dev, p), C=cfg.C, **kw_of(cfg)).cpu().numpy()
        assert rel_err(out, Qt @ p.astype(np.float64)) <= TOL_MV[dtype]
    for j in (0, n - 2):   # columns of the first and the last tile of the visit order
        e = np.zeros(n - 1, dtype=cfg.np_dtype)
        e[j] = 1
        out = P.matvec(Xd, to_dev(torch, dev, e), C=cfg.C, **kw_of(cfg)).cpu().numpy()
        assert rel_err(out, Qt[:, j]) <= TOL_MV[dtype], j
    del Qt


@pytest.mark.parametrize("dtype,kernel,n,d,plan", [TAIL_SHAPES[2], TAIL_SHAPES[3]])
def test_train_tail_split(torch_dev, dtype, kernel, n, d, plan):
    torch, dev = torch_dev
    cfg = small_cfg(kernel, dtype, n, d, C=1.0)
    X, y, Xte, _ = data_of(cfg)
    alpha, b, iters, spread = oracle_cg_with_spread(cfg, X, y)
    f_te = O.decision(X, alpha, b, Xte, spec_of(cfg))
    check_train(torch, dev, cfg, alpha, b, iters, X, y, Xte, f_te, spread)


def _random_cases(count=24, seed=2026):
    """Seeded shapes across kernels and precisions: ragged n and d that land on
    every way a product is laid out (padding, feature splits, split tails)."""
    rng = np.random.default_rng(seed)
    cases = []
    for k in range(count):
        n, d = int(rng.integers(2, 3000)), int(rng.integers(1, 700))
        C = float(rng.choice([0.1, 1.0, 10.0]))
        cases.append((["linear", "poly", "rbf"][k % 3], ["f64", "f32"][(k // 3) % 2], n, d, C))
    return cases


@pytest.mark.parametrize("kernel,dtype,n,d,C", _random_cases())
def test_matvec_random_shapes(torch_dev, kernel, dtype, n, d, C):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d, C=C)
    log(f"matvec random {cfg.name} C={C}")
    X, y, _, _ = data_of(cfg)
    p = S.probe_vector(n - 1, cfg.np_dtype, seed=n)
    out = P.matvec(to_dev(torch, dev, X), to_dev(torch, dev, p), C=C, **kw_of(cfg))
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), C)
    assert rel_err(out.cpu().numpy(), Qt @ p.astype(np.float64)) <= TOL_MV[dtype]


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


def _random_large_cases(count=16, seed=11):
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


@pytest.mark.parametrize("kernel,dtype,n,d,C,kp", _random_large_cases())
def test_matvec_random_large(torch_dev, kernel, dtype, n, d, C, kp):
    """Large random shapes: 64 sampled rows (the first and the last among them)
    against the oracle's rows of Q~."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = S.Config(f"{kernel}_{dtype}_{n}x{d}", dtype, kernel, n, d, mu=1.0, inf_frac=0.5,
                   flip_frac=0.05, C=C, eps=1e-8, **kp)
    log(f"matvec random large {cfg.name} C={C:.3g} {kp}")
    X, _, _ = S.make_train(cfg)
    p = S.probe_vector(n - 1, cfg.np_dtype, seed=n)
    out = P.matvec(to_dev(torch, dev, X), to_dev(torch, dev, p), C=C, **kw_of(cfg)).cpu().numpy()
    rows = np.unique(np.concatenate([[0, n - 2],
                                     np.random.default_rng(n).choice(n - 1, 62, replace=False)]))
    ref = O.reduced_rows(X.astype(np.float64), spec_of(cfg), C, rows) @ p.astype(np.float64)
    assert rel_err(out[rows], ref) <= TOL_MV[dtype]


# Extreme aspect ratios: few points with many features (long feature loops;
# the linear kernel at its largest feature splits), and tens of thousands of
# points with one to three features (one feature block per tile, every
# workgroup's time in its first block and epilogue).
EXTREME_SHAPES = [("linear", "f64", 300, 65536), ("rbf", "f32", 700, 30000),
                  ("poly", "f64", 1000, 16384), ("linear", "f32", 40000, 1),
                  ("rbf", "f64", 33000, 2), ("poly", "f32", 20000, 3)]


@pytest.mark.parametrize("kernel,dtype,n,d", EXTREME_SHAPES)
def test_matvec_extreme_shapes(torch_dev, kernel, dtype, n, d):
    """64 sampled rows (the first and the last among them) against the
    oracle's rows of Q~."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d, C=1.0)
    log(f"matvec extreme {cfg.name}")
    X, _, _ = S.make_train(cfg)
    p = S.probe_vector(n - 1, cfg.np_dtype, seed=n)
    out = P.matvec(to_dev(torch, dev, X), to_dev(torch, dev, p), C=cfg.C,
                   **kw_of(cfg)).cpu().numpy()
    rows = np.unique(np.concatenate([[0, n - 2],
                                     np.random.default_rng(n).choice(n - 1, 62, replace=False)]))
    ref = O.reduced_rows(X.astype(np.float64), spec_of(cfg), cfg.C, rows) @ p.astype(np.float64)
    assert rel_err(out[rows], ref) <= TOL_MV[dtype]


@pytest.mark.parametrize("kernel,dtype", [("linear", "f64"), ("rbf", "f32")])
def test_train_wide(torch_dev, kernel, dtype):
    """300 points with 16384 features: the solution, bias and test labels
    against the oracle's CG."""
    torch, dev = torch_dev
    cfg = small_cfg(kernel, dtype, 300, 16384)
    log(f"train wide {cfg.name}")
    X, y, scale = S.make_train(cfg)
    Xte, _ = S.make_test(cfg, scale, n_test=200)
    alpha, b, iters, spread = oracle_cg_with_spread(cfg, X, y)
    f_te = O.decision(X, alpha, b, Xte, spec_of(cfg))
    check_train(torch, dev, cfg, alpha, b, iters, X, y, Xte, f_te, spread)


@pytest.mark.parametrize("kernel,dtype,n,d,C", [_random_cases()[k] for k in (0, 4, 8, 13, 17, 21)])
def test_train_random_shapes(torch_dev, kernel, dtype, n, d, C):
    """The full alpha / b bar where fp32 can resolve the solution to it
    (kappa u32 <= 1e-3); for fp32 systems conditioned beyond that, two solves
    that both meet eps may differ by up to kappa u32 in alpha, so the check is
    what fp32 CG promises: convergence, the true residual and the test labels
    away from near-ties."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d, C=C)
    X, y, Xte, _ = data_of(cfg)
    alpha, b, iters, spread = oracle_cg_with_spread(cfg, X, y)
    f_te = O.decision(X, alpha, b, Xte, spec_of(cfg))
    sens = fp32_sensitivity(X, cfg) if dtype == "f32" else 0.0
    log(f"  {cfg.name} C={C}: kappa u32 <= {sens:.1e}")
    if sens <= 1e-3:
        check_train(torch, dev, cfg, alpha, b, iters, X, y, Xte, f_te, spread)
        return
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=cfg.eps,
                  true_residual=True, **kw_of(cfg))
    assert res.converged and res.true_rel_residual <= 2 * cfg.eps
    scores, labels = P.predict(to_dev(torch, dev, X), res.alpha, res.b, to_dev(torch, dev, Xte),
                               **kw_of(cfg))
    bad, ties = labels_match(labels.cpu().numpy(), f_te, min(1.0, 10 * sens))
    log(f"  fp32, ill-conditioned: it {res.iterations}, true residual {res.true_rel_residual:.2e},"
        f" {bad} label mismatches outside {ties} near-ties")
    assert bad == 0


@pytest.mark.parametrize("dtype", ["f64", "f32"])
@pytest.mark.parametrize("kernel", ["linear", "poly", "rbf"])
def test_matvec_unit_vectors_give_columns(torch_dev, dtype, kernel):
    """Q~ e_j is column j of Q~: checks single entries, the diagonal and padding."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, 300, 40, C=0.5)
    X, _, _, _ = data_of(cfg)
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    Xd = to_dev(torch, dev, X)
    N = 299
    for j in (0, 127, 128, 200, N - 1):
        e = np.zeros(N, dtype=cfg.np_dtype)
        e[j] = 1
        out = P.matvec(Xd, to_dev(torch, dev, e), C=cfg.C, **kw_of(cfg)).cpu().numpy()
        assert rel_err(out, Qt[:, j]) <= TOL_MV[dtype], j


@pytest.mark.parametrize("name", ["linear_f64_256x64", "linear_f64_4096x1024"])
def test_matvec_configs_live_oracle(torch_dev, name):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = S.CONFIGS[name]
    log(f"matvec {name}")
    X, y, _, _ = data_of(cfg)
    N = cfg.n - 1
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    Xd = to_dev(torch, dev, X)
    for p in (S.probe_vector(N, cfg.np_dtype), O.reduced_rhs(y).astype(cfg.np_dtype)):
        out = P.matvec(Xd, to_dev(torch, dev, p), C=cfg.C, **kw_of(cfg)).cpu().numpy()
        assert rel_err(out, Qt @ p.astype(np.float64)) <= TOL_MV[cfg.dtype]


def golden(name):
    path = os.path.join(GOLDEN, f"{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"golden values for {name} not generated")
    return np.load(path, allow_pickle=False)


@pytest.mark.parametrize("name", list(S.CONFIGS))
def test_matvec_full_configs_golden(torch_dev, name):
    """Full-size product with the seeded probe vector against the stored oracle product,
    plus sampled rows recomputed one by one by the oracle."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = S.CONFIGS[name]
    g = golden(name)
    log(f"matvec full {name}")
    X, y, _, _ = data_of(cfg)
    assert S.sha256_arrays(X, y) == str(g["hash_train"]), "generator drifted"
    N = cfg.n - 1
    p = S.probe_vector(N, cfg.np_dtype)
    out = P.matvec(to_dev(torch, dev, X), to_dev(torch, dev, p), C=cfg.C,
                   **kw_of(cfg)).cpu().numpy()
    ref = g["mv_probe"]
    assert rel_err(out, ref) <= TOL_MV[cfg.dtype]
    rows = [0, N // 3, N - 1]
    sampled = O.matvec_rows(X, spec_of(cfg), cfg.C, p, rows)
    scale = np.abs(ref).max()
    assert np.abs(out[rows] - sampled).max() / scale <= TOL_MV[cfg.dtype]


@pytest.mark.parametrize("kernel,dtype,n,d", [("rbf", "f32", 1000, 300),      # whole tiles
                                              ("linear", "f64", 4096, 1024),   # feature split
                                              ("rbf", "f64", 4096, 256)])      # split tail
def test_matvec_deterministic(torch_dev, kernel, dtype, n, d):
    """Bitwise equal products run to run: fixed-order sums, no atomics, on every
    way a product is split over workgroups."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d)
    X, _, _, _ = data_of(cfg)
    Xd = to_dev(torch, dev, X)
    p = to_dev(torch, dev, S.probe_vector(n - 1, cfg.np_dtype))
    a = P.matvec(Xd, p, C=1.0, **kw_of(cfg)).cpu().numpy()
    for _ in range(2):
        b = P.matvec(Xd, p, C=1.0, **kw_of(cfg)).cpu().numpy()
        assert np.array_equal(a, b)


# ------------------------------------------------------------- train --------

def order_spread(alpha, b, alpha_alt, b_alt):
    """Spread between two oracle CG runs that differ only in summation order."""
    sa = rel_err(alpha_alt, alpha)
    sb = abs(b_alt - b) / max(1.0, abs(b))
    return sa, sb


def oracle_cg_with_spread(cfg, X, y):
    """Oracle CG solution plus the spread of alpha_m and b under a change of the
    product's summation order (the same solver, the same eps)."""
    spec = spec_of(cfg)
    Qt, q, Qmm = O.reduced_matrix(X, spec, cfg.C)
    rhs = O.reduced_rhs(y)
    r1 = O.solve_cg(lambda v: Qt @ v, rhs, cfg.eps, cfg.max_iter)
    N = Qt.shape[0]
    h = max(1, N // 3)
    r2 = O.solve_cg(lambda v: Qt[:, :h] @ v[:h] + Qt[:, h:] @ v[h:], rhs, cfg.eps, cfg.max_iter)
    a1, b1 = O.recover(r1.x, y, q, Qmm)
    a2, b2 = O.recover(r2.x, y, q, Qmm)
    return a1, b1, r1.iterations, order_spread(a1, b1, a2, b2)


def check_train(torch, dev, cfg, ref_alpha, ref_b, ref_iters, X, y, Xte=None, f_te=None,
                spread=(0.0, 0.0)):
    """alpha~ (the CG unknowns) within the bar; alpha_m = -sum(alpha~) and b, which sum
    N rounded unknowns, within max(bar, 4 x the oracle's own summation-order spread)."""
    import paper_2202_12674_amd as P
    res = P.train(to_dev(torch, dev, X), to_dev(torch, dev, y), C=cfg.C, eps=cfg.eps,
                  max_iter=cfg.max_iter, true_residual=True, **kw_of(cfg))
    log(f"  {cfg.name}: status {res.status} it {res.iterations} (oracle {ref_iters}) "
        f"rel {res.rel_residual:.2e} true {res.true_rel_residual:.2e} "
        f"cg {res.t_cg_ms:.1f} ms")
    assert res.converged
    bar = TOL_ALPHA[cfg.dtype]
    alpha = res.alpha.cpu().numpy().astype(np.float64)
    ref_alpha = np.asarray(ref_alpha, dtype=np.float64)
    scale = np.abs(ref_alpha).max()
    e_tilde = float(np.abs(alpha[:-1] - ref_alpha[:-1]).max() / scale)
    e_m = float(abs(alpha[-1] - ref_alpha[-1]) / scale)
    eb = abs(res.b - ref_b) / max(1.0, abs(ref_b))
    tol_a, tol_b = max(bar, 4 * spread[0]), max(bar, 4 * spread[1])
    log(f"  alpha~ err {e_tilde:.2e} (bar {bar:.0e}), alpha_m err {e_m:.2e} (tol {tol_a:.2e}),"
        f" b err {eb:.2e} (tol {tol_b:.2e}); oracle order spread {spread[0]:.2e}/{spread[1]:.2e}")
    assert e_tilde <= bar
    assert e_m <= tol_a
    assert eb <= tol_b
    if cfg.dtype == "f64":
        assert abs(res.iterations - ref_iters) <= max(2, ref_iters // 10)
    else:   # fp32 products perturb the Krylov space: a few more iterations are normal
        assert res.iterations <= 2 * ref_iters + 10
    # alpha_m is minus the sum of the others (last row of Eq. (11)), up to rounding
    tol_sum = (1e-12 if cfg.dtype == "f64" else 1e-5) * max(1.0, np.abs(alpha).sum())
    assert abs(alpha.sum()) <= tol_sum
    if Xte is not None:
        scores, labels = P.predict(to_dev(torch, dev, X), res.alpha, res.b, to_dev(torch, dev, Xte),
                                   **kw_of(cfg))
        bad, ties = labels_match(labels.cpu().numpy(), f_te, bar * 10)
        log(f"  test labels: {bad} mismatches, {ties} near-ties")
        assert bad == 0
    return res


@pytest.mark.parametrize("dtype", ["f64", "f32"])
@pytest.mark.parametrize("kernel", ["linear", "poly", "rbf"])
@pytest.mark.parametrize("n,d", [(2, 3), (130, 7), (600, 50)])
def test_train_small(torch_dev, dtype, kernel, n, d):
    torch, dev = torch_dev
    cfg = small_cfg(kernel, dtype, n, d, C=1.0)
    X, y, Xte, _ = data_of(cfg)
    alpha, b, iters, spread = oracle_cg_with_spread(cfg, X, y)
    f_te = O.decision(X, alpha, b, Xte, spec_of(cfg))
    check_train(torch, dev, cfg, alpha, b, iters, X, y, Xte, f_te, spread)


def test_train_residual_replacement(torch_dev):
    """C = 100 needs more than 50 iterations, so the residual is recomputed on the way."""
    torch, dev = torch_dev
    cfg = small_cfg("rbf", "f64", 700, 12, C=100.0, eps=1e-9)
    X, y, Xte, _ = data_of(cfg)
    alpha, b, iters, spread = oracle_cg_with_spread(cfg, X, y)
    assert iters > 50
    res = check_train(torch, dev, cfg, alpha, b, iters, X, y, spread=spread)
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
    torch, dev = torch_dev
    cfg = S.CONFIGS[name]
    g = golden(name)
    log(f"train {name}")
    X, y, Xte, _ = data_of(cfg)
    assert S.sha256_arrays(X, y) == str(g["hash_train"]), "generator drifted"
    assert S.sha256_arrays(Xte) == str(g["hash_test"]), "generator drifted"
    spread = (0.0, 0.0)
    if "alpha_alt_order" in g.files:
        spread = order_spread(g["alpha"], float(g["b"]), g["alpha_alt_order"],
                              float(g["b_alt_order"]))
    check_train(torch, dev, cfg, g["alpha"], float(g["b"]), int(g["iterations"]), X, y, Xte,
                g["f_test"], spread)


# ----------------------------------------------------------- predict --------

@pytest.mark.parametrize("dtype", ["f64", "f32"])
@pytest.mark.parametrize("kernel", ["linear", "poly", "rbf"])
@pytest.mark.parametrize("n,nt,d", [(1, 5, 3), (300, 1, 9), (517, 300, 70), (700, 1100, 40)])
def test_predict_oracle_model(torch_dev, dtype, kernel, n, nt, d):
    """GPU scores for the oracle's own model equal the oracle's scores. 1100 test
    points are 9 tile rows: a full band of 8 and a band of 1 in the visit order."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg(kernel, dtype, n, d)
    X, y, _, _ = data_of(cfg)
    Xte = S.make_test(cfg, S.minmax_fit(X), n_test=nt, seed=5)[0] if n > 1 else X[:1] * 0.5
    Xte = np.ascontiguousarray(np.resize(Xte, (nt, d)).astype(cfg.np_dtype))
    alpha = np.random.default_rng(3).standard_normal(n).astype(cfg.np_dtype)
    b = 0.125
    f_ref, _ = O.predict(X, alpha, b, Xte, spec_of(cfg))
    scores, labels = P.predict(to_dev(torch, dev, X), to_dev(torch, dev, alpha), b,
                               to_dev(torch, dev, Xte), **kw_of(cfg))
    s = scores.cpu().numpy()
    tol = TOL_MV[dtype]
    assert np.abs(s - f_ref).max() / max(1.0, np.abs(f_ref).max()) <= tol * 10
    bad, _ = labels_match(labels.cpu().numpy(), f_ref, tol * 10)
    assert bad == 0


# ----------------------------------------------------- edge / errors --------

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


@pytest.mark.parametrize("kernel", ["linear", "rbf"])
def test_predict_rejects_nonfinite(torch_dev, kernel):
    """A NaN or an infinity in either point set is reported (ENONFINITE), by the
    tile path and by the linear kernel's weight shortcut alike."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    X = torch.rand(300, 7, dtype=torch.float64, device=dev)
    alpha = torch.rand(300, dtype=torch.float64, device=dev) - 0.5
    Xt = torch.rand(50, 7, dtype=torch.float64, device=dev)
    kw = dict(kernel=kernel, gamma=0.5)
    scores, _ = P.predict(X, alpha, 0.1, Xt, **kw)
    assert bool(torch.isfinite(scores).all())
    for bad_train in (True, False):
        for val in (float("nan"), float("inf")):
            A, B = X.clone(), Xt.clone()
            (A if bad_train else B)[3, 2] = val
            with pytest.raises(P.LssvmError) as e:
                P.predict(A, alpha, 0.1, B, **kw)
            assert e.value.code == -2, (bad_train, val)


def test_matvec_rejects_nonfinite(torch_dev):
    """The product entry point checks its points like training does."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    X = torch.rand(200, 5, dtype=torch.float32, device=dev)
    p = torch.rand(199, dtype=torch.float32, device=dev)
    assert bool(torch.isfinite(P.matvec(X, p, kernel="poly", gamma=0.2, coef0=1.0,
                                        degree=2)).all())
    X[17, 4] = float("nan")
    with pytest.raises(P.LssvmError) as e:
        P.matvec(X, p, kernel="poly", gamma=0.2, coef0=1.0, degree=2)
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


@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_predict_linear_shortcut_large(torch_dev, dtype):
    """Linear decision values through w = sum alpha_i x_i against the oracle's kernel
    rows at 4096 training x 1024 test points."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("linear", dtype, 4096, 1024)
    X, y, Xte, _ = data_of(cfg)
    alpha = np.random.default_rng(4).standard_normal(cfg.n).astype(cfg.np_dtype)
    b = -0.25
    f_ref, _ = O.predict(X, alpha, b, Xte, O.KernelSpec("linear"))
    scores, labels = P.predict(to_dev(torch, dev, X), to_dev(torch, dev, alpha), b,
                               to_dev(torch, dev, Xte))
    tol = TOL_MV[dtype]
    assert rel_err(scores.cpu().numpy(), f_ref) <= tol * 10
    bad, _ = labels_match(labels.cpu().numpy(), f_ref, tol * 10)
    assert bad == 0


def test_eps_sweep_matches_oracle(torch_dev):
    """The eps sweep (Sec. IV-F) against the oracle run at every eps: iterations,
    training and test accuracy, the eps the Sec. IV-B protocol picks, the
    distance between the two solutions within C (||r_gpu|| + ||r_oracle||) at
    every eps, and alpha~ within the bar once CG has converged tightly (mid-run
    CG iterates are as sensitive to rounding as the oracle's own spread shows)."""
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
        if eps <= 1e-8:   # converged tightly: the trajectories agree again
            assert e <= max(1e-9, 4 * spread)
        assert r["train_acc"] == acc_tr and r["test_acc"] == acc_te
    assert tune_eps(rows) == tune_eps(ref_rows)


# ------------------------------------------------------------ lssvm_cg_step ---

@pytest.mark.parametrize("N", [1, 255, 256, 1000, 65537, 600_001, 1 << 22])
def test_cg_step_matches_oracle(torch_dev, N):
    """One step on random vectors, including lengths past the block cap
    of the vector kernels (grid-stride regime)."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    log(f"[cg_step] N={N}")
    rng = np.random.default_rng(N)
    x, r, d = (rng.standard_normal(N) for _ in range(3))
    q = d * rng.uniform(0.5, 2.0, N)            # d^T q > 0
    rr = float(r @ r)
    xo, ro, do, rro, go, ao, bo = O.cg_step(x, r, d, q, rr)
    t = [to_dev(torch, dev, a) for a in (x, r, d, q)]
    sc = torch.tensor([rr, 0.0, 0.0, 0.0], dtype=torch.float64, device=dev)
    P.cg_step(*t, sc)
    torch.cuda.synchronize()
    got = sc.cpu().numpy()
    for name, a, ref in (("x", t[0], xo), ("r", t[1], ro), ("d", t[2], do)):
        e = rel_err(a.cpu().numpy(), ref)
        assert e <= 1e-12, (name, e)
    np.testing.assert_array_equal(t[3].cpu().numpy(), q)          # q is only read
    for k, ref in enumerate((rro, go, ao, bo)):
        assert abs(got[k] - ref) <= 1e-12 * max(abs(ref), 1e-300), (k, got[k], ref)


def test_cg_step_chained_solves_spd_system(torch_dev):
    """Steps chained on the stream with q = A d from a plain fp64 product
    reach the oracle CG iterate and, run to convergence, the direct solve."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    rng = np.random.default_rng(4)
    n = 300
    M = rng.standard_normal((n, n))
    A = M @ M.T / n + np.eye(n)
    b = rng.standard_normal(n)
    Ad = to_dev(torch, dev, A)
    x = torch.zeros(n, dtype=torch.float64, device=dev)
    r = to_dev(torch, dev, b)
    d = r.clone()
    q = torch.empty_like(r)
    sc = torch.tensor([float(b @ b), 0, 0, 0], dtype=torch.float64, device=dev)
    ws = P.alloc_workspace(P.lib().lssvm_cg_step_workspace_bytes(n), dev)
    xo, ro, do, rro = np.zeros(n), b.copy(), b.copy(), float(b @ b)
    for k in range(15):              # well above rounding level: r^T r ~ 1e-13 r0^T r0
        torch.matmul(Ad, d, out=q)
        qo = A @ do
        P.cg_step(x, r, d, q, sc, workspace=ws)
        xo, ro, do, rro, *_ = O.cg_step(xo, ro, do, qo, rro)
    torch.cuda.synchronize()
    assert rel_err(x.cpu().numpy(), xo) <= 1e-9
    assert abs(sc[0].item() - rro) <= 1e-6 * rro
    for k in range(25):
        torch.matmul(Ad, d, out=q)
        P.cg_step(x, r, d, q, sc, workspace=ws)
    torch.cuda.synchronize()
    np.testing.assert_allclose(x.cpu().numpy(), np.linalg.solve(A, b), rtol=1e-10, atol=1e-12)


def test_cg_step_breakdown_keeps_vectors(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    n = 5000
    x = torch.ones(n, dtype=torch.float64, device=dev)
    r = torch.full((n,), 2.0, dtype=torch.float64, device=dev)
    d = torch.ones(n, dtype=torch.float64, device=dev)
    q = -torch.ones(n, dtype=torch.float64, device=dev)          # d^T q < 0
    sc = torch.tensor([7.0, 0, 0, 0], dtype=torch.float64, device=dev)
    P.cg_step(x, r, d, q, sc)
    torch.cuda.synchronize()
    assert torch.all(x == 1.0) and torch.all(r == 2.0) and torch.all(d == 1.0)
    got = sc.cpu().numpy()
    assert got[0] == 7.0 and got[1] == -float(n) and got[3] == 0.0


@pytest.mark.parametrize("dtype,published", [("float32", 157.3), ("float64", 78.6)])
def test_mfma_peak_probe_is_plausible(torch_dev, dtype, published):
    """The measured matrix-core loop rate lies near the published peak (one
    resident round of back-to-back MFMAs sustains ~99% of it on gfx950) and
    not above it (a probe that lost its work would report far more)."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    tf = P.mfma_peak(getattr(torch, dtype), dev)
    log(f"[mfma peak] {dtype}: {tf:.1f} TFLOP/s (published {published})")
    assert 0.9 * published < tf < 1.02 * published


# ------------------------------------------------------------- warm start ---

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


# ---------------------------------------------------------- largest sizes ---

@pytest.mark.parametrize("dtype,kernel,n,d", [("f32", "rbf", 1 << 20, 16),
                                              ("f64", "linear", (1 << 19) + 77, 24)])
def test_matvec_large_n_sampled_rows(torch_dev, dtype, kernel, n, d):
    """The implicit product at n up to 2^20 points (33.6M tiles, a 69 GB
    workspace of tile partials): sampled rows, including the last row and
    the ragged last tile, against the oracle's rows computed one by one; over
    all rows, p^T Q~ p > 0 (Q~ is SPD) and every entry finite."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    log(f"[large n] {kernel} {dtype} n={n} d={d}")
    kw = dict(linear={}, rbf=dict(gamma=1.0 / d))[kernel]
    cfg = S.Config(f"large_{kernel}", dtype, kernel, n, d, mu=1.0, inf_frac=0.5,
                   flip_frac=0.05, C=1.0, eps=1e-6, **kw)
    X, _, _ = S.make_train(cfg)
    N = n - 1
    p = S.probe_vector(N, cfg.np_dtype)
    ws = P.alloc_workspace(P.workspace_bytes(n, d, getattr(torch, "float64" if dtype == "f64"
                                                            else "float32")), dev)
    log(f"  workspace {ws.numel() / 2**30:.1f} GiB")
    out = P.matvec(to_dev(torch, dev, X), to_dev(torch, dev, p), C=cfg.C, workspace=ws,
                   **kw_of(cfg))
    torch.cuda.synchronize()
    o = out.double().cpu().numpy()
    del ws, out
    torch.cuda.empty_cache()
    assert np.isfinite(o).all()
    assert float(p.astype(np.float64) @ o) > 0.0
    rng = np.random.default_rng(n)
    rows = np.unique(np.concatenate([[0, 1, N - 1, N - 2], N - 1 - np.arange(0, 300, 7),
                                     rng.choice(N, 24, replace=False)]))
    ref = O.reduced_rows(X.astype(np.float64), spec_of(cfg), cfg.C, rows) @ p.astype(np.float64)
    err = float(np.abs(o[rows] - ref).max() / np.abs(ref).max())
    log(f"  {len(rows)} sampled rows: max rel err {err:.2e}")
    assert err <= TOL_MV[dtype]


def test_predict_layout_beyond_one_dispatch(torch_dev):
    """2^20 test points of 4100 fp32 features: their panel layout holds 4.4e9
    elements, more than one dispatch can count, so the layout kernel strides.
    Sampled decision values against the oracle; seeded inputs drawn on the
    device."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    n, d, nt = 256, 4100, 1 << 20
    log(f"[layout > 2^32] n={n} n_test={nt} d={d}")
    g = torch.Generator(device=dev)
    g.manual_seed(2024)
    Xtr = torch.rand(n, d, dtype=torch.float32, device=dev, generator=g) * 2 - 1
    Xte = torch.rand(nt, d, dtype=torch.float32, device=dev, generator=g) * 2 - 1
    alpha = torch.randn(n, dtype=torch.float32, device=dev, generator=g)
    gamma = 1.0 / d
    scores, labels = P.predict(Xtr, alpha, 0.25, Xte, kernel="rbf", gamma=gamma)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, nt - 1, nt - 2],
                                     np.random.default_rng(3).choice(nt, 20, replace=False)]))
    idx = torch.from_numpy(rows).to(dev)
    f_ref, lab_ref = O.predict(Xtr.double().cpu().numpy(), alpha.double().cpu().numpy(), 0.25,
                               Xte[idx].double().cpu().numpy(), O.KernelSpec("rbf", gamma=gamma))
    got = scores[idx].double().cpu().numpy()
    err = float(np.abs(got - f_ref).max() / max(1.0, np.abs(f_ref).max()))
    log(f"  sampled decision values: max rel err {err:.2e}")
    assert err <= 2e-4
    del Xte, scores, labels
    torch.cuda.empty_cache()
