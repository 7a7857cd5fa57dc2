"""GPU parity of the implicit product Q~ p (Eqs. (13), (16)) against the CPU
oracle on the same seeded inputs: max-norm relative error within 1e-11 (fp64)
/ 1e-5 (fp32), on small and ragged shapes, every way a product is split over
workgroups, random shapes, extreme aspect ratios, the five workloads and up
to 2^20 points (sampled rows); bitwise run-to-run determinism."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
import synthdata as S
from gpu_common import (GOLDEN, TOL_ALPHA, TOL_MV, SPLIT_SHAPES, TAIL_SHAPES, check_train,  # noqa: F401
                        data_of, golden, golden_tight, kw_of, labels_match, log, oracle_ref,
                        random_cases, random_large_cases, random_param_cases, rel_err, small_cfg,
                        spec_of,
                        to_dev)

pytestmark = pytest.mark.gpu


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


def _check_plan_product(torch, dev, P, cfg, plan):
    """Two probes and three unit columns (the first and the last tile of the
    visit order, and a diagonal entry whose 1/C term comes from one split)
    against the oracle's reduced matrix."""
    n = cfg.n
    log(f"matvec plan {plan} {cfg.name}")
    X, y, _, _ = data_of(cfg)
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), cfg.C)
    Xd = to_dev(torch, dev, X)
    for seed in (7, 8):
        p = S.probe_vector(n - 1, cfg.np_dtype, seed=seed)
        out = P.matvec(Xd, to_dev(torch, dev, p), C=cfg.C, **kw_of(cfg)).cpu().numpy()
        assert rel_err(out, Qt @ p.astype(np.float64)) <= TOL_MV[cfg.dtype]
    for j in (0, n // 2, n - 2):
        e = np.zeros(n - 1, dtype=cfg.np_dtype)
        e[j] = 1
        out = P.matvec(Xd, to_dev(torch, dev, e), C=cfg.C, **kw_of(cfg)).cpu().numpy()
        assert rel_err(out, Qt[:, j]) <= TOL_MV[cfg.dtype], j
    del Qt


@pytest.mark.parametrize("dtype,n,d,plan", SPLIT_SHAPES)
def test_matvec_linear_feature_split(torch_dev, dtype, n, d, plan):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    assert P.tile_plan(n, d, dtype, "linear") == plan
    _check_plan_product(torch, dev, P, small_cfg("linear", dtype, n, d, C=2.0), plan)


@pytest.mark.parametrize("dtype,kernel,n,d,plan", TAIL_SHAPES)
def test_matvec_tail_split(torch_dev, dtype, kernel, n, d, plan):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    assert P.tile_plan(n, d, dtype, kernel) == plan
    _check_plan_product(torch, dev, P, small_cfg(kernel, dtype, n, d, C=2.0), plan)


@pytest.mark.parametrize("kernel,dtype,n,d,C", random_cases())
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


@pytest.mark.parametrize("kernel,dtype,n,d,C,kp", random_param_cases())
def test_matvec_random_params(torch_dev, kernel, dtype, n, d, C, kp):
    """Small random shapes with random kernel parameters and C: the full
    product against the oracle's explicit Q~ p at the bar."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = S.Config(f"{kernel}_{dtype}_{n}x{d}", dtype, kernel, n, d, mu=1.0, inf_frac=0.5,
                   flip_frac=0.05, C=C, eps=1e-8, **kp)
    X, _, _ = S.make_train(cfg)
    p = S.probe_vector(n - 1, cfg.np_dtype, seed=n + d)
    out = P.matvec(to_dev(torch, dev, X), to_dev(torch, dev, p), C=C, **kw_of(cfg)).cpu().numpy()
    Qt, _, _ = O.reduced_matrix(X, spec_of(cfg), C)
    err = rel_err(out, Qt @ p.astype(np.float64))
    log(f"matvec random params {cfg.name} C={C:.3g} {kp} plan {P.tile_plan(n, d, dtype, kernel)}:"
        f" {err:.2e}")
    assert err <= TOL_MV[dtype]


@pytest.mark.parametrize("kernel,dtype,n,d,C,kp", random_large_cases())
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


@pytest.mark.parametrize("dtype,kernel,n,d", [("f32", "rbf", 1 << 20, 16),
                                              ("f64", "linear", (1 << 19) + 77, 24),
                                              ("f64", "linear", 530000, 256)])
def test_matvec_large_n_sampled_rows(torch_dev, dtype, kernel, n, d):
    """The implicit product at n up to 2^20 points (33.6M tiles adding into
    2^21 fixed-point words): sampled rows, including the last row and
    the ragged last tile, against the oracle's rows computed one by one; over
    all rows, p^T Q~ p > 0 (Q~ is SPD) and every entry finite. At 530000 x 256
    fp64 the linear product's 8.6M tiles take two launch chunks and its last
    round (11 tiles split 8 ways) runs as the trailing workgroups of the
    second."""
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


@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_unaligned_points_match_aligned(torch_dev, dtype):
    """Points whose start is not 16-byte aligned (a contiguous view one element
    into a buffer) take the layout's element-wise loads; product, training and
    prediction are bitwise those of the aligned copy, which takes its 16-byte
    loads (d is a multiple of the vector width here)."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    cfg = small_cfg("rbf", dtype, 300, 64)
    X, y, Xte, _ = data_of(cfg)
    Xa = to_dev(torch, dev, X)
    tdt = Xa.dtype

    def unaligned(A):
        buf = torch.zeros(A.size + 1, dtype=tdt, device=dev)
        U = buf[1:].view(*A.shape)
        U.copy_(torch.from_numpy(A).to(dev))
        assert U.is_contiguous() and U.data_ptr() % 16 != 0
        return U

    Xu = unaligned(X)
    p = to_dev(torch, dev, S.probe_vector(cfg.n - 1, cfg.np_dtype))
    a = P.matvec(Xa, p, C=cfg.C, **kw_of(cfg)).cpu().numpy()
    b = P.matvec(Xu, p, C=cfg.C, **kw_of(cfg)).cpu().numpy()
    assert np.array_equal(a, b)
    yd = to_dev(torch, dev, y)
    ra = P.train(Xa, yd, C=cfg.C, eps=cfg.eps, **kw_of(cfg))
    rb = P.train(Xu, yd, C=cfg.C, eps=cfg.eps, **kw_of(cfg))
    assert ra.iterations == rb.iterations and ra.b == rb.b
    assert torch.equal(ra.alpha, rb.alpha)
    sa, la = P.predict(Xa, ra.alpha, ra.b, to_dev(torch, dev, Xte), **kw_of(cfg))
    sb, lb = P.predict(Xu, rb.alpha, rb.b, unaligned(Xte), **kw_of(cfg))
    assert torch.equal(sa, sb) and torch.equal(la, lb)
