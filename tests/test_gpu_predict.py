"""GPU parity of prediction, f(x) = sum_i alpha_i k(x_i, x) + b (Eq. (10)
with the sign carried by alpha), against the CPU oracle on a given model:
scores within 10x the product bar, labels identical away from exact ties; the
linear-kernel weight shortcut; non-finite inputs; a layout beyond one
dispatch."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
import synthdata as S
from gpu_common import (GOLDEN, TOL_ALPHA, TOL_MV, SPLIT_SHAPES, TAIL_SHAPES, check_train,  # noqa: F401
                        data_of, golden, golden_tight, kw_of, labels_match, log, oracle_ref,
                        random_cases, random_large_cases, rel_err, small_cfg, spec_of,
                        to_dev)

pytestmark = pytest.mark.gpu


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
