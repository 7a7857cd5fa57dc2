"""GPU round trip through the file formats: a training file written and read by
the native IO, trained on the GPU, the model written, read back and used for
prediction on the GPU. The model's decision values are checked against the
oracle's f(x) of the trained alpha, b, and against LIBSVM's decision value
of the model file as the plain-Python oracle reads it."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle as O
import synthdata as S
from oracle import libsvm_format as L

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2202_12674_amd as P
    P.lib()
    return torch, torch.device("cuda:0")


@pytest.mark.parametrize("kernel,dtype,n,d", [("linear", "f64", 300, 37), ("rbf", "f64", 257, 20),
                                              ("poly", "f32", 400, 64)])
def test_file_train_model_predict(torch_dev, tmp_path, kernel, dtype, n, d):
    torch, dev = torch_dev
    from paper_2202_12674_amd import _binding as B
    from paper_2202_12674_amd import files as F
    print(f"[io round trip] {kernel} {dtype} {n}x{d}", flush=True)
    sys.stdout.flush()
    kp = dict(linear=dict(gamma=1.0, coef0=0.0, degree=1),
              poly=dict(gamma=1.0 / d, coef0=1.0, degree=3),
              rbf=dict(gamma=1.0 / d, coef0=0.0, degree=1))[kernel]
    cfg = S.Config(f"io_{kernel}", dtype, kernel, n, d, mu=1.0, inf_frac=0.5, flip_frac=0.05,
                   C=1.0, eps=1e-10 if dtype == "f64" else 1e-5, **kp)
    X0, y0, scale = S.make_train(cfg)
    Xte, _ = S.make_test(cfg, scale, n_test=50)
    path = str(tmp_path / "train.libsvm")
    F.write(path, X0, y0)
    X, y = F.read(path, cfg.np_dtype, d=d)
    np.testing.assert_array_equal(X, X0)
    r = B.train(torch.from_numpy(X).to(dev), torch.from_numpy(y).to(dev), C=cfg.C, eps=cfg.eps,
                **{"kernel": kernel, **kp})
    alpha = r.alpha.cpu().numpy()
    mpath = str(tmp_path / "train.model")
    F.write_model(mpath, X, y, alpha, r.b, kernel, **kp)
    m = F.read_model(mpath, cfg.np_dtype)
    assert m.kernel == kernel and m.b == r.b
    order = np.concatenate([np.flatnonzero(y == 1), np.flatnonzero(y == -1)])
    np.testing.assert_array_equal(m.alpha, alpha[order])
    Xte_d = torch.from_numpy(Xte).to(dev)
    s_model, lab_model = B.predict(torch.from_numpy(m.X).to(dev), torch.from_numpy(m.alpha).to(dev),
                                   m.b, Xte_d, kernel=kernel, **kp)
    s_model = s_model.cpu().numpy().astype(np.float64)
    # oracle f(x) of the trained model and LIBSVM's decision value of the file
    spec = O.KernelSpec(kernel, gamma=kp["gamma"], coef0=kp["coef0"], degree=kp["degree"])
    f_ref, _ = O.predict(X, alpha, r.b, Xte, spec)
    model, Xo, coef, _ = L.read_model(mpath, cfg.np_dtype)
    dec, lab_libsvm = L.libsvm_decision(model, Xo, coef, Xte)
    tol = 1e-10 if dtype == "f64" else 2e-4
    scale_f = max(1.0, float(np.abs(f_ref).max()))
    assert np.abs(dec - f_ref).max() <= 1e-12 * scale_f
    assert np.abs(s_model - f_ref).max() <= tol * scale_f
    safe = np.abs(f_ref) > 10 * tol * scale_f
    np.testing.assert_array_equal(lab_model.cpu().numpy()[safe], lab_libsvm[safe])
