"""GPU: the command-line tools end to end. A seeded training file is trained
by lssvm-train, the model file is read by the plain-Python oracle reader and
its LIBSVM decision values are compared with the oracle's f(x) of its own CG
solution; lssvm-predict's labels and printed accuracy are checked against
the oracle's labels."""
from __future__ import annotations

import os
import re
import subprocess
import sys

import numpy as np
import pytest

import oracle as O
import synthdata as S
from oracle import libsvm_format as L

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "paper_2202_12674_amd", "bin")


@pytest.mark.parametrize("kernel,flag,dtype,n,d,eps", [
    ("rbf", "2", "f64", 300, 20, 1e-10), ("linear", "0", "f64", 257, 33, 1e-10),
    ("poly", "1", "f32", 400, 64, 1e-5)])
def test_train_and_predict_tools(tmp_path, kernel, flag, dtype, n, d, eps):
    from paper_2202_12674_amd import files as F
    print(f"[cli] {kernel} {dtype} {n}x{d}", flush=True)
    sys.stdout.flush()
    kp = dict(linear=dict(gamma=1.0, coef0=0.0, degree=1),
              poly=dict(gamma=1.0 / d, coef0=1.0, degree=3),
              rbf=dict(gamma=1.0 / d, coef0=0.0, degree=1))[kernel]
    cfg = S.Config(f"cli_{kernel}", dtype, kernel, n, d, mu=1.0, inf_frac=0.5, flip_frac=0.05,
                   C=1.0, eps=eps, **kp)
    X, y, scale = S.make_train(cfg)
    Xte, yte = S.make_test(cfg, scale, n_test=200)
    train, test = str(tmp_path / "train.libsvm"), str(tmp_path / "test.libsvm")
    F.write(train, X, y)
    F.write(test, Xte, yte)
    model, out = str(tmp_path / "train.model"), str(tmp_path / "pred.txt")
    prec = "64" if dtype == "f64" else "32"
    args = [os.path.join(BIN, "lssvm-train"), "-t", flag, "-c", "1", "-e", repr(eps), "-p", prec]
    if kernel != "linear":
        args += ["-g", repr(kp["gamma"]), "-r", repr(kp["coef0"]), "-d", str(kp["degree"])]
    r = subprocess.run(args + [train, model], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert re.search(r"read .* ms \| transfer .* \| cg .* \| total .* ms", r.stdout), r.stdout
    # oracle solution on the values the tool read (the file reads back exactly)
    spec = O.KernelSpec(kernel, gamma=kp["gamma"], coef0=kp["coef0"], degree=kp["degree"])
    alpha, b, _ = O.train(X.astype(np.float64), y.astype(np.float64), spec, cfg.C, eps)
    f_ref, lab_ref = O.predict(X, alpha, b, Xte, spec)
    mdl, Xm, coef, _ = L.read_model(model, np.float64)
    dec, lab_model = L.libsvm_decision(mdl, Xm, coef, Xte)
    tol = 1e-8 if dtype == "f64" else 2e-4
    scale_f = max(1.0, float(np.abs(f_ref).max()))
    assert np.abs(dec - f_ref).max() <= tol * scale_f
    r = subprocess.run([os.path.join(BIN, "lssvm-predict"), "-p", prec, test, model, out],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    labels = np.loadtxt(out, dtype=np.int64)
    safe = np.abs(f_ref) > 10 * tol * scale_f
    np.testing.assert_array_equal(labels[safe], lab_ref[safe])
    acc = float((labels == yte.astype(np.int64)).mean())
    m = re.search(r"Accuracy = ([0-9.]+)%", r.stdout)
    assert m and abs(float(m.group(1)) - 100 * acc) < 1e-3


def test_train_log_lines(tmp_path):
    """LSSVM_LOG=1 makes the training runtime report each batch of CG
    iterations and the finished training on stderr; unset, it stays silent."""
    from paper_2202_12674_amd import files as F
    cfg = S.Config("cli_log", "f64", "rbf", 200, 10, mu=1.0, inf_frac=0.5, flip_frac=0.05,
                   C=1.0, eps=1e-10, gamma=0.1)
    X, y, _ = S.make_train(cfg)
    train = str(tmp_path / "train.libsvm")
    F.write(train, X, y)
    exe = os.path.join(BIN, "lssvm-train")
    args = [exe, "-t", "2", "-g", "0.1", "-e", "1e-10", "-q", train, str(tmp_path / "m")]
    r = subprocess.run(args, capture_output=True, text=True, timeout=120,
                       env=dict(os.environ, LSSVM_LOG="1"))
    assert r.returncode == 0, r.stderr
    its = [int(m) for m in re.findall(r"\[lssvm\] CG iteration (\d+): relative residual", r.stderr)]
    assert its and its == sorted(its)
    assert re.search(r"\[lssvm\] train n=200 d=10: \d+ iterations", r.stderr)
    env = {k: v for k, v in os.environ.items() if k != "LSSVM_LOG"}
    r = subprocess.run(args, capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 0 and "[lssvm]" not in r.stderr
