"""Native LIBSVM-format IO (include/lssvm_io.h) against the plain-Python oracle.

These calls run on the host only, so the whole suite runs without a GPU.
Reads are compared bit for bit with oracle/libsvm_format.py on seeded files
with varied formatting (signs, exponents, tabs, CRLF, blank lines, float32
near-ties) and on thread counts that move the range boundaries; writes are
read back by the oracle.
"""
from __future__ import annotations

import ctypes
import decimal
import os
import re
from fractions import Fraction

import numpy as np
import pytest

import paper_2202_12674_amd as P
from oracle import libsvm_format as L
from paper_2202_12674_amd import _binding as B
from paper_2202_12674_amd import files as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")
HEADER = os.path.join(ROOT, "include", "lssvm_io.h")


def bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint64 if a.dtype == np.float64 else np.uint32)


def assert_bit_equal(a, b):
    assert a.shape == b.shape and a.dtype == b.dtype
    np.testing.assert_array_equal(bits(a), bits(b))


def _exact(fr: Fraction) -> str:
    with decimal.localcontext() as ctx:
        ctx.prec = 2000
        return format(decimal.Decimal(fr.numerator) / decimal.Decimal(fr.denominator), "f")


def random_token(rng, dtype):
    """A number in one of several spellings, some at float32 rounding ties."""
    kind = rng.integers(0, 9)
    v = float(rng.standard_normal() * 10.0 ** rng.integers(-8, 9))
    if kind == 0:
        return repr(v)
    if kind == 1:
        return f"{v:.6e}".replace("e", "E" if rng.random() < .5 else "e")
    if kind == 2:
        return ("+" if v >= 0 else "") + f"{v:.9f}"
    if kind == 3:
        return str(int(rng.integers(-1000, 1000)))
    if kind == 4:
        return ".%d" % rng.integers(0, 10**6)
    if kind == 5:
        return "-0" if rng.random() < .5 else "0.0"
    if kind == 6:                                      # float32 midpoint +- a hair
        a = np.float32(rng.uniform(-4, 4))
        b_ = np.nextafter(a, np.float32(np.inf))
        mid = (Fraction(float(a)) + Fraction(float(b_))) / 2
        hair = Fraction(float(b_) - float(a)) / 10**15 * int(rng.integers(-1, 2))
        return _exact(mid + hair)
    if kind == 7:
        return "%dE%d" % (rng.integers(1, 99), rng.integers(-40, 41))
    return f"{v:.17g}"


def random_file(path, rng, n, d, dtype, crlf=False, blank_every=0, label_fmt=None):
    lines = []
    for i in range(n):
        if blank_every and i % blank_every == 0:
            lines.append(rng.choice(["", " ", "\t", " \t "]))
        lab = label_fmt(i) if label_fmt else rng.choice(["1", "-1", "+1", "1.0", "-1e0"])
        nnz = int(rng.integers(0, d + 1))
        idx = np.sort(rng.choice(np.arange(1, d + 1), size=nnz, replace=False))
        parts = [lab]
        for j in idx:
            sep = ""
            if rng.random() < .1:
                sep = "0" * int(rng.integers(1, 3))   # leading zeros in the index
            parts.append(f"{sep}{j}:{random_token(rng, dtype)}")
        joiner = rng.choice([" ", "\t", "  "])
        lines.append(rng.choice(["", " "]) + joiner.join(parts) + rng.choice(["", " ", "\t"]))
    eol = "\r\n" if crlf else "\n"
    text = eol.join(lines) + (eol if rng.random() < .5 else "")
    with open(path, "w", newline="") as fh:
        fh.write(text)


def test_library_exports_every_io_function():
    txt = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(lssvm_[a-z_]+)\s*\(", txt)))
    assert {"lssvm_libsvm_scan", "lssvm_libsvm_read", "lssvm_libsvm_write",
            "lssvm_model_write", "lssvm_model_scan", "lssvm_model_read"} == set(names)
    for nm in names:
        assert hasattr(P.lib(), nm), nm


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_golden_small_file(dtype):
    path = os.path.join(GOLDEN, "libsvm_small.txt")
    assert F.scan(path) == (5, 5)
    X, y = F.read(path, dtype)
    Xo, yo = L.read_data(path, dtype)
    assert_bit_equal(X, Xo)
    assert_bit_equal(y, yo)
    X7, _ = F.read(path, dtype, d=7)
    assert_bit_equal(X7, L.read_data(path, dtype, d=7)[0])


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("seed,n,d,crlf,blank", [(1, 40, 7, False, 0), (2, 120, 33, True, 5),
                                                 (3, 1, 1, False, 0), (4, 300, 64, False, 3)])
@pytest.mark.parametrize("threads", [1, 3, 8])
def test_read_matches_oracle(tmp_path, dtype, seed, n, d, crlf, blank, threads):
    rng = np.random.default_rng(seed)
    p = str(tmp_path / "f.txt")
    random_file(p, rng, n, d, dtype, crlf=crlf, blank_every=blank)
    Xo, yo = L.read_data(p, dtype)
    assert F.scan(p) == Xo.shape
    X, y = F.read(p, dtype, threads=threads)
    assert_bit_equal(X, Xo)
    assert_bit_equal(y, yo)


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_read_matches_oracle_many_ranges(tmp_path, dtype):
    """A file of ~1 MB is split into one range per thread (64 KiB minimum)."""
    rng = np.random.default_rng(11)
    p = str(tmp_path / "big.txt")
    random_file(p, rng, 1500, 40, dtype, blank_every=97)
    assert os.path.getsize(p) > 8 * 65536
    Xo, yo = L.read_data(p, dtype)
    for threads in (2, 8, 13):
        X, y = F.read(p, dtype, threads=threads)
        assert_bit_equal(X, Xo)
        assert_bit_equal(y, yo)


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("threads", [1, 4, 16])
def test_write_reads_back_exactly(tmp_path, dtype, threads):
    rng = np.random.default_rng(5)
    n, d = 257, 19
    X = (rng.standard_normal((n, d)) * 10.0 ** rng.integers(-30, 30, (n, d))).astype(dtype)
    X[rng.random((n, d)) < .3] = 0
    X[0, 0] = np.inf
    X[1, 1] = np.finfo(dtype).tiny / 4          # subnormal
    X[2, 2] = np.finfo(dtype).max
    y = np.where(rng.random(n) < .5, 1, -1).astype(dtype)
    p = str(tmp_path / "w.txt")
    F.write(p, X, y, threads=threads)
    Xo, yo = L.read_data(p, dtype, d=d)           # the oracle's strict grammar accepts it
    assert_bit_equal(Xo, X)
    assert_bit_equal(yo, y)
    Xn, yn = F.read(p, dtype, d=d)
    assert_bit_equal(Xn, X)
    with open(p) as fh:
        first = fh.readline()
    assert ":0 " not in first and not re.search(r":0$", first)   # zeros are omitted


def test_write_negative_zero_reads_as_absent(tmp_path):
    X = np.array([[-0.0, 1.0]])
    p = str(tmp_path / "z.txt")
    F.write(p, X, np.array([1.0]))
    Xr, _ = F.read(p, d=2)
    assert Xr[0, 0] == 0 and not np.signbit(Xr[0, 0])
    assert open(p).read() == "1 2:1\n"


def test_empty_file(tmp_path):
    p = str(tmp_path / "e.txt")
    open(p, "w").close()
    assert F.scan(p) == (0, 0)
    X, y = F.read(p)
    assert X.shape == (0, 0) and y.shape == (0,)
    p2 = str(tmp_path / "b.txt")
    open(p2, "w").write("\n  \n\t\n")
    assert F.scan(p2) == (0, 0)


@pytest.mark.parametrize("text", [
    "1 1:1\n1 2:1 2:3\n", "1 3:1 2:1\n", "1 1:1\n\n1 0:4\n", "1 1:\n", "1 1:x\n", "x 1:1\n",
    "1 1 :2\n", "1 1:2:3\n", "1 +1:2\n", "1 1:1\n-1 2:1e\n", "1 1:++2\n", "1\x0b1:1\n",
])
def test_malformed_lines_match_oracle(tmp_path, text):
    p = str(tmp_path / "bad.txt")
    with open(p, "w", newline="") as fh:
        fh.write(text)
    with pytest.raises(L.FormatError) as eo:
        L.read_data(p)
    n = sum(1 for ln in text.split("\n") if ln.strip(" \t\r"))
    L_ = P.lib()
    X = np.zeros((n, 8))
    y = np.zeros(n)
    code = L_.lssvm_libsvm_read(p.encode(), 0, X.ctypes.data, y.ctypes.data, n, 8, 2)
    assert code == B.EINVAL
    assert f"{p}:{eo.value.line}:" in P.last_error()


def test_read_argument_errors(tmp_path):
    p = str(tmp_path / "f.txt")
    open(p, "w").write("1 1:1 4:2\n-1 2:3\n")
    L_ = P.lib()
    X = np.zeros((2, 4))
    y = np.zeros(2)
    assert L_.lssvm_libsvm_read(p.encode(), 0, X.ctypes.data, y.ctypes.data, 3, 4, 0) == B.EINVAL
    assert "holds 2 points" in P.last_error()
    assert L_.lssvm_libsvm_read(p.encode(), 0, X.ctypes.data, y.ctypes.data, 2, 3, 0) == B.EINVAL
    assert f"{p}:1:" in P.last_error() and "exceeds d" in P.last_error()
    assert L_.lssvm_libsvm_read(p.encode(), 5, X.ctypes.data, y.ctypes.data, 2, 4, 0) == B.EINVAL
    assert L_.lssvm_libsvm_read(p.encode(), 0, None, y.ctypes.data, 2, 4, 0) == B.EINVAL
    assert L_.lssvm_libsvm_read(str(tmp_path / "none").encode(), 0, X.ctypes.data,
                                y.ctypes.data, 2, 4, 0) == B.EINVAL
    assert "cannot open" in P.last_error()
    n, d = ctypes.c_int64(), ctypes.c_int64()
    assert L_.lssvm_libsvm_scan(str(tmp_path).encode(), ctypes.byref(n), ctypes.byref(d), 0) \
        == B.EINVAL
    assert "not a regular file" in P.last_error()
    assert L_.lssvm_libsvm_scan(None, ctypes.byref(n), ctypes.byref(d), 0) == B.EINVAL
    assert L_.lssvm_libsvm_write(str(tmp_path / "no" / "dir.txt").encode(), 0, X.ctypes.data,
                                 y.ctypes.data, 2, 4, 0) == B.EINVAL
    assert "cannot create" in P.last_error()


# ------------------------------------------------------------------- models --

def _model_case(dtype, n=61, d=9, seed=8):
    rng = np.random.default_rng(seed)
    X = rng.uniform(-1, 1, (n, d)).astype(dtype)
    X[rng.random((n, d)) < .2] = 0
    y = np.where(rng.random(n) < .4, 1, -1).astype(dtype)
    alpha = (rng.standard_normal(n) * 10.0 ** rng.integers(-9, 3, n)).astype(dtype)
    return X, y, alpha


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("kernel,kt", [("linear", "linear"), ("poly", "polynomial"),
                                       ("rbf", "rbf")])
def test_model_write_read(tmp_path, dtype, kernel, kt):
    X, y, alpha = _model_case(dtype)
    b = -0.123456789012345678
    gamma, coef0, degree = 1.0 / 3.0, 0.7, 4
    p = str(tmp_path / "m.model")
    F.write_model(p, X, y, alpha, b, kernel, gamma, coef0, degree, threads=5)
    model, Xo, coef, yo = L.read_model(p, dtype)
    order = np.concatenate([np.flatnonzero(y == 1), np.flatnonzero(y == -1)])
    assert model["svm_type"] == "c_svc" and model["kernel_type"] == kt
    assert model["nr_class"] == 2 and model["label"] == [1, -1]
    assert model["nr_sv"] == [int((y == 1).sum()), int((y == -1).sum())]
    assert model["rho"] == -b
    if kernel != "linear":
        assert model["gamma"] == gamma
    if kernel == "poly":
        assert model["degree"] == degree and model["coef0"] == coef0
    assert_bit_equal(Xo, X[order])
    assert_bit_equal(coef, alpha[order])
    assert_bit_equal(yo, y[order])
    m = F.read_model(p, dtype)
    assert m.kernel == kernel and m.b == b
    assert_bit_equal(m.X, X[order])
    assert_bit_equal(m.alpha, alpha[order])
    assert_bit_equal(m.y, y[order])
    if kernel != "linear":
        assert m.gamma == gamma
    if kernel == "poly":
        assert (m.coef0, m.degree) == (coef0, degree)


def test_model_with_labels_listed_minus_first(tmp_path):
    """LIBSVM lists the classes in the order it met them; with "label -1 1" its
    decision value is -f(x), so the reader flips the signs of coef and rho."""
    text = ("svm_type c_svc\nkernel_type rbf\ngamma 0.5\nnr_class 2\ntotal_sv 3\nrho -0.25\n"
            "label -1 1\nnr_sv 1 2\nSV\n0.5 1:1 2:-1\n-0.25 2:2\n-0.25 1:-1 3:0.5\n")
    p = str(tmp_path / "neg.model")
    open(p, "w").write(text)
    m = F.read_model(p)
    model, Xo, coef, yo = L.read_model(p)
    np.testing.assert_array_equal(m.y, [-1, 1, 1])
    np.testing.assert_array_equal(m.alpha, -coef)
    assert m.b == model["rho"]
    rng = np.random.default_rng(0)
    Xt = rng.uniform(-1, 1, (20, 3))
    dec, lab = L.libsvm_decision(model, Xo, coef, Xt)
    import oracle as O
    f, lab_ls = O.predict(m.X, m.alpha, m.b, Xt, O.KernelSpec("rbf", gamma=m.gamma))
    np.testing.assert_allclose(f, -dec, rtol=1e-13, atol=1e-13)
    np.testing.assert_array_equal(lab_ls, lab)


def test_golden_model_native():
    m = F.read_model(os.path.join(GOLDEN, "model_small.txt"))
    assert m.kernel == "linear" and m.b == -0.5
    np.testing.assert_array_equal(m.X, [[1, 2, 0], [0, -1, 4], [2, 0, 1]])
    np.testing.assert_array_equal(m.alpha, [0.25, 0.5, -0.75])
    np.testing.assert_array_equal(m.y, [1, 1, -1])


@pytest.mark.parametrize("edit,msg", [
    (("nr_class 2", "nr_class 3"), "nr_class"),
    (("kernel_type rbf", "kernel_type sigmoid"), "kernel_type"),
    (("svm_type c_svc", "svm_type nu_svc"), "svm_type"),
    (("total_sv 2", "total_sv 3"), "nr_sv does not add up"),
    (("label 1 -1", "label 1 2"), "label"),
    (("gamma 0.5\n", ""), "gamma missing"),
    (("SV\n0.5 1:1\n-0.5 1:-1\n", ""), "no SV section"),
    (("SV\n", ""), "unknown model header key"),
    (("rho 0.1", "rho x"), "rho"),
    (("nr_sv 1 1", "nr_sv 2 1"), "nr_sv does not add up"),
    (("rho 0.1", "rho 0.1\nfoo 3"), "unknown model header key"),
    (("1:-1\n", "1:-1 1:2\n"), "increase"),
])
def test_model_header_errors(tmp_path, edit, msg):
    text = ("svm_type c_svc\nkernel_type rbf\ngamma 0.5\nnr_class 2\ntotal_sv 2\nrho 0.1\n"
            "label 1 -1\nnr_sv 1 1\nSV\n0.5 1:1\n-0.5 1:-1\n")
    assert edit[0] in text
    p = str(tmp_path / "bad.model")
    open(p, "w").write(text.replace(edit[0], edit[1]))
    with pytest.raises(B.LssvmError) as e:
        F.read_model(p)
    assert msg in str(e.value)


def test_model_write_rejects_bad_input(tmp_path):
    X, y, alpha = _model_case(np.float64, n=4, d=2)
    p = str(tmp_path / "m")
    y2 = y.copy()
    y2[0] = 0.5
    with pytest.raises(B.LssvmError, match="labels"):
        F.write_model(p, X, y2, alpha, 0.0)
    with pytest.raises(B.LssvmError, match="b must be finite"):
        F.write_model(p, X, y, alpha, float("nan"))
    with pytest.raises(B.LssvmError, match="gamma"):
        F.write_model(p, X, y, alpha, 0.0, "rbf", gamma=0.0)
